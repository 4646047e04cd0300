// frontend.hip -- the two pieces of the paper's example interface around the
// search and aggregation (Appendix "Pytorch Example"):
//  * flow chaining: the example's search takes one forward (t -> t+1) and one
//    backward (t -> t-1) flow per frame while its window spans wt frames each
//    way; the offsets to frames t +- s are composed along the motion path,
//    F_{s}(x) = F_{s-1}(x) + f_{t+s-1}(x + F_{s-1}(x)) (mirrored with the
//    backward flows), each one-step flow read bilinearly at a position clamped
//    into the frame;
//  * the aggregation that keeps the k neighbours apart (the example's gather
//    returns (B, HD, K, T, F', H, W) and reduces over K afterwards, Sec. 3.2
//    aggregation): slice l holds, per output pixel, the w_l-weighted l-th
//    neighbours of the covering query patches divided by the cover count.
#include "snls_internal.h"

namespace snls {

// Bilinear read of one flow component plane at a position clamped into the frame.
SNLS_DEV float clamped_read(const float* __restrict__ f, int H, int W, float y, float x) {
  const float yc = fminf(fmaxf(y, 0.f), (float)(H - 1)), xc = fminf(fmaxf(x, 0.f), (float)(W - 1));
  const float fy = floorf(yc), fx = floorf(xc);
  const int y0 = (int)fy, x0 = (int)fx;
  const float ay = yc - fy, ax = xc - fx;
  const int y1 = min(y0 + 1, H - 1), x1 = min(x0 + 1, W - 1);
  const float top = (1.f - ax) * f[(long long)y0 * W + x0] + ax * f[(long long)y0 * W + x1];
  const float bot = (1.f - ax) * f[(long long)y1 * W + x0] + ax * f[(long long)y1 * W + x1];
  return (1.f - ay) * top + ay * bot;
}

// One thread per (b, t, direction, pixel): the chain of one-step offsets.
__global__ void __launch_bounds__(256) chain_flows_kernel(const float* __restrict__ fflow,
                                                          const float* __restrict__ bflow, int B, int T, int H,
                                                          int W, int wt, float* __restrict__ flows) {
  const long long HW = (long long)H * W;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)B * T * 2 * HW) return;
  const long long pix = gid % HW;
  const int dir = (int)((gid / HW) % 2) ? 1 : -1;
  const int t = (int)((gid / (2 * HW)) % T), b = (int)(gid / (2 * HW * T));
  const int y = (int)(pix / W), x = (int)(pix % W);
  const float* one = dir > 0 ? fflow : bflow;
  float fh = 0.f, fw = 0.f;
  for (int s = 1; s <= wt; ++s) {
    const int t1 = t + dir * (s - 1), t2 = t + dir * s;
    const int slot = dir < 0 ? wt - s : wt + s - 1;
    float* o = flows + ((((long long)b * T + t) * 2 * wt + slot) * 2) * HW + pix;
    if (t2 < 0 || t2 >= T) {  // frame outside the clip: never searched
      o[0] = 0.f;
      o[HW] = 0.f;
      continue;
    }
    const float* f1 = one + (((long long)b * T + t1) * 2) * HW;
    const float py = (float)y + fh, px = (float)x + fw;
    const float dh = clamped_read(f1, H, W, py, px), dw = clamped_read(f1 + HW, H, W, py, px);
    fh += dh;
    fw += dw;
    o[0] = fh;
    o[HW] = fw;
  }
}

snls_status launch_chain_flows(const float* fflow, const float* bflow, int B, int T, int H, int W, int wt,
                               float* flows, hipStream_t s) {
  const long long n = (long long)B * T * 2 * H * W;
  if (wt == 0 || n == 0) return SNLS_OK;
  hipLaunchKernelGGL(chain_flows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, fflow, bflow, B, T, H,
                     W, wt, flows);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

// One thread per (b, hd, l, t, channel chunk, pixel).
constexpr int kStChunk = 16;

__global__ void __launch_bounds__(256) aggregate_stacked_kernel(const float* __restrict__ v,
                                                                const float* __restrict__ wts,
                                                                const float* __restrict__ inds, Geo g,
                                                                float* __restrict__ stacked) {
  const int nchunk = (g.Ch + kStChunk - 1) / kStChunk;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (long long)g.B * g.HD * g.k * g.T * nchunk * g.HW) return;
  long long r = gid;
  const int x = (int)(r % g.W);
  r /= g.W;
  const int y = (int)(r % g.H);
  r /= g.H;
  const int chunk = (int)(r % nchunk);
  r /= nchunk;
  const int t = (int)(r % g.T);
  r /= g.T;
  const int l = (int)(r % g.k);
  r /= g.k;
  const int hd = (int)(r % g.HD);
  const int b = (int)(r / g.HD);
  const int c0 = chunk * kStChunk, nc = min(kStChunk, g.Ch - c0);
  float acc[kStChunk];
#pragma unroll
  for (int c = 0; c < kStChunk; ++c) acc[c] = 0.f;
  for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
    const int h = y - ph;
    if (h < 0 || h % g.s0 || h / g.s0 >= g.nH) continue;
    for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
      const int w = x - pw;
      if (w < 0 || w % g.s0 || w / g.s0 >= g.nW) continue;
      const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + h / g.s0) * g.nW + w / g.s0;
      const float wl = wts[row * g.k + l];
      const float* ind = inds + (row * g.k + l) * 3;
      // a neighbour adds nothing when its weight is 0, its frame is not an
      // integer in [0, T) or its offset is not finite
      if (wl == 0.f || !(ind[0] >= 0.f && ind[0] < (float)g.T) || ind[0] != floorf(ind[0]) ||
          !(fabsf(ind[1]) < kFarDisp) || !(fabsf(ind[2]) < kFarDisp))
        continue;
      int ny, nx;
      float ay, ax;
      split_disp(ind[1], &ny, &ay);
      split_disp(ind[2], &nx, &ax);
      const float* vb = v + (((long long)b * g.T + (int)ind[0]) * g.C + (long long)hd * g.Ch + c0) * g.HW;
#pragma unroll
      for (int c = 0; c < kStChunk; ++c)
        if (c < nc) acc[c] = fmaf(wl, bilinear_plane(vb + c * g.HW, g.H, g.W, y + ny, x + nx, ay, ax), acc[c]);
    }
  }
  const int cnt = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps) * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps);
  const float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
  float* ob = stacked + (((((long long)b * g.HD + hd) * g.k + l) * g.T + t) * g.Ch + c0) * g.HW +
              (long long)y * g.W + x;
#pragma unroll
  for (int c = 0; c < kStChunk; ++c)
    if (c < nc) ob[c * g.HW] = cnt > 0 ? acc[c] * inv : 0.f;
}

size_t aggregate_stacked_ws_bytes(const Geo& g) { return (size_t)g.rows * (size_t)g.k * sizeof(float); }

// The stacked gather with the caller's weights, one thread per output.
snls_status launch_gather_stacked_plain(const float* v, const float* weights, const float* inds, const Geo& g,
                                        float* stacked, hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  const int nchunk = (g.Ch + kStChunk - 1) / kStChunk;
  const long long n = (long long)g.B * g.HD * g.k * g.T * nchunk * g.HW;
  hipLaunchKernelGGL(aggregate_stacked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, v, weights, inds,
                     g, stacked);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_aggregate_stacked(const float* v, const float* dists, const float* inds, const Geo& g,
                                     float scale, float* stacked, void* ws, hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  float* wts = static_cast<float*>(ws);
  snls_status st = launch_softmax_weights(dists, inds, g, scale, wts, s);
  if (st != SNLS_OK) return st;
  const int nchunk = (g.Ch + kStChunk - 1) / kStChunk;
  const long long n = (long long)g.B * g.HD * g.k * g.T * nchunk * g.HW;
  hipLaunchKernelGGL(aggregate_stacked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, v, wts, inds, g,
                     stacked);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

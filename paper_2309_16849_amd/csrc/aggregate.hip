// aggregate.hip -- weighted patch aggregation (Sec. 3.2 "Aggregation").
//
// Gather form (no atomics, deterministic): each thread owns one output pixel
// and a chunk of channels of one head, visits every query patch covering the
// pixel, recomputes that query's softmax weights from its k scores and adds
// the weighted bilinear reads of its neighbours, then divides by the number
// of covering patches (a product of two 1-D counts).
#include "snls_internal.h"

namespace snls {

constexpr int kAggChunk = 16;  // channels per thread

// Softmax statistics of one query row: max of sign*scale*d over finite
// entries and the normaliser.
SNLS_DEV void row_softmax_stats(const float* __restrict__ d, int k, float sscale, float* m, float* z) {
  float mx = -INFINITY;
  for (int l = 0; l < k; ++l) {
    float v = d[l];
    if (isfinite(v)) mx = fmaxf(mx, sscale * v);
  }
  float s = 0.f;
  for (int l = 0; l < k; ++l) {
    float v = d[l];
    if (isfinite(v)) s += expf(sscale * v - mx);
  }
  *m = mx;
  *z = s;
}

__global__ void __launch_bounds__(256) aggregate_gather_kernel(const float* __restrict__ v,
                                                               const float* __restrict__ dists,
                                                               const float* __restrict__ inds, Geo g, float scale,
                                                               float* __restrict__ out) {
  const int nchunk = (g.Ch + kAggChunk - 1) / kAggChunk;
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long total = (long long)g.B * g.T * g.HD * nchunk * g.HW;
  if (gid >= total) return;
  int x = (int)(gid % g.W);
  long long r = gid / g.W;
  int y = (int)(r % g.H);
  r /= g.H;
  int chunk = (int)(r % nchunk);
  r /= nchunk;
  int hd = (int)(r % g.HD);
  r /= g.HD;
  int t = (int)(r % g.T);
  int b = (int)(r / g.T);
  const int c0 = hd * g.Ch + chunk * kAggChunk;
  const int nc = min(kAggChunk, g.Ch - chunk * kAggChunk);
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;

  float acc[kAggChunk];
#pragma unroll
  for (int c = 0; c < kAggChunk; ++c) acc[c] = 0.f;

  for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
    int h = y - ph;
    if (h < 0 || h % g.s0) continue;
    int mh = h / g.s0;
    if (mh >= g.nH) continue;
    for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
      int w = x - pw;
      if (w < 0 || w % g.s0) continue;
      int mw = w / g.s0;
      if (mw >= g.nW) continue;
      long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
      const float* drow = dists + row * g.k;
      const float* irow = inds + row * g.k * 3;
      float m, z;
      row_softmax_stats(drow, g.k, sscale, &m, &z);
      if (!(z > 0.f)) continue;
      float inv = 1.f / z;
      for (int l = 0; l < g.k; ++l) {
        float dl = drow[l];
        if (!isfinite(dl)) continue;
        float tf = irow[3 * l + 0];
        if (!(tf >= 0.f && tf < (float)g.T) || tf != floorf(tf)) continue;
        float py = (float)y + irow[3 * l + 1];
        float px = (float)x + irow[3 * l + 2];
        if (!(py > -1.f && py < (float)g.H && px > -1.f && px < (float)g.W)) continue;
        float wl = expf(sscale * dl - m) * inv;
        int t2 = (int)tf;
        int ny, nx;
        float ay, ax;
        split_disp(irow[3 * l + 1], &ny, &ay);
        split_disp(irow[3 * l + 2], &nx, &ax);
        const float* vb = v + (((long long)b * g.T + t2) * g.C + c0) * g.HW;
#pragma unroll
        for (int c = 0; c < kAggChunk; ++c) {
          if (c < nc) acc[c] = fmaf(wl, bilinear_plane(vb + c * g.HW, g.H, g.W, y + ny, x + nx, ay, ax), acc[c]);
        }
      }
    }
  }
  int cnt = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps) * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps);
  float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
  float* ob = out + (((long long)b * g.T + t) * g.C + c0) * g.HW + (long long)y * g.W + x;
#pragma unroll
  for (int c = 0; c < kAggChunk; ++c) {
    if (c < nc) ob[c * g.HW] = cnt > 0 ? acc[c] * inv : 0.f;
  }
}

snls_status launch_aggregate(const float* v, const float* dists, const float* inds, const Geo& g, float scale,
                             float* out, hipStream_t s) {
  const int nchunk = (g.Ch + kAggChunk - 1) / kAggChunk;
  long long total = (long long)g.B * g.T * g.HD * nchunk * g.HW;
  if (total == 0) return SNLS_OK;
  unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(aggregate_gather_kernel, dim3(blocks), dim3(256), 0, s, v, dists, inds, g, scale, out);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

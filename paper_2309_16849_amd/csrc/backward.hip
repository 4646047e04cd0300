// backward.hip -- gradients of the search + aggregation (the differentiable
// grid search of Sec. 1, through the aggregation of Sec. 3.2), with the top-k
// set held fixed.
//
// Two passes over query rows, one wave per row (lanes = channels of the
// head, 64 at a time), on channels-last copies of q, k, v and grad_out so
// that every read and every scatter of one (row, neighbour, patch pixel, tap)
// touches 64 consecutive floats:
//  1. aggregation: G_l = sum_{p,c} g~(p,c) v~_l(p,c) with g~ = grad_out/count,
//     dV += w_l g~ scattered through the bilinear taps, and the position
//     gradient w_l * g~ . dv~_l/dpos into the row's flow slot;
//  2. softmax + similarity: dd_l = sign*scale*w_l*(G_l - sum_m w_m G_m)
//     (+ grad_dists), then dQ, dK (through the taps) and the position
//     gradient dd_l * dscore/dpos into the flow slot.
// Scatters are float atomics into channels-last accumulators (the order of
// the additions, hence the last bits, may vary between runs), transposed into
// the caller's gradients at the end.
#include "snls_internal.h"

namespace snls {

namespace bwd {
constexpr int WAVES = 4;  // rows per workgroup
}

struct RowPos {
  int b, hd, t, h, w;
};

SNLS_DEV RowPos row_pos(long long row, const Geo& g) {
  RowPos rp;
  int mw = (int)(row % g.nW);
  row /= g.nW;
  int mh = (int)(row % g.nH);
  row /= g.nH;
  rp.t = (int)(row % g.T);
  row /= g.T;
  rp.hd = (int)(row % g.HD);
  rp.b = (int)(row / g.HD);
  rp.h = mh * g.s0;
  rp.w = mw * g.s0;
  return rp;
}

SNLS_DEV float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

SNLS_DEV float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Softmax statistics of a row (lanes over the k entries): max and sum of
// exp(sscale*d - max) over the finite entries.
SNLS_DEV void softmax_stats(const float* __restrict__ d, int k, float sscale, int lane, float* m, float* z) {
  float mx = -INFINITY;
  for (int l = lane; l < k; l += 64)
    if (isfinite(d[l])) mx = fmaxf(mx, sscale * d[l]);
  mx = wave_max(mx);
  float s = 0.f;
  for (int l = lane; l < k; l += 64)
    if (isfinite(d[l])) s += expf(sscale * d[l] - mx);
  *m = mx;
  *z = wave_sum(s);
}

// Neighbour l of a row: frame and decomposed displacement; false if it
// contributes nothing (frame not an integer in [0,T), displacement not finite
// or absurdly large).
SNLS_DEV bool neighbour(const float* __restrict__ irow, int l, const Geo& g, int* t2, int* ny, int* nx, float* ay,
                        float* ax) {
  float tf = irow[3 * l + 0];
  if (!(tf >= 0.f && tf < (float)g.T) || tf != floorf(tf)) return false;
  float dh = irow[3 * l + 1], dw = irow[3 * l + 2];
  if (!(fabsf(dh) < kFarDisp && fabsf(dw) < kFarDisp)) return false;
  *t2 = (int)tf;
  split_disp(dh, ny, ay);
  split_disp(dw, nx, ax);
  return true;
}

SNLS_DEV void add_flow_grad(float* grad_flows, const Geo& g, const RowPos& rp, int t2, float gh, float gw) {
  if (t2 == rp.t || !grad_flows) return;
  int slot = flow_slot(t2 - rp.t, g.wt);
  if (slot < 0 || slot >= g.nslot) return;
  long long base = (((long long)rp.b * g.T + rp.t) * g.nslot + slot) * 2;
  long long pix = (long long)rp.h * g.W + rp.w;
  atomicAdd(grad_flows + base * g.HW + pix, gh);
  atomicAdd(grad_flows + (base + 1) * g.HW + pix, gw);
}

// The four taps of a bilinear read with corner (y0, x0): channels-last
// offsets (pixel index * C), weights and in-frame flags; wave-uniform.
struct Taps {
  long long o[4];
  float w[4];
  bool in[4];
};

SNLS_DEV Taps make_taps(long long fbase, int y0, int x0, float ay, float ax, const Geo& g) {
  Taps tp;
  const int ys[4] = {y0, y0, y0 + 1, y0 + 1};
  const int xs[4] = {x0, x0 + 1, x0, x0 + 1};
  const float wy[4] = {1.f - ay, 1.f - ay, ay, ay};
  const float wx[4] = {1.f - ax, ax, 1.f - ax, ax};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tp.in[i] = ys[i] >= 0 && ys[i] < g.H && xs[i] >= 0 && xs[i] < g.W;
    tp.o[i] = (fbase + (long long)ys[i] * g.W + xs[i]) * g.C;
    tp.w[i] = wy[i] * wx[i];
  }
  return tp;
}

// Value, d/dy and d/dx of the bilinear read of channel column cc.
SNLS_DEV void tap_eval(const float* __restrict__ xcl, const Taps& tp, int cc, bool act, float ay, float ax,
                       float* val, float* gy, float* gx) {
  float v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = act && tp.in[i] ? xcl[tp.o[i] + cc] : 0.f;
  *val = tp.w[0] * v[0] + tp.w[1] * v[1] + tp.w[2] * v[2] + tp.w[3] * v[3];
  *gy = (1.f - ax) * (v[2] - v[0]) + ax * (v[3] - v[1]);
  *gx = (1.f - ay) * (v[1] - v[0]) + ay * (v[3] - v[2]);
}

SNLS_DEV void tap_scatter(float* xcl, const Taps& tp, int cc, bool act, float val) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (act && tp.in[i] && tp.w[i] != 0.f) atomicAdd(xcl + tp.o[i] + cc, tp.w[i] * val);
}

__global__ void __launch_bounds__(256) zero_kernel(float* __restrict__ p, long long n) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long stride = (long long)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = 0.f;
}

// (B,T,H,W,C) -> (B,T,C,H,W) through 64 x 64 LDS tiles.
__global__ void __launch_bounds__(256) from_channels_last_kernel(const float* __restrict__ xcl, Geo g,
                                                                 float* __restrict__ x) {
  __shared__ float tileb[64][65];
  const long long bt = blockIdx.z;
  const int c0 = blockIdx.y * 64;
  const long long p0 = (long long)blockIdx.x * 64;
  const float* src = xcl + bt * g.C * g.HW;
  float* dst = x + bt * g.C * g.HW;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const long long p = p0 + i;
    const int c = c0 + tx;
    tileb[i][tx] = (c < g.C && p < g.HW) ? src[p * g.C + c] : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i;
    const long long p = p0 + tx;
    if (c < g.C && p < g.HW) dst[(long long)c * g.HW + p] = tileb[tx][i];
  }
}

__global__ void __launch_bounds__(256) backward_agg_kernel(const float* __restrict__ vcl,
                                                           const float* __restrict__ dists,
                                                           const float* __restrict__ inds,
                                                           const float* __restrict__ gocl, Geo g, float scale,
                                                           float* __restrict__ dvcl, float* __restrict__ grad_flows,
                                                           float* __restrict__ Gws) {
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + (threadIdx.x >> 6);
  if (row >= g.rows) return;  // whole wave
  const RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, lane, &m, &z);
  const long long qbase = ((long long)rp.b * g.T + rp.t) * g.HW;  // pixel index base of the query frame
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !(z > 0.f) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) {
      if (lane == 0) Gws[row * g.k + l] = 0.f;
      continue;
    }
    const float wl = expf(sscale * drow[l] - m) / z;
    const long long fbase = ((long long)rp.b * g.T + t2) * g.HW;
    float Gl = 0.f, fh = 0.f, fw = 0.f;
    for (int c0 = 0; c0 < g.Ch; c0 += 64) {
      const int cc = rp.hd * g.Ch + c0 + lane;
      const bool act = c0 + lane < g.Ch;
      for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
        const int y = rp.h + ph;
        if (y < 0 || y >= g.H) continue;
        const int cy = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps);
        for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
          const int x = rp.w + pw;
          if (x < 0 || x >= g.W) continue;
          const float inv = 1.f / (float)(cy * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps));
          const float gg = act ? gocl[(qbase + (long long)y * g.W + x) * g.C + cc] * inv : 0.f;
          const Taps tp = make_taps(fbase, y + ny, x + nx, ay, ax, g);
          float val, gy, gx;
          tap_eval(vcl, tp, cc, act, ay, ax, &val, &gy, &gx);
          Gl = fmaf(gg, val, Gl);
          fh = fmaf(gg, gy, fh);
          fw = fmaf(gg, gx, fw);
          tap_scatter(dvcl, tp, cc, act, wl * gg);
        }
      }
    }
    Gl = wave_sum(Gl);
    fh = wave_sum(fh);
    fw = wave_sum(fw);
    if (lane == 0) {
      Gws[row * g.k + l] = Gl;
      add_flow_grad(grad_flows, g, rp, t2, wl * fh, wl * fw);
    }
  }
}

__global__ void __launch_bounds__(256) backward_search_kernel(const float* __restrict__ qcl,
                                                              const float* __restrict__ kcl,
                                                              const float* __restrict__ dists,
                                                              const float* __restrict__ inds,
                                                              const float* __restrict__ grad_dists, Geo g,
                                                              float scale, const float* __restrict__ Gws,
                                                              float* __restrict__ dqcl, float* __restrict__ dkcl,
                                                              float* __restrict__ grad_flows) {
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + (threadIdx.x >> 6);
  if (row >= g.rows) return;  // whole wave
  const RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float* Grow = Gws + row * g.k;
  const float sign = g.dist == SNLS_DIST_PROD ? 1.f : -1.f;
  const float sscale = sign * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, lane, &m, &z);
  float wg = 0.f;
  if (z > 0.f)
    for (int l = lane; l < g.k; l += 64)
      if (isfinite(drow[l])) wg += expf(sscale * drow[l] - m) / z * Grow[l];
  wg = wave_sum(wg);
  const long long qbase = ((long long)rp.b * g.T + rp.t) * g.HW;
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) continue;
    float dd = 0.f;
    if (z > 0.f) dd = sscale * (expf(sscale * drow[l] - m) / z) * (Grow[l] - wg);
    if (grad_dists) dd += grad_dists[row * g.k + l];
    if (dd == 0.f) continue;
    const long long fbase = ((long long)rp.b * g.T + t2) * g.HW;
    float fh = 0.f, fw = 0.f;
    for (int c0 = 0; c0 < g.Ch; c0 += 64) {
      const int cc = rp.hd * g.Ch + c0 + lane;
      const bool act = c0 + lane < g.Ch;
      for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
        const int y = rp.h + ph;
        if (y < 0 || y >= g.H) continue;
        for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
          const int x = rp.w + pw;
          if (x < 0 || x >= g.W) continue;
          const Taps tp = make_taps(fbase, y + ny, x + nx, ay, ax, g);
          const long long qo = (qbase + (long long)y * g.W + x) * g.C + cc;
          const float qv = act ? qcl[qo] : 0.f;
          float kv, gy, gx;
          tap_eval(kcl, tp, cc, act, ay, ax, &kv, &gy, &gx);
          float dq, dk;
          if (g.dist == SNLS_DIST_PROD) {
            dq = dd * kv;
            dk = dd * qv;
          } else {
            dq = 2.f * dd * (qv - kv);
            dk = -dq;
          }
          if (act) atomicAdd(dqcl + qo, dq);
          tap_scatter(dkcl, tp, cc, act, dk);
          fh = fmaf(dk, gy, fh);
          fw = fmaf(dk, gx, fw);
        }
      }
    }
    fh = wave_sum(fh);
    fw = wave_sum(fw);
    if (lane == 0) add_flow_grad(grad_flows, g, rp, t2, fh, fw);
  }
}

// ---- merged scatters (P <= 7, at most 64 channels per head) ----
//
// For one neighbour l of a row, the taps of the P x P patch pixels cover a
// (P+1) x (P+1) block of key positions at the neighbour's integer offset;
// each lane (channel) sums the block in registers and adds it with (P+1)^2
// atomics instead of 4 P^2.  dQ of a patch pixel sums over all k neighbours
// of the row and is added once per pixel.
template <int P>
__global__ void __launch_bounds__(256) backward_agg_block_kernel(const float* __restrict__ vcl,
                                                                 const float* __restrict__ dists,
                                                                 const float* __restrict__ inds,
                                                                 const float* __restrict__ gocl, Geo g,
                                                                 float scale, float* __restrict__ dvcl,
                                                                 float* __restrict__ grad_flows,
                                                                 float* __restrict__ Gws) {
  constexpr int PB = P + 1;
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + (threadIdx.x >> 6);
  if (row >= g.rows) return;  // whole wave
  const RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, lane, &m, &z);
  const long long qbase = ((long long)rp.b * g.T + rp.t) * g.HW;
  const int cc = rp.hd * g.Ch + lane;
  const bool act = lane < g.Ch;
  const int lo = -(P / 2);
  // g~ = grad_out / count of the patch pixels (0 outside the frame)
  float gg[P * P];
#pragma unroll
  for (int ph = 0; ph < P; ++ph)
#pragma unroll
    for (int pw = 0; pw < P; ++pw) {
      const int y = rp.h + lo + ph, x = rp.w + lo + pw;
      float v = 0.f;
      if (act && y >= 0 && y < g.H && x >= 0 && x < g.W) {
        const float inv =
            1.f / (float)(cover_count_1d(y, g.s0, g.nH, lo, P) * cover_count_1d(x, g.s0, g.nW, lo, P));
        v = gocl[(qbase + (long long)y * g.W + x) * g.C + cc] * inv;
      }
      gg[ph * P + pw] = v;
    }
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !(z > 0.f) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) {
      if (lane == 0) Gws[row * g.k + l] = 0.f;
      continue;
    }
    const float wl = expf(sscale * drow[l] - m) / z;
    const float* vf = vcl + ((long long)rp.b * g.T + t2) * g.HW * g.C + cc;
    const int Y0 = rp.h + lo + ny, X0 = rp.w + lo + nx;  // block origin
    // the block of V values (0 outside the frame)
    float vb[PB * PB];
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int Y = Y0 + a, X = X0 + c;
        vb[a * PB + c] = act && Y >= 0 && Y < g.H && X >= 0 && X < g.W ? vf[((long long)Y * g.W + X) * g.C] : 0.f;
      }
    const float w00 = (1.f - ay) * (1.f - ax), w01 = (1.f - ay) * ax, w10 = ay * (1.f - ax), w11 = ay * ax;
    float Gl = 0.f, fh = 0.f, fw = 0.f;
    float blk[PB * PB];
#pragma unroll
    for (int i = 0; i < PB * PB; ++i) blk[i] = 0.f;
#pragma unroll
    for (int ph = 0; ph < P; ++ph)
#pragma unroll
      for (int pw = 0; pw < P; ++pw) {
        const float gv = gg[ph * P + pw];
        const float v00 = vb[ph * PB + pw], v01 = vb[ph * PB + pw + 1];
        const float v10 = vb[(ph + 1) * PB + pw], v11 = vb[(ph + 1) * PB + pw + 1];
        const float val = w00 * v00 + w01 * v01 + w10 * v10 + w11 * v11;
        Gl = fmaf(gv, val, Gl);
        fh = fmaf(gv, (1.f - ax) * (v10 - v00) + ax * (v11 - v01), fh);
        fw = fmaf(gv, (1.f - ay) * (v01 - v00) + ay * (v11 - v10), fw);
        const float sv = wl * gv;
        blk[ph * PB + pw] = fmaf(w00, sv, blk[ph * PB + pw]);
        blk[ph * PB + pw + 1] = fmaf(w01, sv, blk[ph * PB + pw + 1]);
        blk[(ph + 1) * PB + pw] = fmaf(w10, sv, blk[(ph + 1) * PB + pw]);
        blk[(ph + 1) * PB + pw + 1] = fmaf(w11, sv, blk[(ph + 1) * PB + pw + 1]);
      }
    float* dvf = dvcl + ((long long)rp.b * g.T + t2) * g.HW * g.C + cc;
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int Y = Y0 + a, X = X0 + c;
        if (act && Y >= 0 && Y < g.H && X >= 0 && X < g.W && blk[a * PB + c] != 0.f)
          atomicAdd(dvf + ((long long)Y * g.W + X) * g.C, blk[a * PB + c]);
      }
    Gl = wave_sum(Gl);
    fh = wave_sum(fh);
    fw = wave_sum(fw);
    if (lane == 0) {
      Gws[row * g.k + l] = Gl;
      add_flow_grad(grad_flows, g, rp, t2, wl * fh, wl * fw);
    }
  }
}

template <int P>
__global__ void __launch_bounds__(256) backward_search_block_kernel(const float* __restrict__ qcl,
                                                                    const float* __restrict__ kcl,
                                                                    const float* __restrict__ dists,
                                                                    const float* __restrict__ inds,
                                                                    const float* __restrict__ grad_dists, Geo g,
                                                                    float scale, const float* __restrict__ Gws,
                                                                    float* __restrict__ dqcl,
                                                                    float* __restrict__ dkcl,
                                                                    float* __restrict__ grad_flows) {
  constexpr int PB = P + 1;
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + (threadIdx.x >> 6);
  if (row >= g.rows) return;  // whole wave
  const RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float* Grow = Gws + row * g.k;
  const bool ip = g.dist == SNLS_DIST_PROD;
  const float sscale = (ip ? 1.f : -1.f) * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, lane, &m, &z);
  float wg = 0.f;
  if (z > 0.f)
    for (int l = lane; l < g.k; l += 64)
      if (isfinite(drow[l])) wg += expf(sscale * drow[l] - m) / z * Grow[l];
  wg = wave_sum(wg);
  const long long qbase = ((long long)rp.b * g.T + rp.t) * g.HW;
  const int cc = rp.hd * g.Ch + lane;
  const bool act = lane < g.Ch;
  const int lo = -(P / 2);
  float qv[P * P], dq[P * P];
#pragma unroll
  for (int ph = 0; ph < P; ++ph)
#pragma unroll
    for (int pw = 0; pw < P; ++pw) {
      const int y = rp.h + lo + ph, x = rp.w + lo + pw;
      const bool in = act && y >= 0 && y < g.H && x >= 0 && x < g.W;
      qv[ph * P + pw] = in ? qcl[(qbase + (long long)y * g.W + x) * g.C + cc] : 0.f;
      dq[ph * P + pw] = 0.f;
    }
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) continue;
    float dd = 0.f;
    if (z > 0.f) dd = sscale * (expf(sscale * drow[l] - m) / z) * (Grow[l] - wg);
    if (grad_dists) dd += grad_dists[row * g.k + l];
    if (dd == 0.f) continue;
    const float* kf = kcl + ((long long)rp.b * g.T + t2) * g.HW * g.C + cc;
    const int Y0 = rp.h + lo + ny, X0 = rp.w + lo + nx;
    float kb[PB * PB];
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int Y = Y0 + a, X = X0 + c;
        kb[a * PB + c] = act && Y >= 0 && Y < g.H && X >= 0 && X < g.W ? kf[((long long)Y * g.W + X) * g.C] : 0.f;
      }
    const float w00 = (1.f - ay) * (1.f - ax), w01 = (1.f - ay) * ax, w10 = ay * (1.f - ax), w11 = ay * ax;
    float fh = 0.f, fw = 0.f;
    float blk[PB * PB];
#pragma unroll
    for (int i = 0; i < PB * PB; ++i) blk[i] = 0.f;
#pragma unroll
    for (int ph = 0; ph < P; ++ph) {
      const int y = rp.h + lo + ph;
#pragma unroll
      for (int pw = 0; pw < P; ++pw) {
        const int x = rp.w + lo + pw;
        if (y < 0 || y >= g.H || x < 0 || x >= g.W) continue;  // patch pixels outside the frame
        const float k00 = kb[ph * PB + pw], k01 = kb[ph * PB + pw + 1];
        const float k10 = kb[(ph + 1) * PB + pw], k11 = kb[(ph + 1) * PB + pw + 1];
        const float kv = w00 * k00 + w01 * k01 + w10 * k10 + w11 * k11;
        const float q = qv[ph * P + pw];
        float dqv, dk;
        if (ip) {
          dqv = dd * kv;
          dk = dd * q;
        } else {
          dqv = 2.f * dd * (q - kv);
          dk = -dqv;
        }
        dq[ph * P + pw] += dqv;
        blk[ph * PB + pw] = fmaf(w00, dk, blk[ph * PB + pw]);
        blk[ph * PB + pw + 1] = fmaf(w01, dk, blk[ph * PB + pw + 1]);
        blk[(ph + 1) * PB + pw] = fmaf(w10, dk, blk[(ph + 1) * PB + pw]);
        blk[(ph + 1) * PB + pw + 1] = fmaf(w11, dk, blk[(ph + 1) * PB + pw + 1]);
        fh = fmaf(dk, (1.f - ax) * (k10 - k00) + ax * (k11 - k01), fh);
        fw = fmaf(dk, (1.f - ay) * (k01 - k00) + ay * (k11 - k10), fw);
      }
    }
    float* dkf = dkcl + ((long long)rp.b * g.T + t2) * g.HW * g.C + cc;
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        const int Y = Y0 + a, X = X0 + c;
        if (act && Y >= 0 && Y < g.H && X >= 0 && X < g.W && blk[a * PB + c] != 0.f)
          atomicAdd(dkf + ((long long)Y * g.W + X) * g.C, blk[a * PB + c]);
      }
    fh = wave_sum(fh);
    fw = wave_sum(fw);
    if (lane == 0) add_flow_grad(grad_flows, g, rp, t2, fh, fw);
  }
#pragma unroll
  for (int ph = 0; ph < P; ++ph)
#pragma unroll
    for (int pw = 0; pw < P; ++pw) {
      const int y = rp.h + lo + ph, x = rp.w + lo + pw;
      if (act && y >= 0 && y < g.H && x >= 0 && x < g.W && dq[ph * P + pw] != 0.f)
        atomicAdd(dqcl + (qbase + (long long)y * g.W + x) * g.C + cc, dq[ph * P + pw]);
    }
}

// Workspace: G (rows x k), channels-last copies of q, k, v and grad_out, and
// channels-last accumulators of dq, dk and dv (256-byte aligned pieces).
static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t backward_ws_bytes(const Geo& g) {
  const size_t nvid = (size_t)g.B * g.T * g.C * g.HW * sizeof(float);
  return align256((size_t)g.rows * (size_t)g.k * sizeof(float)) + 7 * align256(nvid);
}

static void zero(float* p, long long n, hipStream_t s) {
  if (!p || n == 0) return;
  long long blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
}

snls_status launch_backward(const float* q, const float* k, const float* v, const float* dists, const float* inds,
                            const float* grad_out, const float* grad_dists, const Geo& g, float scale,
                            float* grad_q, float* grad_k, float* grad_v, float* grad_flows, float* ws,
                            hipStream_t s) {
  const long long nvid = (long long)g.B * g.T * g.C * g.HW;
  const long long nflow = (long long)g.B * g.T * g.nslot * 2 * g.HW;
  const size_t vb = align256((size_t)nvid * sizeof(float));
  char* base = reinterpret_cast<char*>(ws);
  float* Gws = reinterpret_cast<float*>(base);
  base += align256((size_t)g.rows * (size_t)g.k * sizeof(float));
  float* qcl = reinterpret_cast<float*>(base);
  float* kcl = reinterpret_cast<float*>(base + vb);
  float* vcl = reinterpret_cast<float*>(base + 2 * vb);
  float* gocl = reinterpret_cast<float*>(base + 3 * vb);
  float* dqcl = reinterpret_cast<float*>(base + 4 * vb);
  float* dkcl = reinterpret_cast<float*>(base + 5 * vb);
  float* dvcl = reinterpret_cast<float*>(base + 6 * vb);
  zero(dqcl, nvid, s);
  zero(dkcl, nvid, s);
  zero(dvcl, nvid, s);
  zero(grad_flows, nflow, s);
  if (nvid > 0) {
    launch_to_channels_last(q, g, qcl, s);
    launch_to_channels_last(k, g, kcl, s);
    launch_to_channels_last(v, g, vcl, s);
    launch_to_channels_last(grad_out, g, gocl, s);
  }
  if (g.rows > 0) {
    const unsigned blocks = (unsigned)((g.rows + bwd::WAVES - 1) / bwd::WAVES);
    const dim3 grid(blocks), block(64 * bwd::WAVES);
    if (g.ps <= 7 && g.Ch <= 64) {
      switch (g.ps) {
#define SNLS_BWD_CASE(P)                                                                                        \
  case P:                                                                                                       \
    hipLaunchKernelGGL(backward_agg_block_kernel<P>, grid, block, 0, s, vcl, dists, inds, gocl, g, scale, dvcl, \
                       grad_flows, Gws);                                                                        \
    hipLaunchKernelGGL(backward_search_block_kernel<P>, grid, block, 0, s, qcl, kcl, dists, inds, grad_dists, g, \
                       scale, Gws, dqcl, dkcl, grad_flows);                                                     \
    break;
        SNLS_BWD_CASE(1)
        SNLS_BWD_CASE(2)
        SNLS_BWD_CASE(3)
        SNLS_BWD_CASE(4)
        SNLS_BWD_CASE(5)
        SNLS_BWD_CASE(6)
        SNLS_BWD_CASE(7)
#undef SNLS_BWD_CASE
      }
    } else {
      hipLaunchKernelGGL(backward_agg_kernel, grid, block, 0, s, vcl, dists, inds, gocl, g, scale, dvcl, grad_flows,
                         Gws);
      hipLaunchKernelGGL(backward_search_kernel, grid, block, 0, s, qcl, kcl, dists, inds, grad_dists, g, scale,
                         Gws, dqcl, dkcl, grad_flows);
    }
  }
  if (nvid > 0) {
    dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
    hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dqcl, g, grad_q);
    hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dkcl, g, grad_k);
    hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dvcl, g, grad_v);
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

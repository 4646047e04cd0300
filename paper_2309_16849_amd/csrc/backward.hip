// backward.hip -- gradients of the search + aggregation (the differentiable
// grid search of Sec. 1, through the aggregation of Sec. 3.2), with the top-k
// set held fixed.
//
// Two passes over query rows (one thread per row):
//  1. aggregation: G_l = sum_{p,c} g~(p,c) v~_l(p,c) with g~ = grad_out/count,
//     dV += w_l g~ scattered through the bilinear taps, and the position
//     gradient w_l * g~ . dv~_l/dpos into the row's flow slot;
//  2. softmax + similarity: dd_l = sign*scale*w_l*(G_l - sum_m w_m G_m)
//     (+ grad_dists), then dQ, dK (through the taps) and the position
//     gradient dd_l * dscore/dpos into the flow slot.
// Scatters use float atomics.
#include "snls_internal.h"

namespace snls {

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

// Tap positions and weights of a bilinear read at (y0 + ay, x0 + ax).
struct Taps {
  long long o[4];
  float w[4];
  bool in[4];
};

SNLS_DEV Taps make_taps(int y0, int x0, float ay, float ax, int H, int W) {
  Taps tp;
  const int ys[4] = {y0, y0, y0 + 1, y0 + 1};
  const int xs[4] = {x0, x0 + 1, x0, x0 + 1};
  const float wy[4] = {1.f - ay, 1.f - ay, ay, ay};
  const float wx[4] = {1.f - ax, ax, 1.f - ax, ax};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tp.in[i] = ys[i] >= 0 && ys[i] < H && xs[i] >= 0 && xs[i] < W;
    tp.o[i] = (long long)ys[i] * W + xs[i];
    tp.w[i] = wy[i] * wx[i];
  }
  return tp;
}

// Value, d/dy and d/dx of the bilinear read (cell with corner (y0, x0)).
SNLS_DEV void tap_eval(const float* __restrict__ plane, const Taps& tp, float ay, float ax, float* val, float* gy,
                       float* gx) {
  float v[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = tp.in[i] ? plane[tp.o[i]] : 0.f;
  *val = tp.w[0] * v[0] + tp.w[1] * v[1] + tp.w[2] * v[2] + tp.w[3] * v[3];
  *gy = (1.f - ax) * (v[2] - v[0]) + ax * (v[3] - v[1]);
  *gx = (1.f - ay) * (v[1] - v[0]) + ay * (v[3] - v[2]);
}

SNLS_DEV void tap_scatter(float* plane, const Taps& tp, float val) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (tp.in[i] && tp.w[i] != 0.f) atomicAdd(plane + tp.o[i], tp.w[i] * val);
}

// Neighbour l of a row: frame and decomposed displacement; false if it
// contributes nothing (non-finite score, frame not an integer in [0,T),
// read position entirely outside the frame).
SNLS_DEV bool neighbour(const float* __restrict__ irow, int l, const Geo& g, int* t2, int* ny, int* nx, float* ay,
                        float* ax) {
  float tf = irow[3 * l + 0];
  if (!(tf >= 0.f && tf < (float)g.T) || tf != floorf(tf)) return false;
  float dh = irow[3 * l + 1], dw = irow[3 * l + 2];
  if (!(fabsf(dh) < 4.0e6f && fabsf(dw) < 4.0e6f)) return false;
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

SNLS_DEV void softmax_stats(const float* __restrict__ d, int k, float sscale, float* m, float* z) {
  float mx = -INFINITY;
  for (int l = 0; l < k; ++l)
    if (isfinite(d[l])) mx = fmaxf(mx, sscale * d[l]);
  float s = 0.f;
  for (int l = 0; l < k; ++l)
    if (isfinite(d[l])) s += expf(sscale * d[l] - mx);
  *m = mx;
  *z = s;
}

__global__ void __launch_bounds__(256) zero_kernel(float* __restrict__ p, long long n) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long stride = (long long)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = 0.f;
}

__global__ void __launch_bounds__(128) backward_agg_kernel(const float* __restrict__ v,
                                                           const float* __restrict__ dists,
                                                           const float* __restrict__ inds,
                                                           const float* __restrict__ grad_out, Geo g, float scale,
                                                           float* __restrict__ grad_v, float* __restrict__ grad_flows,
                                                           float* __restrict__ Gws) {
  long long row = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= g.rows) return;
  RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  float* Grow = Gws + row * g.k;
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, &m, &z);
  const long long cbase = (long long)rp.hd * g.Ch;
  for (int l = 0; l < g.k; ++l) {
    float Gl = 0.f;
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !(z > 0.f) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) {
      Grow[l] = 0.f;
      continue;
    }
    float wl = expf(sscale * drow[l] - m) / z;
    float fh = 0.f, fw = 0.f;
    const float* vb = v + (((long long)rp.b * g.T + t2) * g.C + cbase) * g.HW;
    float* gvb = grad_v + (((long long)rp.b * g.T + t2) * g.C + cbase) * g.HW;
    const float* gob = grad_out + (((long long)rp.b * g.T + rp.t) * g.C + cbase) * g.HW;
    for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
      int y = rp.h + ph;
      if (y < 0 || y >= g.H) continue;
      int cy = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps);
      for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
        int x = rp.w + pw;
        if (x < 0 || x >= g.W) continue;
        float inv = 1.f / (float)(cy * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps));
        Taps tp = make_taps(y + ny, x + nx, ay, ax, g.H, g.W);
        for (int c = 0; c < g.Ch; ++c) {
          float gg = gob[c * g.HW + (long long)y * g.W + x] * inv;
          float val, gy, gx;
          tap_eval(vb + c * g.HW, tp, ay, ax, &val, &gy, &gx);
          Gl = fmaf(gg, val, Gl);
          fh = fmaf(gg, gy, fh);
          fw = fmaf(gg, gx, fw);
          tap_scatter(gvb + c * g.HW, tp, wl * gg);
        }
      }
    }
    Grow[l] = Gl;
    add_flow_grad(grad_flows, g, rp, t2, wl * fh, wl * fw);
  }
}

__global__ void __launch_bounds__(128) backward_search_kernel(const float* __restrict__ q,
                                                              const float* __restrict__ k,
                                                              const float* __restrict__ dists,
                                                              const float* __restrict__ inds,
                                                              const float* __restrict__ grad_dists, Geo g,
                                                              float scale, const float* __restrict__ Gws,
                                                              float* __restrict__ grad_q,
                                                              float* __restrict__ grad_k,
                                                              float* __restrict__ grad_flows) {
  long long row = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= g.rows) return;
  RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float* Grow = Gws + row * g.k;
  const float sign = g.dist == SNLS_DIST_PROD ? 1.f : -1.f;
  const float sscale = sign * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, &m, &z);
  float wg = 0.f;
  if (z > 0.f)
    for (int l = 0; l < g.k; ++l)
      if (isfinite(drow[l])) wg += expf(sscale * drow[l] - m) / z * Grow[l];
  const long long cbase = (long long)rp.hd * g.Ch;
  const float* qb = q + (((long long)rp.b * g.T + rp.t) * g.C + cbase) * g.HW;
  float* gqb = grad_q + (((long long)rp.b * g.T + rp.t) * g.C + cbase) * g.HW;
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) continue;
    float dd = 0.f;
    if (z > 0.f) dd = sscale * (expf(sscale * drow[l] - m) / z) * (Grow[l] - wg);
    if (grad_dists) dd += grad_dists[row * g.k + l];
    if (dd == 0.f) continue;
    const float* kb = k + (((long long)rp.b * g.T + t2) * g.C + cbase) * g.HW;
    float* gkb = grad_k + (((long long)rp.b * g.T + t2) * g.C + cbase) * g.HW;
    float fh = 0.f, fw = 0.f;
    for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
      int y = rp.h + ph;
      if (y < 0 || y >= g.H) continue;
      for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
        int x = rp.w + pw;
        if (x < 0 || x >= g.W) continue;
        Taps tp = make_taps(y + ny, x + nx, ay, ax, g.H, g.W);
        long long qo = (long long)y * g.W + x;
        for (int c = 0; c < g.Ch; ++c) {
          float qv = qb[c * g.HW + qo];
          float kv, gy, gx;
          tap_eval(kb + c * g.HW, tp, ay, ax, &kv, &gy, &gx);
          float dq, dk;
          if (g.dist == SNLS_DIST_PROD) {
            dq = dd * kv;
            dk = dd * qv;
          } else {
            dq = 2.f * dd * (qv - kv);
            dk = -dq;
          }
          atomicAdd(gqb + c * g.HW + qo, dq);
          tap_scatter(gkb + c * g.HW, tp, dk);
          fh = fmaf(dk, gy, fh);
          fw = fmaf(dk, gx, fw);
        }
      }
    }
    add_flow_grad(grad_flows, g, rp, t2, fh, fw);
  }
}

static void zero(float* p, long long n, hipStream_t s) {
  if (!p || n == 0) return;
  long long blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
}

snls_status launch_backward(const float* q, const float* k, const float* v, const float* dists, const float* inds,
                            const float* grad_out, const float* grad_dists, const Geo& g, float scale,
                            float* grad_q, float* grad_k, float* grad_v, float* grad_flows, float* Gws,
                            hipStream_t s) {
  long long nvid = (long long)g.B * g.T * g.C * g.HW;
  long long nflow = (long long)g.B * g.T * g.nslot * 2 * g.HW;
  zero(grad_q, nvid, s);
  zero(grad_k, nvid, s);
  zero(grad_v, nvid, s);
  zero(grad_flows, nflow, s);
  if (g.rows > 0) {
    unsigned blocks = (unsigned)((g.rows + 127) / 128);
    hipLaunchKernelGGL(backward_agg_kernel, dim3(blocks), dim3(128), 0, s, v, dists, inds, grad_out, g, scale, grad_v,
                       grad_flows, Gws);
    hipLaunchKernelGGL(backward_search_kernel, dim3(blocks), dim3(128), 0, s, q, k, dists, inds, grad_dists, g,
                       scale, Gws, grad_q, grad_k, grad_flows);
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

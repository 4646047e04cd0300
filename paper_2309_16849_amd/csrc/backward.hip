// backward.hip -- gradients of the search + aggregation (the differentiable
// grid search of Sec. 1, through the aggregation of Sec. 3.2), with the top-k
// set held fixed.
//
// Two passes over query rows, one wave per row (lanes = channels of the
// head, 64 at a time), on channels-last copies of q, k, v and grad_out so
// that every read of one (row, neighbour, patch pixel, tap) touches 64
// consecutive floats:
//  1. aggregation: G_l = sum_{p,c} g~(p,c) v~_l(p,c) with g~ = grad_out/count,
//     the softmax weight w_l, and the position gradient w_l * g~ . dv~_l/dpos
//     into the row's flow slot;
//  2. softmax + similarity: dd_l = sign*scale*w_l*(G_l - sum_m w_m G_m)
//     (+ grad_dists), dQ, and the position gradient dd_l * dscore/dpos.
// The terms on the key frames -- dV = w_l g~ and dK = dd_l q (L2: 2 dd_l
// (k~ - q)) spread through the bilinear taps -- are then summed per 8 x 8
// key tile: the (row, neighbour) pairs are sorted by the tiles their tap
// blocks touch and one wave per tile adds their terms in LDS and writes the
// tile once.  dQ and the flow gradients are float atomics, and the order of
// a tile's entries follows the atomics of the sort, so the last bits may
// vary between runs.
// Heads wider than 64 channels (and P > 7) scatter every term with float
// atomics instead.  All accumulators are channels-last, transposed into the
// caller's gradients at the end.
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

// p[off] when ok, else 0, with the load itself unconditional (address 0
// when !ok, which the caller keeps valid), so that a run of such reads is
// issued back to back instead of one per branch.
SNLS_DEV float load_or_zero(const float* __restrict__ p, long long off, bool ok) {
  const float v = p[ok ? off : 0];
  return ok ? v : 0.f;
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

// The same with 16-byte accesses (C a multiple of 4): a thread reads 4
// consecutive channels of one pixel and writes 4 consecutive pixels of one
// channel (the frame's last pixels one at a time).
__global__ void __launch_bounds__(256) from_channels_last4_kernel(const float* __restrict__ xcl, Geo g,
                                                                  float* __restrict__ x) {
  __shared__ float tileb[64][65];  // [pixel][channel]
  const long long bt = blockIdx.z;
  const int c0 = blockIdx.y * 64;
  const long long p0 = (long long)blockIdx.x * 64;
  const float* src = xcl + bt * g.C * g.HW;
  float* dst = x + bt * g.C * g.HW;
  const int q4 = threadIdx.x & 15, r16 = threadIdx.x >> 4;
  for (int j = r16; j < 64; j += 16) {
    const long long p = p0 + j;
    const int c = c0 + 4 * q4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c < g.C && p < g.HW) v = *reinterpret_cast<const float4*>(src + p * g.C + c);
    tileb[j][4 * q4] = v.x;
    tileb[j][4 * q4 + 1] = v.y;
    tileb[j][4 * q4 + 2] = v.z;
    tileb[j][4 * q4 + 3] = v.w;
  }
  __syncthreads();
  for (int i = r16; i < 64; i += 16) {
    const int c = c0 + i;
    const long long p = p0 + 4 * q4;
    if (c >= g.C || p >= g.HW) continue;
    float* dp = dst + (long long)c * g.HW + p;
    if (p + 3 < g.HW && (((long long)c * g.HW + p) & 3) == 0) {
      *reinterpret_cast<float4*>(dp) = make_float4(tileb[4 * q4][i], tileb[4 * q4 + 1][i], tileb[4 * q4 + 2][i],
                                                   tileb[4 * q4 + 3][i]);
    } else {
      for (int e = 0; e < 4 && p + e < g.HW; ++e) dp[e] = tileb[4 * q4 + e][i];
    }
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

// 32-bit buffer view of a channels-last video (below 2^30 bytes on the
// paths that use it): a read sums the byte offsets of a row, a pixel column
// and the lane's channel, each kOOB when outside the frame (or, for the
// channel, past the head's channels); any sum with a kOOB term lies in
// [2^30, 3 * 2^30], past the buffer and without wrapping, so it reads 0.
constexpr unsigned kOOB = 1u << 30, kOOB2 = kOOB;
struct ClView {
  __amdgpu_buffer_rsrc_t rs;
  unsigned rowb, colb;
  SNLS_DEV float ld(unsigned off) const {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
  }
};
SNLS_DEV ClView cl_view(const float* x, const Geo& g) {
  ClView v;
  v.rs = __builtin_amdgcn_make_buffer_rsrc((void*)x, (short)0, (int)(unsigned)((long long)g.B * g.T * g.HW * g.C * 4),
                                           0x00020000);
  v.rowb = (unsigned)(g.W * g.C) * 4u;
  v.colb = (unsigned)g.C * 4u;
  return v;
}

// ---- per-row terms (P <= 7, at most 64 channels per head) ----
//
// For one neighbour l of a row, the taps of the P x P patch pixels cover a
// (P+1) x (P+1) block of key positions at the neighbour's integer offset,
// read once into registers.  These kernels form the per-row terms -- G_l,
// the flow gradients, dQ (summed over all k neighbours of the row and added
// once per patch pixel) -- and store the pair scalars w_l and dd_l; the dK and
// dV terms on the key blocks are summed per key tile further below.
template <int P>
__global__ void __launch_bounds__(256) backward_agg_block_kernel(const float* __restrict__ vcl,
                                                                 const float* __restrict__ dists,
                                                                 const float* __restrict__ inds,
                                                                 const float* __restrict__ gs, Geo g,
                                                                 float scale, float* __restrict__ grad_flows,
                                                                 float* __restrict__ Gws, float* __restrict__ wl_out) {
  constexpr int PB = P + 1;
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  if (row >= g.rows) return;  // whole wave
  const RowPos rp = row_pos(row, g);
  const float* drow = dists + row * g.k;
  const float* irow = inds + row * g.k * 3;
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  float m, z;
  softmax_stats(drow, g.k, sscale, lane, &m, &z);
  const bool act = lane < g.Ch;
  const unsigned ch4 = act ? (unsigned)(rp.hd * g.Ch + lane) * 4u : kOOB2;
  const int lo = -(P / 2);
  const ClView gv_ = cl_view(gs, g), vv = cl_view(vcl, g);
  // g~ = grad_out / count of the patch pixels (gs holds it; 0 outside the frame)
  float gg[P * P];
  {
    unsigned ro[P], co[P];
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int y = rp.h + lo + i, x = rp.w + lo + i;
      ro[i] = y >= 0 && y < g.H ? (unsigned)((rp.b * g.T + rp.t) * g.H + y) * gv_.rowb : kOOB;
      co[i] = x >= 0 && x < g.W ? (unsigned)x * gv_.colb : kOOB;
    }
#pragma unroll
    for (int ph = 0; ph < P; ++ph)
#pragma unroll
      for (int pw = 0; pw < P; ++pw) gg[ph * P + pw] = gv_.ld(ro[ph] + co[pw] + ch4);
  }
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    if (!isfinite(drow[l]) || !(z > 0.f) || !neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) {
      if (lane == 0) {
        Gws[row * g.k + l] = 0.f;
        wl_out[row * g.k + l] = 0.f;
      }
      continue;
    }
    const float wl = expf(sscale * drow[l] - m) / z;
    if (lane == 0) wl_out[row * g.k + l] = wl;
    const int Y0 = rp.h + lo + ny, X0 = rp.w + lo + nx;  // block origin
    // the block of V values (0 outside the frame)
    float vb[PB * PB];
    {
      unsigned kr[PB], kc[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        const int Y = Y0 + i, X = X0 + i;
        kr[i] = Y >= 0 && Y < g.H ? (unsigned)((rp.b * g.T + t2) * g.H + Y) * vv.rowb : kOOB;
        kc[i] = X >= 0 && X < g.W ? (unsigned)X * vv.colb : kOOB;
      }
#pragma unroll
      for (int a = 0; a < PB; ++a)
#pragma unroll
        for (int c = 0; c < PB; ++c) vb[a * PB + c] = vv.ld(kr[a] + kc[c] + ch4);
    }
    const float w00 = (1.f - ay) * (1.f - ax), w01 = (1.f - ay) * ax, w10 = ay * (1.f - ax), w11 = ay * ax;
    float Gl = 0.f, fh = 0.f, fw = 0.f;
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
                                                                    float* __restrict__ grad_flows,
                                                                    float* __restrict__ dd_out) {
  constexpr int PB = P + 1;
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * bwd::WAVES + __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
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
  const bool act = lane < g.Ch;
  const int cc = rp.hd * g.Ch + (act ? lane : 0);  // a channel of the head for every lane
  const unsigned ch4 = act ? (unsigned)cc * 4u : kOOB2;
  const int lo = -(P / 2);
  const ClView qv_ = cl_view(qcl, g), kv_ = cl_view(kcl, g);
  float qv[P * P], dq[P * P];
  {
    unsigned ro[P], co[P];
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int y = rp.h + lo + i, x = rp.w + lo + i;
      ro[i] = y >= 0 && y < g.H ? (unsigned)((rp.b * g.T + rp.t) * g.H + y) * qv_.rowb : kOOB;
      co[i] = x >= 0 && x < g.W ? (unsigned)x * qv_.colb : kOOB;
    }
#pragma unroll
    for (int ph = 0; ph < P; ++ph)
#pragma unroll
      for (int pw = 0; pw < P; ++pw) {
        qv[ph * P + pw] = qv_.ld(ro[ph] + co[pw] + ch4);
        dq[ph * P + pw] = 0.f;
      }
  }
  for (int l = 0; l < g.k; ++l) {
    int t2, ny, nx;
    float ay, ax;
    const bool ok = isfinite(drow[l]) && neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax);
    float dd = 0.f;
    if (ok) {
      if (z > 0.f) dd = sscale * (expf(sscale * drow[l] - m) / z) * (Grow[l] - wg);
      if (grad_dists) dd += grad_dists[row * g.k + l];
    }
    if (lane == 0) dd_out[row * g.k + l] = dd;
    if (!ok || dd == 0.f) continue;
    const int Y0 = rp.h + lo + ny, X0 = rp.w + lo + nx;
    float kb[PB * PB];
    {
      unsigned kr[PB], kc[PB];
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        const int Y = Y0 + i, X = X0 + i;
        kr[i] = Y >= 0 && Y < g.H ? (unsigned)((rp.b * g.T + t2) * g.H + Y) * kv_.rowb : kOOB;
        kc[i] = X >= 0 && X < g.W ? (unsigned)X * kv_.colb : kOOB;
      }
#pragma unroll
      for (int a = 0; a < PB; ++a)
#pragma unroll
        for (int c = 0; c < PB; ++c) kb[a * PB + c] = kv_.ld(kr[a] + kc[c] + ch4);
    }
    const float w00 = (1.f - ay) * (1.f - ax), w01 = (1.f - ay) * ax, w10 = ay * (1.f - ax), w11 = ay * ax;
    float fh = 0.f, fw = 0.f;
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
        fh = fmaf(dk, (1.f - ax) * (k10 - k00) + ax * (k11 - k01), fh);
        fw = fmaf(dk, (1.f - ay) * (k01 - k00) + ay * (k11 - k10), fw);
      }
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

// ---- dK and dV gathered per key tile (P <= 7, at most 64 channels per head) ----
//
// The dK and dV terms of one (row, neighbour) pair fall on the (P+1) x (P+1)
// block of key pixels its taps read.  Instead of adding them to global memory
// with float atomics, the pairs are sorted by the tile of the key frame that
// holds their block origin (4 x 8 tiles of origins; a counting sort: counts
// per tile, exclusive scan, fill).  One wave per tile sums the terms of its
// pairs in a private LDS region -- the tile's pixels plus the P rows above
// and P columns left of it, so that every block of the tile lies inside --
// and writes the region to a scratch buffer; a merge pass then adds, for
// every key pixel, the copies of the (up to 3 x 2) regions that hold it, in
// a fixed order.  The row kernels above provide the per-pair scalars: the
// softmax weight w_l (dV = w_l g~ through the taps) and dd_l (dK = dd_l q, or
// 2 dd_l (k~ - q) for L2, through the taps).
namespace bin {
constexpr int TH = 4, TW = 8;    // tile of block origins (rows, columns)
constexpr int SORT_THREADS = 256;
}  // namespace bin

// What the tile pass needs of one pair, decoded once: query frame and pixel,
// tap-block origin and fractions, dd_l.
struct alignas(32) PairRec {
  int t, h, w, Y0, X0;
  float ay, ax, dd;
};
constexpr unsigned kNoBin = 0xffffffffu;

// Adds, for every lane with `has`, one to cnt[key] -- one atomic per distinct
// key of the wave -- and returns the lane's slot: the counter's previous value
// plus the number of lower lanes with the same key.
SNLS_DEV unsigned wave_count_add(unsigned* cnt, bool has, unsigned key) {
  const int lane = (int)__lane_id();
  unsigned long long pend = __ballot(has);
  unsigned slot = 0;
  while (pend) {
    const int leader = (int)__builtin_ctzll(pend);
    const unsigned lk = (unsigned)__builtin_amdgcn_readlane((int)key, leader);
    const bool mine = ((pend >> lane) & 1ull) && key == lk;
    const unsigned long long same = __ballot(mine);
    unsigned base = 0;
    if (lane == leader) base = atomicAdd(cnt + lk, (unsigned)__popcll(same));
    base = (unsigned)__builtin_amdgcn_readlane((int)base, leader);
    if (mine) slot = base + (unsigned)lanes_below(same);
    pend &= ~same;
  }
  return slot;
}

// Per pair (one thread each, pair indices below 2^29): decode the row and the
// neighbour, write its record and its tile (kNoBin when its block misses the
// frame or the pair contributes nothing) and count it.  Block origins lie in
// [-P, H-1] x [-P, W-1]: tile (ty, tx) holds the origins with
// (Y0 + P) / TH == ty and (X0 + P) / TW == tx.
__global__ void __launch_bounds__(bin::SORT_THREADS) bin_count_kernel(const float* __restrict__ dists,
                                                                      const float* __restrict__ inds,
                                                                      const float* __restrict__ dd, Geo g, int nty,
                                                                      int ntx, PairRec* __restrict__ recs,
                                                                      unsigned* __restrict__ binfo,
                                                                      unsigned* __restrict__ counts) {
  const unsigned pair = blockIdx.x * bin::SORT_THREADS + threadIdx.x;
  const unsigned npair = (unsigned)(g.rows * g.k);
  unsigned bi = kNoBin;
  if (pair < npair) {
    const unsigned k = (unsigned)g.k;
    unsigned row = pair / k;
    const int l = (int)(pair - row * k);
    const float* irow = inds + (size_t)row * k * 3;
    const float dist = dists[pair];
    // row -> (b, hd, t, mh, mw), 32-bit (rows below 2^29)
    const int mw = (int)(row % (unsigned)g.nW);
    row /= (unsigned)g.nW;
    const int mh = (int)(row % (unsigned)g.nH);
    row /= (unsigned)g.nH;
    const int t = (int)(row % (unsigned)g.T);
    row /= (unsigned)g.T;
    const int hd = (int)(row % (unsigned)g.HD);
    const int b = (int)(row / (unsigned)g.HD);
    const int h = mh * g.s0, w = mw * g.s0;
    int t2, ny, nx;
    float ay, ax;
    if (isfinite(dist) && neighbour(irow, l, g, &t2, &ny, &nx, &ay, &ax)) {
      const int Y0 = h + g.lo + ny, X0 = w + g.lo + nx;
      if (Y0 + g.ps >= 0 && Y0 < g.H && X0 + g.ps >= 0 && X0 < g.W) {
        const int ty = (Y0 + g.ps) / bin::TH, tx = (X0 + g.ps) / bin::TW;
        bi = ((unsigned)(((b * g.HD + hd) * g.T + t2) * nty + ty)) * (unsigned)ntx + (unsigned)tx;
        PairRec r;
        r.t = t;
        r.h = h;
        r.w = w;
        r.Y0 = Y0;
        r.X0 = X0;
        r.ay = ay;
        r.ax = ax;
        r.dd = dd[pair];
        recs[pair] = r;
      }
    }
    binfo[pair] = bi;
  }
  (void)wave_count_add(counts, bi != kNoBin, bi != kNoBin ? bi : 0u);
}

// Exclusive scan of the counts (one workgroup): offsets[i] = sum of counts
// below i, offsets[nbins] = total.
__global__ void __launch_bounds__(1024) bin_scan_kernel(const unsigned* __restrict__ counts, int nbins,
                                                        unsigned* __restrict__ offsets) {
  __shared__ unsigned part[1024];
  const int tid = threadIdx.x;
  const int per = (nbins + 1023) / 1024;
  const int i0 = min(tid * per, nbins), i1 = min(i0 + per, nbins);
  unsigned sum = 0;
  for (int i = i0; i < i1; ++i) sum += counts[i];
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const unsigned v = tid >= off ? part[tid - off] : 0u;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  unsigned run = part[tid] - sum;  // exclusive prefix of this thread's segment
  for (int i = i0; i < i1; ++i) {
    offsets[i] = run;
    run += counts[i];
  }
  if (tid == 1023) offsets[nbins] = part[1023];
}

__global__ void __launch_bounds__(bin::SORT_THREADS) bin_fill_kernel(const unsigned* __restrict__ binfo, Geo g,
                                                                     const unsigned* __restrict__ offsets,
                                                                     unsigned* __restrict__ cursor,
                                                                     unsigned* __restrict__ entries) {
  const unsigned pair = blockIdx.x * bin::SORT_THREADS + threadIdx.x;
  const unsigned bi = pair < (unsigned)(g.rows * g.k) ? binfo[pair] : kNoBin;
  const bool has = bi != kNoBin;
  const unsigned slot = wave_count_add(cursor, has, has ? bi : 0u);
  if (has) entries[offsets[bi] + slot] = pair;
}

// One wave per (tile, term): blockIdx.y + term0 = 0 sums dK, 1 sums dV.  The
// wave owns its region -- key rows [TH ty - P, TH ty + TH), columns
// [TW tx - P, TW tx + TW) -- in LDS, so every addition is a plain
// read-add-write (float atomics in LDS are far slower here) at a fixed
// offset from the block origin, in the order of the tile's entry list; lanes
// are the head's channels.  Entries go in batches of 64: lane i decodes
// entry i of the batch (read offsets of its patch rows and columns, LDS index
// of its block origin, its tap weights times its scalar), and the wave then
// takes the entries from the lanes one at a time, two per step, the reads of
// a step issued a step before its additions.  Reads are 32-bit buffer loads
// whose offset is pushed past the buffer (reads 0) for pixels outside the
// frame.  The region goes to scratch (all of it, every tile: the merge reads
// no stale value).  gs is grad_out already divided by the cover count of its
// pixel.
template <int P, bool L2K>
__global__ void __launch_bounds__(64) bin_accumulate_kernel(const float* __restrict__ qcl,
                                                            const float* __restrict__ kcl,
                                                            const float* __restrict__ gs,
                                                            const PairRec* __restrict__ recs,
                                                            const float* __restrict__ wl,
                                                            const unsigned* __restrict__ offsets,
                                                            const unsigned* __restrict__ entries, Geo g, int nty,
                                                            int ntx, int term0, float* __restrict__ scratch) {
  using namespace bin;
  constexpr int PB = P + 1;
  constexpr int lo = -(P / 2);
  constexpr int RH = TH + P, RW = TW + P, RPIX = RH * RW;
  __shared__ float acc[RPIX * 64];
  const int lane = threadIdx.x;
  const int term = (int)blockIdx.y + term0;
  const bool is_v = term == 1;
  const int nbins = (int)gridDim.x;
  const int bn = (int)blockIdx.x;
  const int tx = bn % ntx, ty = (bn / ntx) % nty;
  const int f = bn / (ntx * nty);
  const int t2 = f % g.T, hd = (f / g.T) % g.HD, b = f / (g.T * g.HD);
  const int ry0 = ty * TH - P, rx0 = tx * TW - P;  // region origin
  const int ch = hd * g.Ch + (lane < g.Ch ? lane : 0);  // a channel of the head for every lane
  const unsigned ch4 = (unsigned)ch * 4u;
  constexpr bool l2k = L2K;  // the dK pass of the L2 distance (reads the key block too)
  const int H = g.H, W = g.W;
  const ClView sv = cl_view(is_v ? gs : qcl, g), kv = cl_view(kcl, g);
  const unsigned kframe = (unsigned)((b * g.T + t2) * H) * kv.rowb;  // byte offset of key frame (b, t2)
#pragma unroll
  for (int i = 0; i < RPIX; ++i) acc[i * 64 + lane] = 0.f;

  // What the wave needs of one entry (per lane: the entry of that lane).
  struct Ent {
    unsigned ro[P], co[P];     // byte offsets of the patch rows / columns (kOOB outside the frame)
    unsigned kr[PB], kc[PB];   // the same for the key block (L2 only)
    int pin;                   // patch rows | columns << 8 inside the frame (L2 only)
    int base;                  // LDS index of the block origin
    float w00, w01, w10, w11;  // tap weights (times the scalar unless L2)
    float sc;                  // the scalar (0: nothing to add)
  };
  auto decode = [&](const PairRec& r, float s) {
    Ent en;
    const unsigned qrow0 = (unsigned)((b * g.T + r.t) * H) * sv.rowb;
    int pr = 0, pc = 0;
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int y = r.h + lo + i, x = r.w + lo + i;
      const bool yin = y >= 0 && y < H, xin = x >= 0 && x < W;
      en.ro[i] = yin ? qrow0 + (unsigned)y * sv.rowb : kOOB;
      en.co[i] = xin ? (unsigned)x * sv.colb : kOOB;
      pr |= (int)yin << i;
      pc |= (int)xin << i;
    }
    en.pin = pr | (pc << 8);
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      const int Y = r.Y0 + i, X = r.X0 + i;
      en.kr[i] = Y >= 0 && Y < H ? kframe + (unsigned)Y * kv.rowb : kOOB;
      en.kc[i] = X >= 0 && X < W ? (unsigned)X * kv.colb : kOOB;
    }
    en.base = ((r.Y0 - ry0) * RW + (r.X0 - rx0)) * 64;
    const float m = l2k ? 1.f : s;
    en.w00 = (1.f - r.ay) * (1.f - r.ax) * m;
    en.w01 = (1.f - r.ay) * r.ax * m;
    en.w10 = r.ay * (1.f - r.ax) * m;
    en.w11 = r.ay * r.ax * m;
    en.sc = s;
    return en;
  };
  // entry i of the batch, from lane i
  auto get = [&](const Ent& v, int i) {
    Ent en;
    auto rd = [&](unsigned x) { return (unsigned)__builtin_amdgcn_readlane((int)x, i); };
    auto rdf = [&](float x) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), i)); };
#pragma unroll
    for (int j = 0; j < P; ++j) {
      en.ro[j] = rd(v.ro[j]);
      en.co[j] = rd(v.co[j]);
    }
    if (l2k) {
#pragma unroll
      for (int j = 0; j < PB; ++j) {
        en.kr[j] = rd(v.kr[j]);
        en.kc[j] = rd(v.kc[j]);
      }
      en.pin = (int)rd((unsigned)v.pin);
    }
    en.base = (int)rd((unsigned)v.base) + lane;
    en.w00 = rdf(v.w00);
    en.w01 = rdf(v.w01);
    en.w10 = rdf(v.w10);
    en.w11 = rdf(v.w11);
    en.sc = rdf(v.sc);
    return en;
  };
  // patch values (and for L2 the key block) of one entry
  auto load = [&](const Ent& en, float (&tp)[P * P], float (&kb)[PB * PB]) {
#pragma unroll
    for (int ph = 0; ph < P; ++ph)
#pragma unroll
      for (int pw = 0; pw < P; ++pw) tp[ph * P + pw] = sv.ld(en.ro[ph] + en.co[pw] + ch4);
    if (l2k) {
#pragma unroll
      for (int a = 0; a < PB; ++a)
#pragma unroll
        for (int c = 0; c < PB; ++c) kb[a * PB + c] = kv.ld(en.kr[a] + en.kc[c] + ch4);
    }
  };
  // term of each patch pixel, spread through the taps into the region:
  // block pixel (a, c) collects w00, w01, w10, w11 of patch pixels (a, c),
  // (a, c-1), (a-1, c), (a-1, c-1)
  auto spread = [&](const Ent& en, float (&tp)[P * P], const float (&kb)[PB * PB]) {
    if (l2k) {
      // dK of patch pixel p: 2 dd (k~ - q); patch pixels outside the frame
      // add nothing (their q and taps read 0, but the k~ term would not vanish)
#pragma unroll
      for (int ph = 0; ph < P; ++ph)
#pragma unroll
        for (int pw = 0; pw < P; ++pw) {
          const float kvv = en.w00 * kb[ph * PB + pw] + en.w01 * kb[ph * PB + pw + 1] +
                            en.w10 * kb[(ph + 1) * PB + pw] + en.w11 * kb[(ph + 1) * PB + pw + 1];
          const bool in = ((en.pin >> ph) & (en.pin >> (8 + pw)) & 1) != 0;
          tp[ph * P + pw] = in ? -(2.f * en.sc * (tp[ph * P + pw] - kvv)) : 0.f;
        }
    }
    float cur[PB * PB];
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) cur[a * PB + c] = acc[en.base + (a * RW + c) * 64];
#pragma unroll
    for (int a = 0; a < PB; ++a)
#pragma unroll
      for (int c = 0; c < PB; ++c) {
        float v = cur[a * PB + c];
        if (a > 0 && c > 0) v = fmaf(en.w11, tp[(a - 1) * P + c - 1], v);
        if (a > 0 && c < P) v = fmaf(en.w10, tp[(a - 1) * P + c], v);
        if (a < P && c > 0) v = fmaf(en.w01, tp[a * P + c - 1], v);
        if (a < P && c < P) v = fmaf(en.w00, tp[a * P + c], v);
        acc[en.base + (a * RW + c) * 64] = v;
      }
  };

  const int e0 = (int)offsets[bn], e1 = (int)offsets[bn + 1];
  for (int eb = e0; eb < e1; eb += 64) {
    const int n = min(64, e1 - eb);
    const bool mine = lane < n;
    const unsigned pr = entries[eb + (mine ? lane : 0)];
    const PairRec rv = recs[pr];
    const float s = is_v ? wl[pr] : rv.dd;
    const Ent vb = decode(rv, mine ? s : 0.f);
    // Two entries per step, pipelined D steps deep: the reads of step
    // i + D - 1 are issued before the additions of step i (D = 2 for P <= 3
    // without the key block, else 1: what the registers hold).
    constexpr int D = P <= 3 && !L2K ? 2 : 1;
    Ent es[D][2];
    float ts[D][2][P * P];
    float ks[D][2][PB * PB];
    auto fetch = [&](int step, Ent (&e)[2], float (&t)[2][P * P], float (&kk)[2][PB * PB]) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int idx = 2 * step + u;
        e[u] = get(vb, idx & 63);
        if (idx >= n) e[u].sc = 0.f;
        if (e[u].sc != 0.f) load(e[u], t[u], kk[u]);
      }
    };
#pragma unroll
    for (int d = 0; d < D - 1; ++d) fetch(d, es[d], ts[d], ks[d]);
    for (int st = 0; 2 * st < n; st += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int nd = (d + D - 1) % D;
        fetch(st + d + D - 1, es[nd], ts[nd], ks[nd]);
#pragma unroll
        for (int u = 0; u < 2; ++u)
          if (es[d][u].sc != 0.f) spread(es[d][u], ts[d][u], ks[d][u]);
      }
    }
  }
  float* dst = scratch + ((long long)term * nbins + bn) * (RPIX * 64) + lane;
#pragma unroll
  for (int px = 0; px < RPIX; ++px) dst[px * 64] = acc[px * 64 + lane];
}

// Key pixel (Y, X) of frame (b, hd, t2) sums the copies of the regions of
// tiles ty in [Y / TH, (Y + P) / TH], tx in [X / TW, (X + P) / TW] (those
// that exist), in that order, into the channels-last accumulator.  One wave
// per pixel, lanes over the head's channels; blockIdx.y + term0 picks dK / dV.
__global__ void __launch_bounds__(256) bin_merge_kernel(const float* __restrict__ scratch, Geo g, int nty, int ntx,
                                                        int term0, float* __restrict__ dkcl,
                                                        float* __restrict__ dvcl) {
  using namespace bin;
  const long long pid = (long long)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const long long npix = (long long)g.B * g.HD * g.T * g.HW;
  if (pid >= npix) return;  // whole wave
  const int lane = threadIdx.x & 63;
  const int term = (int)blockIdx.y + term0;
  const int P = g.ps, RH = TH + P, RW = TW + P;
  const long long nbins = (long long)g.B * g.HD * g.T * nty * ntx;
  const int X = (int)(pid % g.W), Y = (int)((pid / g.W) % g.H);
  const int f = (int)(pid / g.HW);
  const int t2 = f % g.T, hd = (f / g.T) % g.HD, b = f / (g.T * g.HD);
  float v = 0.f;
  const int ty1 = min((Y + P) / TH, nty - 1), tx1 = min((X + P) / TW, ntx - 1);
  for (int ty = Y / TH; ty <= ty1; ++ty)
    for (int tx = X / TW; tx <= tx1; ++tx) {
      const long long bn = ((long long)f * nty + ty) * ntx + tx;
      const int px = (Y - (ty * TH - P)) * RW + (X - (tx * TW - P));
      v += scratch[((term * nbins + bn) * (RH * RW) + px) * 64 + lane];
    }
  if (lane < g.Ch)
    (term == 1 ? dvcl : dkcl)[(((long long)b * g.T + t2) * g.HW + (long long)Y * g.W + X) * g.C + hd * g.Ch + lane] = v;
}

// grad_out (channels-last) divided in place by the number of query patches
// covering each pixel: 4 pixels per workgroup, lanes over the channels.
__global__ void __launch_bounds__(256) scale_by_cover_kernel(float* __restrict__ gcl, Geo g, int lo, int P) {
  const long long pix = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pix >= (long long)g.B * g.T * g.HW) return;
  const long long p = pix % g.HW;
  const int y = (int)(p / g.W), x = (int)(p % g.W);
  const int n = cover_count_1d(y, g.s0, g.nH, lo, P) * cover_count_1d(x, g.s0, g.nW, lo, P);
  const float inv = n > 0 ? 1.f / (float)n : 0.f;
  float* row = gcl + pix * g.C;
  for (int c = threadIdx.x & 63; c < g.C; c += 64) row[c] = row[c] * inv;
}

// Tiles of block origins per frame: origins lie in [-P, H-1] x [-P, W-1].
static int bin_nty(const Geo& g) { return (g.H - 1 + g.ps) / bin::TH + 1; }
static int bin_ntx(const Geo& g) { return (g.W - 1 + g.ps) / bin::TW + 1; }
static long long bin_count(const Geo& g) { return (long long)g.B * g.HD * g.T * bin_nty(g) * bin_ntx(g); }
// floats of the scratch regions of both terms
static long long bin_scratch_floats(const Geo& g) {
  return 2 * bin_count(g) * (bin::TH + g.ps) * (bin::TW + g.ps) * 64;
}

// The binned path: P <= 7, at most 64 channels per head, pair indices in 29
// bits, videos below 2^30 bytes (32-bit buffer offsets).
static bool bin_supported(const Geo& g) {
  if (g.ps > 7 || g.Ch > 64) return false;
  if (g.rows * (long long)g.k >= (1LL << 29)) return false;
  if ((long long)g.B * g.T * g.HW * g.C * 4 >= (1LL << 30)) return false;
  return bin_count(g) < (1LL << 30);
}

// Workspace: G (rows x k), channels-last copies of q, k, v and grad_out, and
// channels-last accumulators of dq, dk and dv (256-byte aligned pieces); on
// the binned path also the pair scalars dd and w (rows x k each), the pair
// records and tiles, the tile counts, cursors and offsets, the sorted
// entries (one per pair) and the scratch regions of both terms.
static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t backward_ws_bytes(const Geo& g) {
  const size_t nvid = (size_t)g.B * g.T * g.C * g.HW * sizeof(float);
  const size_t pairs = (size_t)g.rows * (size_t)g.k;
  size_t b = align256(pairs * sizeof(float)) + 7 * align256(nvid);
  if (bin_supported(g)) {
    const size_t nb = (size_t)bin_count(g);
    b += 2 * align256(pairs * sizeof(float)) + align256(pairs * sizeof(PairRec)) + align256(pairs * sizeof(unsigned)) +
         2 * align256(nb * sizeof(unsigned)) + align256((nb + 1) * sizeof(unsigned)) +
         align256(pairs * sizeof(unsigned)) + align256((size_t)bin_scratch_floats(g) * sizeof(float));
  }
  return b;
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
  const long long pairs = g.rows * (long long)g.k;
  const size_t vb = align256((size_t)nvid * sizeof(float));
  const size_t pb = align256((size_t)pairs * sizeof(float));
  char* base = reinterpret_cast<char*>(ws);
  float* Gws = reinterpret_cast<float*>(base);
  base += pb;
  float* qcl = reinterpret_cast<float*>(base);
  float* kcl = reinterpret_cast<float*>(base + vb);
  float* vcl = reinterpret_cast<float*>(base + 2 * vb);
  float* gocl = reinterpret_cast<float*>(base + 3 * vb);
  float* dqcl = reinterpret_cast<float*>(base + 4 * vb);
  float* dkcl = reinterpret_cast<float*>(base + 5 * vb);
  float* dvcl = reinterpret_cast<float*>(base + 6 * vb);
  base += 7 * vb;
  const bool binned = bin_supported(g) && g.rows > 0;
  const int nty = bin_nty(g), ntx = bin_ntx(g);
  const long long nbins = bin_count(g);
  float *ddws = nullptr, *wlws = nullptr;
  PairRec* recs = nullptr;
  unsigned *binfo = nullptr, *counts = nullptr, *cursor = nullptr, *offsets = nullptr, *entries = nullptr;
  float* scratch = nullptr;
  if (binned) {
    const size_t nbb = align256((size_t)nbins * sizeof(unsigned));
    ddws = reinterpret_cast<float*>(base);
    base += pb;
    wlws = reinterpret_cast<float*>(base);
    base += pb;
    recs = reinterpret_cast<PairRec*>(base);
    base += align256((size_t)pairs * sizeof(PairRec));
    binfo = reinterpret_cast<unsigned*>(base);
    base += align256((size_t)pairs * sizeof(unsigned));
    counts = reinterpret_cast<unsigned*>(base);
    cursor = reinterpret_cast<unsigned*>(base + nbb);
    offsets = reinterpret_cast<unsigned*>(base + 2 * nbb);
    base += 2 * nbb + align256((size_t)(nbins + 1) * sizeof(unsigned));
    entries = reinterpret_cast<unsigned*>(base);
    base += align256((size_t)pairs * sizeof(unsigned));
    scratch = reinterpret_cast<float*>(base);
    zero(reinterpret_cast<float*>(counts), 2 * (long long)(nbb / sizeof(unsigned)), s);  // counts and cursors
  } else {
    zero(dkcl, nvid, s);
    zero(dvcl, nvid, s);
  }
  zero(dqcl, nvid, s);
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
    if (binned) {
      const unsigned pix = (unsigned)((g.B * g.T * g.HW + 3) / 4);
      hipLaunchKernelGGL(scale_by_cover_kernel, dim3(pix), dim3(256), 0, s, gocl, g, g.lo, g.ps);
      switch (g.ps) {
#define SNLS_BWD_ROWS_CASE(P)                                                                                     \
  case P:                                                                                                         \
    hipLaunchKernelGGL(backward_agg_block_kernel<P>, grid, block, 0, s, vcl, dists, inds, gocl, g, scale,          \
                       grad_flows, Gws, wlws);                                                                    \
    hipLaunchKernelGGL(backward_search_block_kernel<P>, grid, block, 0, s, qcl, kcl, dists, inds, grad_dists, g,   \
                       scale, Gws, dqcl, grad_flows, ddws);                                                       \
    break;
        SNLS_BWD_ROWS_CASE(1)
        SNLS_BWD_ROWS_CASE(2)
        SNLS_BWD_ROWS_CASE(3)
        SNLS_BWD_ROWS_CASE(4)
        SNLS_BWD_ROWS_CASE(5)
        SNLS_BWD_ROWS_CASE(6)
        SNLS_BWD_ROWS_CASE(7)
#undef SNLS_BWD_ROWS_CASE
      }
      const unsigned sblocks = (unsigned)((pairs + bin::SORT_THREADS - 1) / bin::SORT_THREADS);
      hipLaunchKernelGGL(bin_count_kernel, dim3(sblocks), dim3(bin::SORT_THREADS), 0, s, dists, inds, ddws, g, nty,
                         ntx, recs, binfo, counts);
      hipLaunchKernelGGL(bin_scan_kernel, dim3(1), dim3(1024), 0, s, counts, (int)nbins, offsets);
      hipLaunchKernelGGL(bin_fill_kernel, dim3(sblocks), dim3(bin::SORT_THREADS), 0, s, binfo, g, offsets, cursor,
                         entries);
      // one wave per (tile, term); the L2 dK pass is a kernel of its own (it
      // also reads the key block)
      const bool l2 = g.dist != SNLS_DIST_PROD;
      const dim3 agrid((unsigned)nbins, l2 ? 1 : 2), ablock(64);
      switch (g.ps) {
#define SNLS_BWD_ACC_CASE(P)                                                                                        \
  case P:                                                                                                           \
    if (l2) {                                                                                                       \
      hipLaunchKernelGGL((bin_accumulate_kernel<P, true>), agrid, ablock, 0, s, qcl, kcl, gocl, recs, wlws, offsets, \
                         entries, g, nty, ntx, 0, scratch);                                                         \
      hipLaunchKernelGGL((bin_accumulate_kernel<P, false>), agrid, ablock, 0, s, qcl, kcl, gocl, recs, wlws,        \
                         offsets, entries, g, nty, ntx, 1, scratch);                                                \
    } else {                                                                                                        \
      hipLaunchKernelGGL((bin_accumulate_kernel<P, false>), agrid, ablock, 0, s, qcl, kcl, gocl, recs, wlws,        \
                         offsets, entries, g, nty, ntx, 0, scratch);                                                \
    }                                                                                                               \
    break;
        SNLS_BWD_ACC_CASE(1)
        SNLS_BWD_ACC_CASE(2)
        SNLS_BWD_ACC_CASE(3)
        SNLS_BWD_ACC_CASE(4)
        SNLS_BWD_ACC_CASE(5)
        SNLS_BWD_ACC_CASE(6)
        SNLS_BWD_ACC_CASE(7)
#undef SNLS_BWD_ACC_CASE
      }
      const long long npix = (long long)g.B * g.HD * g.T * g.HW;
      hipLaunchKernelGGL(bin_merge_kernel, dim3((unsigned)((npix + 3) / 4), 2), dim3(256), 0, s, scratch, g, nty, ntx,
                         0, dkcl, dvcl);
    } else {
      hipLaunchKernelGGL(backward_agg_kernel, grid, block, 0, s, vcl, dists, inds, gocl, g, scale, dvcl, grad_flows,
                         Gws);
      hipLaunchKernelGGL(backward_search_kernel, grid, block, 0, s, qcl, kcl, dists, inds, grad_dists, g, scale,
                         Gws, dqcl, dkcl, grad_flows);
    }
  }
  if (nvid > 0) {
    dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
    const bool a16 = (((uintptr_t)grad_q | (uintptr_t)grad_k | (uintptr_t)grad_v) & 15) == 0;
    if (g.C % 4 == 0 && a16) {
      hipLaunchKernelGGL(from_channels_last4_kernel, tgrid, dim3(256), 0, s, dqcl, g, grad_q);
      hipLaunchKernelGGL(from_channels_last4_kernel, tgrid, dim3(256), 0, s, dkcl, g, grad_k);
      hipLaunchKernelGGL(from_channels_last4_kernel, tgrid, dim3(256), 0, s, dvcl, g, grad_v);
    } else {
      hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dqcl, g, grad_q);
      hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dkcl, g, grad_k);
      hipLaunchKernelGGL(from_channels_last_kernel, tgrid, dim3(256), 0, s, dvcl, g, grad_v);
    }
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

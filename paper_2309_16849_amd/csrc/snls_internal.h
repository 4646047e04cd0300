// snls_internal.h -- shared definitions of the HIP implementation (not part
// of the public ABI).
//
// Geometry and conventions follow the paper's Sec. 3.1-3.2 as restated in
// include/snls.h: query grid with stride S_Q, Ws x Ws window cells at
// displacement F + S_K*(d - Ws/2) in each of the W_t = 2wt+1 frames,
// P x P patches at offsets -(P/2) .. P-1-(P/2), bilinear reads with zero
// outside the frame.
#pragma once

#include <limits.h>
#include <stdint.h>
#include "../../include/snls.h"

#ifdef __HIPCC__
#include <hip/hip_runtime.h>
#endif

namespace snls {

// Derived geometry of one call, passed to kernels by value.
struct Geo {
  int B, T, C, H, W, HD;
  int ws, wt, ps, s0;
  float s1;
  int k, dist;
  int nH, nW, Ch, r, lo, ncand, nslot;
  long long HW;    // H*W
  long long rows;  // B*HD*T*nH*nW query rows
};

// Offsets and displacements of magnitude kFarDisp or more lie outside every
// frame (check_params limits H and W to below it): every tap of such a read
// is out of the frame, so such a neighbour contributes nothing and its
// window needs no key region.  One constant for the forward and backward
// kernels.
constexpr float kFarDisp = 1.0e6f;

// Host-side checks (validate.cpp).  Return SNLS_OK or an error code; they
// never touch the GPU.
snls_status check_params(const snls_params* p, bool need_k, Geo* g);
snls_status check_topk_args(int64_t rows, int32_t n_cand, int32_t k, int32_t dist_type);

// Device workspace of snls_aggregate: softmax weights (rows x k) then a
// channels-last copy of V, 256-byte aligned.
size_t aggregate_ws_bytes(const Geo& g);
// Device workspace of snls_backward: per-neighbour aggregation terms (rows x
// k), channels-last copies of q, k, v, grad_out and accumulators of dq, dk, dv.
size_t backward_ws_bytes(const Geo& g);
// Device workspace of snls_aggregate_stacked: softmax weights (rows x k).
size_t aggregate_stacked_ws_bytes(const Geo& g);
// The code example's gather with caller weights and its reduction over the
// neighbours: tiled kernels when a head has at most 64 channels (a multiple
// of 4) and a tile at most 256 covering queries; their workspace is a
// channels-last copy of v (0 bytes when the plain gather runs instead).
bool gather_tile_supported(const Geo& g);
bool reduce_supported(const Geo& g, int cout);
size_t gather_ws_bytes(const Geo& g);

// The tiled search path (S_Q = 1, P <= 7, Ws <= 9; inner product with
// S_K <= 1, squared L2 with S_K = 1) and its workspace: the inner-product
// score of every candidate (rows x candidates fp32), plus for L2 the key-norm
// term of every candidate and the query-norm term of every row.
bool tile_supported(const Geo& g);
size_t tile_ws_bytes(const Geo& g);
// Single-pixel patches (P = 1), any S_Q, S_K = 1, inner product, Ws <= 15:
// same workspace layout (scores of every candidate) for k > 32; for k <= 32
// (p1_fused) the selection runs inside the scoring kernel, no workspace.
bool p1_supported(const Geo& g);
bool p1_fused(const Geo& g);

// Kernels a top-k search (k >= 1) runs on.
enum class SearchRoute { Direct, Tile, P1Scored, P1Fused };
SearchRoute search_route(const Geo& g);

#ifdef __HIPCC__

// Launchers (one per kernel family); all return SNLS_OK or SNLS_ERR_HIP.
snls_status launch_search_full(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, hipStream_t s);
snls_status launch_search_topk(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, void* ws, hipStream_t s);
snls_status launch_search_topk_direct(const float* q, const float* k, const float* flows, const Geo& g,
                                      float* dists, float* inds, hipStream_t s);
snls_status launch_search_tile(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, float* scores, hipStream_t s);
snls_status launch_search_p1(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                             float* inds, float* scores, hipStream_t s);
snls_status launch_search_p1_scores(const float* q, const float* k, const float* flows, const Geo& g, float* scores,
                                    int pitch, hipStream_t s);
snls_status launch_search_p1_topk(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                                  float* inds, hipStream_t s);
// L2 norm terms: key pair planes (workspace of l2_planes_bytes(g) bytes),
// then the key-norm terms G (rows x pitch) and the query norms Qn (rows).
size_t l2_planes_bytes(const Geo& g);
snls_status launch_l2_norms(const float* q, const float* k, const float* flows, const Geo& g, float* G, int pitch,
                            float* Qn, float* planes, hipStream_t s);
snls_status launch_topk(const float* dall, const float* iall, int64_t rows, int ncand, int k, int dist,
                        float* dists, float* inds, hipStream_t s);
snls_status launch_aggregate(const float* v, const float* dists, const float* inds, const Geo& g, float scale,
                             float* out, void* ws, hipStream_t s);
snls_status launch_to_channels_last(const float* x, const Geo& g, float* xcl, hipStream_t s);
snls_status launch_softmax_weights(const float* dists, const float* inds, const Geo& g, float scale, float* wts,
                                   hipStream_t s);
snls_status launch_chain_flows(const float* fflow, const float* bflow, int B, int T, int H, int W, int wt,
                               float* flows, hipStream_t s);
snls_status launch_aggregate_stacked(const float* v, const float* dists, const float* inds, const Geo& g,
                                     float scale, float* stacked, void* ws, hipStream_t s);
snls_status launch_gather_stacked_plain(const float* v, const float* weights, const float* inds, const Geo& g,
                                        float* stacked, hipStream_t s);
snls_status launch_gather_stacked(const float* v, const float* weights, const float* inds, const Geo& g,
                                  float* stacked, void* ws, hipStream_t s);
snls_status launch_stacked_reduce(const float* stacked, const float* proj, const Geo& g, int cout, float* out,
                                  hipStream_t s);
snls_status launch_gather_reduce(const float* v, const float* weights, const float* inds, const float* proj,
                                 const Geo& g, int cout, float* out, void* ws, hipStream_t s);
snls_status launch_backward(const float* q, const float* k, const float* v, const float* dists, const float* inds,
                            const float* grad_out, const float* grad_dists, const Geo& g, float scale,
                            float* grad_q, float* grad_k, float* grad_v, float* grad_flows, float* Gws,
                            hipStream_t s);

// ---------------------------------------------------------------- device --

#define SNLS_DEV __device__ __forceinline__


// Candidate displacement disp = fl32(F + fl32(S_K * (d - r))), rounded once
// per operation (no contraction), the fp32 convention of the outputs.
SNLS_DEV float cand_disp(float F, float s1, int d, int r) {
#pragma clang fp contract(off)  // two roundings, never one fused multiply-add
  return F + s1 * (float)(d - r);
}

// Centre (h + disp) inside [0, H-1]; exact: -h and H-1-h are exact in fp32.
SNLS_DEV bool centre_ok(int h, float disp, int H) { return disp >= (float)(-h) && disp <= (float)(H - 1 - h); }

// Neighbour slot of a frame step dt != 0 (dt = -wt..-1 -> 0..wt-1, 1..wt -> wt..2wt-1).
SNLS_DEV int flow_slot(int dt, int wt) { return dt < 0 ? dt + wt : dt + wt - 1; }

// Score with "larger is better" for both distances: s = d (inner product),
// s = -d (L2).  Invalid candidates map to -inf either way.
SNLS_DEV float to_score(float d, int dist) { return dist == SNLS_DIST_PROD ? d : -d; }
SNLS_DEV float from_score(float s, int dist) { return dist == SNLS_DIST_PROD ? s : -s; }

// (s1, id1) ranks before (s2, id2): larger score, ties to the smaller id.
SNLS_DEV bool ranks_before(float s1, int id1, float s2, int id2) { return s1 > s2 || (s1 == s2 && id1 < id2); }

// Bilinear read of one channel plane at integer corner (y0, x0) with
// fractional weights (ay, ax); taps outside the frame read 0.
SNLS_DEV float bilinear_plane(const float* __restrict__ plane, int H, int W, int y0, int x0, float ay, float ax) {
  const bool y0in = y0 >= 0 && y0 < H, y1in = y0 + 1 >= 0 && y0 + 1 < H;
  const bool x0in = x0 >= 0 && x0 < W, x1in = x0 + 1 >= 0 && x0 + 1 < W;
  const long long o = (long long)y0 * W + x0;
  float v00 = (y0in && x0in) ? plane[o] : 0.f;
  float v01 = (y0in && x1in) ? plane[o + 1] : 0.f;
  float v10 = (y1in && x0in) ? plane[o + W] : 0.f;
  float v11 = (y1in && x1in) ? plane[o + W + 1] : 0.f;
  float top = (1.f - ax) * v00 + ax * v01;
  float bot = (1.f - ax) * v10 + ax * v11;
  return (1.f - ay) * top + ay * bot;
}

// Split a displacement into integer part and fraction (disp = n + a, a in [0,1)).
SNLS_DEV void split_disp(float disp, int* n, float* a) {
  float f = floorf(disp);
  *n = (int)f;
  *a = disp - f;
}

// Number of query patches covering pixel coordinate y along one axis: grid
// positions m*S (0 <= m < n) with y - m*S in [lo, lo+P-1].
SNLS_DEV int cover_count_1d(int y, int S, int n, int lo, int P) {
  int a = y - lo - P + 1;  // m*S >= a
  int b = y - lo;          // m*S <= b
  if (b < 0) return 0;
  int mmin = a <= 0 ? 0 : (a + S - 1) / S;
  int mmax = b / S;
  if (mmax > n - 1) mmax = n - 1;
  return mmax >= mmin ? mmax - mmin + 1 : 0;
}

// Patch similarity of a valid candidate with displacement (disp_h, disp_w)
// in frame t2 for the query (b, hd, t, h, w): inner product or squared L2
// over the query pixels inside the frame and the head's channels, with
// bilinear reads of the key frame (the direct in-place computation).
SNLS_DEV float score_candidate(const float* __restrict__ q, const float* __restrict__ k, const Geo& g, int b,
                               int hd, int t, int h, int w, int t2, float disp_h, float disp_w) {
  int nh, nw;
  float ah, aw;
  split_disp(disp_h, &nh, &ah);
  split_disp(disp_w, &nw, &aw);
  const float* qbase = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;
  const float* kbase = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
  float acc = 0.f;
  for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
    int y = h + ph;
    if (y < 0 || y >= g.H) continue;
    for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
      int x = w + pw;
      if (x < 0 || x >= g.W) continue;
      for (int c = 0; c < g.Ch; ++c) {
        float qv = qbase[c * g.HW + (long long)y * g.W + x];
        float kv = bilinear_plane(kbase + c * g.HW, g.H, g.W, y + nh, x + nw, ah, aw);
        if (g.dist == SNLS_DIST_PROD) {
          acc = fmaf(qv, kv, acc);
        } else {
          float e = qv - kv;
          acc = fmaf(e, e, acc);
        }
      }
    }
  }
  // a NaN similarity (non-finite inputs) scores as an invalid candidate
  return acc != acc ? from_score(-INFINITY, g.dist) : acc;
}

// Order this wave's earlier LDS accesses before its later ones (lanes of the
// wave read what other lanes of the same wave wrote).
SNLS_DEV void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 32-bit keys ordered like the scores they encode (unsigned comparison):
// -inf maps to 0x007fffff, so 0 lies below every score.
SNLS_DEV unsigned order_key(float f) {
  const unsigned b = __float_as_uint(f);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
SNLS_DEV float key_score(unsigned u) { return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u); }
// Number of lanes below this one whose bit is set in m.
SNLS_DEV int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}
SNLS_DEV unsigned long long shfl_xor64(unsigned long long x, int m) {
  const unsigned lo = __shfl_xor((unsigned)x, m), hi = __shfl_xor((unsigned)(x >> 32), m);
  return ((unsigned long long)hi << 32) | lo;
}

// Sorted top-k list in registers, best first, for 1 <= k <= KMAX.  The
// first KMAX - k slots hold sentinels (+inf, id -1) that rank before every
// candidate and never move, so the k kept entries are slots KMAX-k .. KMAX-1
// and the k-th best is always the last slot (a fixed register).
template <int KMAX>
struct TopList {
  float s[KMAX];
  int id[KMAX];

  SNLS_DEV void init(int k) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      const bool sentinel = i < KMAX - k;
      s[i] = sentinel ? INFINITY : -INFINITY;
      id[i] = sentinel ? -1 : 0x7fffffff;
    }
  }
  SNLS_DEV float thr_s() const { return s[KMAX - 1]; }
  SNLS_DEV int thr_id() const { return id[KMAX - 1]; }
  // Insert (sc, cid) if it ranks before the current k-th entry.
  SNLS_DEV void push(float sc, int cid) {
    if (!ranks_before(sc, cid, s[KMAX - 1], id[KMAX - 1])) return;
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      bool sw = ranks_before(sc, cid, s[i], id[i]);
      float ts = s[i];
      int ti = id[i];
      s[i] = sw ? sc : ts;
      id[i] = sw ? cid : ti;
      sc = sw ? ts : sc;
      cid = sw ? ti : cid;
    }
  }
};

#endif  // __HIPCC__

}  // namespace snls

// search_direct.hip -- direct shifted non-local search kernels (Sec. 3.2):
// each thread scores candidates straight from the video tensors with
// bilinear reads (the in-place computation of Sec. 3.4), for any parameter
// combination.  k == 0 writes every candidate; k >= 1 keeps the top-k per
// query row in registers.  These kernels are the general path; the tiled
// kernel in search_tile.hip covers the common S_Q = S_K = 1 case faster.
#include "snls_internal.h"

namespace snls {

// Decoded query row (b, hd, t, h, w) of a flattened row index over
// (B, HD, T, nH, nW).
struct QueryPos {
  int b, hd, t, h, w;
};

SNLS_DEV QueryPos decode_row(long long row, const Geo& g) {
  QueryPos qp;
  int mw = (int)(row % g.nW);
  row /= g.nW;
  int mh = (int)(row % g.nH);
  row /= g.nH;
  qp.t = (int)(row % g.T);
  row /= g.T;
  qp.hd = (int)(row % g.HD);
  qp.b = (int)(row / g.HD);
  qp.h = mh * g.s0;
  qp.w = mw * g.s0;
  return qp;
}

// Window offset F of frame step dt at the query pixel (zero for dt == 0).
SNLS_DEV void read_shift(const float* __restrict__ flows, const Geo& g, const QueryPos& qp, int dt, float* fh,
                         float* fw) {
  if (dt == 0) {
    *fh = 0.f;
    *fw = 0.f;
    return;
  }
  long long base = (((long long)qp.b * g.T + qp.t) * g.nslot + flow_slot(dt, g.wt)) * 2;
  long long pix = (long long)qp.h * g.W + qp.w;
  *fh = flows[base * g.HW + pix];
  *fw = flows[(base + 1) * g.HW + pix];
}

// One thread per (query row, candidate): every candidate in id order.
__global__ void __launch_bounds__(256) search_full_kernel(const float* __restrict__ q, const float* __restrict__ k,
                                                          const float* __restrict__ flows, Geo g,
                                                          float* __restrict__ dists, float* __restrict__ inds) {
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= g.rows * g.ncand) return;
  int cid = (int)(gid % g.ncand);
  QueryPos qp = decode_row(gid / g.ncand, g);
  int dw = cid % g.ws;
  int dh = (cid / g.ws) % g.ws;
  int dt = cid / (g.ws * g.ws) - g.wt;
  float fh, fw;
  read_shift(flows, g, qp, dt, &fh, &fw);
  float disp_h = cand_disp(fh, g.s1, dh, g.r);
  float disp_w = cand_disp(fw, g.s1, dw, g.r);
  int t2 = qp.t + dt;
  bool ok = t2 >= 0 && t2 < g.T && centre_ok(qp.h, disp_h, g.H) && centre_ok(qp.w, disp_w, g.W);
  float d = ok ? score_candidate(q, k, g, qp.b, qp.hd, qp.t, qp.h, qp.w, t2, disp_h, disp_w) : from_score(-INFINITY, g.dist);
  dists[gid] = d;
  inds[3 * gid + 0] = (float)t2;
  inds[3 * gid + 1] = disp_h;
  inds[3 * gid + 2] = disp_w;
}

// One thread per query row: all candidates, top-k kept in registers.
template <int KMAX>
__global__ void __launch_bounds__(128) search_topk_direct_kernel(const float* __restrict__ q,
                                                                 const float* __restrict__ k,
                                                                 const float* __restrict__ flows, Geo g,
                                                                 float* __restrict__ dists,
                                                                 float* __restrict__ inds) {
  long long row = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= g.rows) return;
  QueryPos qp = decode_row(row, g);
  TopList<KMAX> lst;
  lst.init(g.k);
  for (int dt = -g.wt; dt <= g.wt; ++dt) {
    int t2 = qp.t + dt;
    if (t2 < 0 || t2 >= g.T) continue;  // frame outside the clip: never selected ahead of a valid one
    float fh, fw;
    read_shift(flows, g, qp, dt, &fh, &fw);
    for (int dh = 0; dh < g.ws; ++dh) {
      float disp_h = cand_disp(fh, g.s1, dh, g.r);
      bool okh = centre_ok(qp.h, disp_h, g.H);
      for (int dw = 0; dw < g.ws; ++dw) {
        float disp_w = cand_disp(fw, g.s1, dw, g.r);
        int cid = ((dt + g.wt) * g.ws + dh) * g.ws + dw;
        float sc = -INFINITY;
        if (okh && centre_ok(qp.w, disp_w, g.W)) sc = to_score(score_candidate(q, k, g, qp.b, qp.hd, qp.t, qp.h, qp.w, t2, disp_h, disp_w), g.dist);
        lst.push(sc, cid);
      }
    }
  }
  // Rows with fewer than k valid candidates are completed with the invalid
  // candidates of smallest id (frames outside the clip included), matching
  // a full sort of all candidates.
  for (int dt = -g.wt; dt <= g.wt; ++dt) {
    int t2 = qp.t + dt;
    if (t2 >= 0 && t2 < g.T) continue;
    for (int c = 0; c < g.ws * g.ws; ++c) lst.push(-INFINITY, (dt + g.wt) * g.ws * g.ws + c);
  }
  float* drow = dists + row * g.k;
  float* irow = inds + row * g.k * 3;
  const int first = KMAX - g.k;  // slot of the best entry
#pragma unroll
  for (int e = 0; e < KMAX; ++e) {
    if (e >= first) {
      const int i = e - first;
      int cid = min(max(lst.id[e], 0), g.ncand - 1);  // every candidate was ranked: ids are real
      int dw = cid % g.ws;
      int dh = (cid / g.ws) % g.ws;
      int dt = cid / (g.ws * g.ws) - g.wt;
      float fh, fw;
      read_shift(flows, g, qp, dt, &fh, &fw);
      drow[i] = from_score(lst.s[e], g.dist);
      irow[3 * i + 0] = (float)(qp.t + dt);
      irow[3 * i + 1] = cand_disp(fh, g.s1, dh, g.r);
      irow[3 * i + 2] = cand_disp(fw, g.s1, dw, g.r);
    }
  }
}

snls_status launch_search_full(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, hipStream_t s) {
  long long total = g.rows * g.ncand;
  if (total == 0) return SNLS_OK;
  long long blocks = (total + 255) / 256;
  hipLaunchKernelGGL(search_full_kernel, dim3((unsigned)blocks), dim3(256), 0, s, q, k, flows, g, dists, inds);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_search_topk_direct(const float* q, const float* k, const float* flows, const Geo& g,
                                      float* dists, float* inds, hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  unsigned blocks = (unsigned)((g.rows + 127) / 128);
  if (g.k <= 16)
    hipLaunchKernelGGL(search_topk_direct_kernel<16>, dim3(blocks), dim3(128), 0, s, q, k, flows, g, dists, inds);
  else if (g.k <= 32)
    hipLaunchKernelGGL(search_topk_direct_kernel<32>, dim3(blocks), dim3(128), 0, s, q, k, flows, g, dists, inds);
  else if (g.k <= 64)
    hipLaunchKernelGGL(search_topk_direct_kernel<64>, dim3(blocks), dim3(128), 0, s, q, k, flows, g, dists, inds);
  else
    hipLaunchKernelGGL(search_topk_direct_kernel<128>, dim3(blocks), dim3(128), 0, s, q, k, flows, g, dists, inds);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

SearchRoute search_route(const Geo& g) {
  // single-pixel patches: no patch overlap for the tiles to share.  The fused
  // per-query kernel (k <= 32) is faster at any query stride (320 x 320,
  // S_Q = 1, Ws = 9: 2.03 vs 2.11 ms) and needs no score workspace; the
  // scored single-pixel route only at a query stride above 1.
  if (g.ps == 1 && p1_fused(g)) return SearchRoute::P1Fused;
  if (g.ps == 1 && g.s0 > 1 && p1_supported(g)) return SearchRoute::P1Scored;
  if (tile_supported(g)) return SearchRoute::Tile;
  if (p1_supported(g)) return p1_fused(g) ? SearchRoute::P1Fused : SearchRoute::P1Scored;
  return SearchRoute::Direct;
}

snls_status launch_search_topk(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, void* ws, hipStream_t s) {
  switch (search_route(g)) {
    case SearchRoute::P1Fused: return launch_search_p1_topk(q, k, flows, g, dists, inds, s);
    case SearchRoute::P1Scored: return launch_search_p1(q, k, flows, g, dists, inds, static_cast<float*>(ws), s);
    case SearchRoute::Tile: return launch_search_tile(q, k, flows, g, dists, inds, static_cast<float*>(ws), s);
    default: return launch_search_topk_direct(q, k, flows, g, dists, inds, s);
  }
}

}  // namespace snls

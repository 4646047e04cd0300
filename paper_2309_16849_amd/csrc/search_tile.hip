// search_tile.hip -- tiled shifted non-local search with fused top-k for
// the inner-product distance, query stride 1 and key stride 1 (Sec. 3.2).
//
// With S_K = 1 every window cell of a query shares the fractional part a of
// its offset F (Sec. 3.2 reads fractional positions bilinearly), so with
// N = floor(F) the score of cell d is an exact 4-tap combination
//     S(d) = sum_e w_e(a) * B_{N + d - r + e}(j),      e in {0,1}^2,
// of box sums over the patch of pixel correlations
//     B_D(j) = sum_p c_D(j + p),   c_D(x) = <q(x), K(x + D)>  (head channels,
//     query pixels outside the frame and key pixels outside the frame give 0).
// A tile of queries needs c_D only on its halo (tile + patch - 1) and only
// for the union of integer shifts D its windows cover.  Computing c_D once
// per (halo pixel, shift) instead of once per (query, patch pixel, cell) is
// what removes the redundancy of the in-place search (Sec. 3.4 notes that
// shifted windows defeat plain tiling; the union of the shifted windows is
// still shared by neighbouring queries).
//
// Work split (one workgroup = one 10 x 8 query tile of one (b, head, t),
// looping over the frames of the temporal window):
//  * 64 groups of 16 lanes; lane y of a group is halo row y (16 halo rows =
//    tile rows + P - 1), a group owns one task = (shift row D_h, block of
//    6 shift columns D_w);
//  * per channel chunk the halo of q and the union region of K are staged
//    in LDS (channel-major planes); each lane accumulates c for its halo row
//    over all halo columns x and its 6 shifts (84 accumulators);
//  * the horizontal box sum over the patch width is done in registers, the
//    vertical one across the lanes of the group (shuffles), and lane j_h
//    writes B for its tile row into the per-query window table Bw (every
//    (query, cell) entry is written by exactly one lane: deterministic);
//  * the 4-tap combination, the exact validity test and the top-k update
//    then run per query.
// A frame whose union of shifts is too wide for the LDS layout is scored
// directly instead (per candidate, canonical positions).
#include "snls_internal.h"

namespace snls {

namespace tile {

constexpr int TQW = 8;                  // tile width (queries)
constexpr int HROWS = 16;               // halo rows = lanes per group
constexpr int NGROUP = 64;              // groups per workgroup
constexpr int NTHREADS = HROWS * NGROUP;
constexpr int S = 6;                    // shift columns per task
constexpr int XMAX = 14;                // halo width limit (TQW + P - 1, P <= 7)
constexpr int CC = 8;                   // channels per staging chunk
constexpr int KR = 40;                  // K rows in LDS
constexpr int KP = 44;                  // K row pitch (floats)
constexpr int QP = 20;                  // q row pitch (floats)
constexpr int MAXBLK = 5;               // shift-column blocks: union width <= 30
constexpr int WSMAX = 9;
constexpr int WIN = (WSMAX + 1) * (WSMAX + 1);
constexpr int QMAX = HROWS * TQW;       // queries per tile (P = 1)
constexpr int KLIST = 16;               // top-k capacity

constexpr int KST_F = CC * KR * KP;     // 14080 floats
constexpr int QST_F = CC * HROWS * QP;  // 2560
constexpr int BW_F = QMAX * WIN;        // 12800
constexpr int LIST_W = QMAX * KLIST;    // scores + ids, 2048 each

struct Smem {
  float kst[KST_F];  // K union region chunk; reused as the candidate score table
  float qst[QST_F];  // q halo chunk
  float bw[BW_F];    // per-query window of box sums, (WSMAX+1)^2 cells
  float lst_s[LIST_W];
  int lst_id[LIST_W];
  int qn_h[QMAX], qn_w[QMAX];  // integer part of the offset
  float qf_h[QMAX], qf_w[QMAX];  // the offset itself
  int uni[4];  // min N_h, max N_h, min N_w, max N_w
};

}  // namespace tile

// Value of lane (i + N) of the same 16-lane row (DPP row_shl:N); lanes whose
// source lies past the end of the row read 0.
template <int N>
SNLS_DEV float row_shl(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + N, 0xf, 0xf, true));
}

// Sum of lanes i .. i+P-1 of the 16-lane row (a box sum down the halo rows).
template <int P>
struct RowBox {
  static SNLS_DEV float sum(float v) { return RowBox<P - 1>::sum(v) + row_shl<P - 1>(v); }
};
template <>
struct RowBox<1> {
  static SNLS_DEV float sum(float v) { return v; }
};

template <int PS>
__global__ void __launch_bounds__(tile::NTHREADS) search_tile_kernel(const float* __restrict__ q,
                                                                      const float* __restrict__ k,
                                                                      const float* __restrict__ flows, Geo g,
                                                                      int tiles_x, int tiles_y,
                                                                      float* __restrict__ dists,
                                                                      float* __restrict__ inds) {
  using namespace tile;
  constexpr int TQH = HROWS - PS + 1;
  constexpr int HW = TQW + PS - 1;
  constexpr int LO = -(PS / 2);
  __shared__ Smem sm;

  const int tid = threadIdx.x;
  const int lane16 = tid & 15;
  const int grp = tid >> 4;

  // XCD-aware order: consecutive workgroups land on different XCDs, so give
  // each XCD a contiguous run of tiles (neighbouring tiles share K in L2).
  const long long nwg = (long long)gridDim.x;
  const long long xcd = blockIdx.x % 8, xq = nwg / 8, xrem = nwg % 8;
  const long long wg = xcd * xq + (xcd < xrem ? xcd : xrem) + blockIdx.x / 8;
  const long long tiles_img = (long long)tiles_x * tiles_y;
  const int img = (int)(wg / tiles_img);
  const int trem = (int)(wg % tiles_img);
  const int ty = trem / tiles_x, tx = trem % tiles_x;
  const int t = img % g.T;
  const int hd = (img / g.T) % g.HD;
  const int b = img / (g.T * g.HD);
  const int y0 = ty * TQH, x0 = tx * TQW;  // tile origin (query = pixel, stride 1)
  const int Y0 = y0 + LO, X0 = x0 + LO;    // halo origin
  const int ws = g.ws, r = g.r;
  const int nq_tile = TQH * TQW;

  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;

  for (int i = tid; i < nq_tile * KLIST; i += NTHREADS) {
    sm.lst_s[i] = -INFINITY;
    sm.lst_id[i] = 0x7fffffff;
  }

  for (int dt = -g.wt; dt <= g.wt; ++dt) {
    const int t2 = t + dt;
    if (t2 < 0 || t2 >= g.T) continue;
    const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;

    // ---- offsets of the tile's queries and the union of shifts ----
    if (tid < 4) sm.uni[tid] = (tid & 1) ? INT_MIN : INT_MAX;
    __syncthreads();
    if (tid < nq_tile) {
      const int jh = tid / TQW, jw = tid % TQW;
      const int h = y0 + jh, w = x0 + jw;
      float fh = 0.f, fw = 0.f;
      int nh = 0, nw = 0;
      const bool inside = h < g.H && w < g.W;
      if (dt != 0 && inside) {
        long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
        long long pix = (long long)h * g.W + w;
        fh = flows[base * g.HW + pix];
        fw = flows[(base + 1) * g.HW + pix];
      }
      // Offsets that are not finite or absurdly large leave the union alone;
      // their candidates fail the exact validity test below.
      if (fabsf(fh) < 1.0e6f) nh = (int)floorf(fh);
      if (fabsf(fw) < 1.0e6f) nw = (int)floorf(fw);
      sm.qn_h[tid] = nh;
      sm.qn_w[tid] = nw;
      sm.qf_h[tid] = fh;
      sm.qf_w[tid] = fw;
      if (inside) {
        atomicMin(&sm.uni[0], nh);
        atomicMax(&sm.uni[1], nh);
        atomicMin(&sm.uni[2], nw);
        atomicMax(&sm.uni[3], nw);
      }
    }
    __syncthreads();
    const int dmin_h = sm.uni[0] - r, UH = sm.uni[1] - sm.uni[0] + ws + 1;
    const int dmin_w = sm.uni[2] - r, UW = sm.uni[3] - sm.uni[2] + ws + 1;
    const int nblk = (UW + S - 1) / S;
    float* const dbuf = sm.kst;  // candidate scores of this frame (after staging)

    if (nblk <= MAXBLK) {
      const int ntask = UH * nblk;
      const int span_max = KR - HROWS + 1;                 // shift rows per round
      const int tasks_per_round = min(NGROUP, span_max * nblk);
      for (int r0 = 0; r0 < ntask; r0 += tasks_per_round) {
        const int r1 = min(ntask, r0 + tasks_per_round);
        const int dh_lo = dmin_h + r0 / nblk;
        const int dh_hi = dmin_h + (r1 - 1) / nblk;
        const int krows = HROWS + dh_hi - dh_lo;
        const int kcols = HW + nblk * S - 1;
        const int task = r0 + grp;
        const bool active = task < r1;
        const int d_h = dmin_h + task / nblk;
        const int blk = task % nblk;
        const int krow = lane16 + d_h - dh_lo;

        float acc[HW][S];
#pragma unroll
        for (int x = 0; x < HW; ++x)
#pragma unroll
          for (int i = 0; i < S; ++i) acc[x][i] = 0.f;

        for (int c0 = 0; c0 < g.Ch; c0 += CC) {
          __syncthreads();  // previous chunk consumed
          // stage q halo: HROWS x HW per channel
          for (int e = tid; e < CC * HROWS * HW; e += NTHREADS) {
            const int c = e / (HROWS * HW);
            const int rem = e % (HROWS * HW);
            const int yy = rem / HW, xx = rem % HW;
            const int gy = Y0 + yy, gx = X0 + xx;
            float v = 0.f;
            if (c0 + c < g.Ch && gy >= 0 && gy < g.H && gx >= 0 && gx < g.W)
              v = qb[(long long)(c0 + c) * g.HW + (long long)gy * g.W + gx];
            sm.qst[(c * HROWS + yy) * QP + xx] = v;
          }
          // stage K union region: krows x kcols per channel
          for (int e = tid; e < CC * krows * kcols; e += NTHREADS) {
            const int c = e / (krows * kcols);
            const int rem = e % (krows * kcols);
            const int yy = rem / kcols, xx = rem % kcols;
            const int gy = Y0 + dh_lo + yy, gx = X0 + dmin_w + xx;
            float v = 0.f;
            if (c0 + c < g.Ch && gy >= 0 && gy < g.H && gx >= 0 && gx < g.W)
              v = kb[(long long)(c0 + c) * g.HW + (long long)gy * g.W + gx];
            sm.kst[(c * KR + yy) * KP + xx] = v;
          }
          __syncthreads();
          if (active) {
#pragma unroll 1
            for (int c = 0; c < CC; ++c) {
              const float* qr = &sm.qst[(c * HROWS + lane16) * QP];
              const float* kr = &sm.kst[(c * KR + krow) * KP + blk * S];
              // sliding window kw[i] = K(x + i) along the halo row
              float kw[S];
#pragma unroll
              for (int i = 0; i < S - 1; ++i) kw[i] = kr[i];
#pragma unroll
              for (int x = 0; x < HW; ++x) {
                kw[S - 1] = kr[x + S - 1];
                const float qx = qr[x];
#pragma unroll
                for (int i = 0; i < S; ++i) acc[x][i] = fmaf(qx, kw[i], acc[x][i]);
#pragma unroll
                for (int i = 0; i < S - 1; ++i) kw[i] = kw[i + 1];
              }
            }
          }
        }

        // horizontal box over the patch width, in place (registers)
#pragma unroll
        for (int jw = 0; jw < TQW; ++jw)
#pragma unroll
          for (int i = 0; i < S; ++i) {
#pragma unroll
            for (int pw = 1; pw < PS; ++pw) acc[jw][i] += acc[jw + pw][i];
          }
        // vertical box over the patch height, across the 16 lanes of the group
#pragma unroll
        for (int jw = 0; jw < TQW; ++jw)
#pragma unroll
          for (int i = 0; i < S; ++i) {
            float s = RowBox<PS>::sum(acc[jw][i]);
            asm volatile("" : "+v"(s));  // materialise the sum here: keeps the row moves short-lived
            acc[jw][i] = s;
          }
        if (active && lane16 < TQH) {
          const int jh = lane16;
#pragma unroll
          for (int jw = 0; jw < TQW; ++jw) {
            const int j = jh * TQW + jw;
            const int u = d_h - (sm.qn_h[j] - r);
            const int vbase = dmin_w + blk * S - (sm.qn_w[j] - r);
            if (u >= 0 && u <= ws) {
#pragma unroll
              for (int i = 0; i < S; ++i) {
                const int v = vbase + i;
                if (v >= 0 && v <= ws) sm.bw[j * WIN + u * (WSMAX + 1) + v] = acc[jw][i];
              }
            }
          }
        }
      }
      __syncthreads();
      // ---- 4-tap combination + exact validity -> candidate scores ----
      for (int e = tid; e < nq_tile * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int h = y0 + j / TQW, w = x0 + j % TQW;
        const float fh = sm.qf_h[j], fw = sm.qf_w[j];
        const float ah = fh - (float)sm.qn_h[j];
        const float aw = fw - (float)sm.qn_w[j];
        const float* r0p = &sm.bw[j * WIN + dh * (WSMAX + 1)];
        const float* r1p = r0p + (WSMAX + 1);
        const float disp_h = cand_disp(fh, 1.f, dh, r);
        const bool okh = centre_ok(h, disp_h, g.H);
        for (int dw = 0; dw < ws; ++dw) {
          const float top = (1.f - aw) * r0p[dw] + aw * r0p[dw + 1];
          const float bot = (1.f - aw) * r1p[dw] + aw * r1p[dw + 1];
          const float d = (1.f - ah) * top + ah * bot;
          const bool ok = okh && centre_ok(w, cand_disp(fw, 1.f, dw, r), g.W);
          dbuf[j * WIN + dh * ws + dw] = ok ? d : -INFINITY;
        }
      }
    } else {
      // Union too wide for the LDS layout: score this frame directly.
      __syncthreads();
      for (int e = tid; e < nq_tile * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int h = y0 + j / TQW, w = x0 + j % TQW;
        if (h >= g.H || w >= g.W) continue;
        const float fh = sm.qf_h[j], fw = sm.qf_w[j];
        const float disp_h = cand_disp(fh, 1.f, dh, r);
        const bool okh = centre_ok(h, disp_h, g.H);
        for (int dw = 0; dw < ws; ++dw) {
          const float disp_w = cand_disp(fw, 1.f, dw, r);
          float d = -INFINITY;
          if (okh && centre_ok(w, disp_w, g.W)) d = score_candidate(q, k, g, b, hd, t, h, w, t2, disp_h, disp_w);
          dbuf[j * WIN + dh * ws + dw] = d;
        }
      }
    }
    __syncthreads();
    // ---- top-k update, one thread per query ----
    if (tid < nq_tile) {
      const int j = tid;
      TopList<KLIST> lst;
#pragma unroll
      for (int i = 0; i < KLIST; ++i) {
        lst.s[i] = sm.lst_s[j * KLIST + i];
        lst.id[i] = sm.lst_id[j * KLIST + i];
      }
      lst.thr_s = -INFINITY;
      lst.thr_id = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < KLIST; ++i)
        if (i == g.k - 1) {
          lst.thr_s = lst.s[i];
          lst.thr_id = lst.id[i];
        }
      const int idb = (dt + g.wt) * ws * ws;
      for (int c = 0; c < ws * ws; ++c) lst.push(dbuf[j * WIN + c], idb + c, g.k);
#pragma unroll
      for (int i = 0; i < KLIST; ++i) {
        sm.lst_s[j * KLIST + i] = lst.s[i];
        sm.lst_id[j * KLIST + i] = lst.id[i];
      }
    }
    __syncthreads();
  }

  // ---- output: complete short lists with the frames outside the clip ----
  if (tid < nq_tile) {
    const int j = tid;
    const int h = y0 + j / TQW, w = x0 + j % TQW;
    if (h < g.H && w < g.W) {
      TopList<KLIST> lst;
#pragma unroll
      for (int i = 0; i < KLIST; ++i) {
        lst.s[i] = sm.lst_s[j * KLIST + i];
        lst.id[i] = sm.lst_id[j * KLIST + i];
      }
      lst.thr_s = -INFINITY;
      lst.thr_id = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < KLIST; ++i)
        if (i == g.k - 1) {
          lst.thr_s = lst.s[i];
          lst.thr_id = lst.id[i];
        }
      if (lst.thr_s == -INFINITY) {
        for (int dt = -g.wt; dt <= g.wt; ++dt) {
          if (t + dt >= 0 && t + dt < g.T) continue;
          for (int c = 0; c < ws * ws; ++c) lst.push(-INFINITY, (dt + g.wt) * ws * ws + c, g.k);
        }
      }
      const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + h) * g.nW + w;
      float* drow = dists + row * g.k;
      float* irow = inds + row * g.k * 3;
      const long long pix = (long long)h * g.W + w;
#pragma unroll
      for (int i = 0; i < KLIST; ++i) {
        if (i < g.k) {
          const int cid = lst.id[i];
          const int dw = cid % ws, dh = (cid / ws) % ws, dt = cid / (ws * ws) - g.wt;
          float fh = 0.f, fw = 0.f;
          if (dt != 0) {
            long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
            fh = flows[base * g.HW + pix];
            fw = flows[(base + 1) * g.HW + pix];
          }
          drow[i] = lst.s[i];
          irow[3 * i + 0] = (float)(t + dt);
          irow[3 * i + 1] = cand_disp(fh, 1.f, dh, r);
          irow[3 * i + 2] = cand_disp(fw, 1.f, dw, r);
        }
      }
    }
  }
}

// The tiled kernel handles: inner product, S_Q = S_K = 1, P <= 7, Ws <= 9, k <= 16.
bool tile_supported(const Geo& g) {
  return g.dist == SNLS_DIST_PROD && g.s0 == 1 && g.s1 == 1.0f && g.ps <= 7 && g.ws <= tile::WSMAX &&
         g.k >= 1 && g.k <= tile::KLIST;
}

snls_status launch_search_tile(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, hipStream_t s) {
  const int tqh = tile::HROWS - g.ps + 1;
  const int tiles_x = (g.W + tile::TQW - 1) / tile::TQW;
  const int tiles_y = (g.H + tqh - 1) / tqh;
  const long long nwg = (long long)tiles_x * tiles_y * g.B * g.HD * g.T;
  if (nwg == 0) return SNLS_OK;
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  dim3 grid((unsigned)nwg), block(tile::NTHREADS);
  switch (g.ps) {
#define SNLS_TILE_CASE(P)                                                                                  \
  case P:                                                                                                  \
    hipLaunchKernelGGL(search_tile_kernel<P>, grid, block, 0, s, q, k, flows, g, tiles_x, tiles_y, dists, \
                       inds);                                                                              \
    break;
    SNLS_TILE_CASE(1)
    SNLS_TILE_CASE(2)
    SNLS_TILE_CASE(3)
    SNLS_TILE_CASE(4)
    SNLS_TILE_CASE(5)
    SNLS_TILE_CASE(6)
    SNLS_TILE_CASE(7)
#undef SNLS_TILE_CASE
    default:
      return SNLS_ERR_UNSUPPORTED;
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

// search_tile.hip -- tiled shifted non-local search: scores of every
// candidate for the inner product (key stride S_K <= 1, any query stride),
// then the top-k of the scored rows (Sec. 3.2).
//
// Window cell d of a query sits at displacement disp_d = F + S_K (d - r);
// with n_d = floor(disp_d) and a_d = disp_d - n_d its bilinear score is an
// exact 4-tap combination
//     S(d) = sum_e w_e(a_d) * B_{n_d + e}(j),      e in {0,1}^2,
// of box sums over the patch of pixel correlations
//     B_D(j) = sum_p c_D(j + p),   c_D(x) = <q(x), K(x + D)>  (head channels,
//     query pixels outside the frame and key pixels outside the frame give 0).
// All integer shifts D of a query lie in [floor(disp_0), floor(disp_last)+1]
// (at most Ws + 1 per axis for S_K <= 1; for S_K = 1/2 about half that), so
// a tile of queries needs c_D only on its halo (tile + patch - 1) and only
// for the union of those shift ranges.  Computing c_D once per (halo pixel,
// shift) instead of once per (query, patch pixel, cell) is what removes the
// redundancy of the in-place search (Sec. 3.4 notes that shifted windows
// defeat plain tiling; the union of the shifted windows is still shared by
// neighbouring queries).
//
// Work split (one workgroup = one query tile of one (b, head, t), looping
// over the frames of the temporal window; at query stride 1 and P = 7 the
// tile is 10 x 8 queries, at stride S_Q the queries whose patches fit the
// same 16-row halo, e.g. 5 x 4 at S_Q = 2):
//  * 64 groups of 16 lanes; lane y of a group is halo row y (16 halo rows =
//    tile rows + P - 1), a group owns one task = (shift row D_h, block of
//    6 shift columns D_w) or one channel part of a task (tasks that would
//    leave groups idle have their channels split, the parts summed before
//    the tables are written);
//  * per channel chunk the halo of q and the union region of K are staged
//    in LDS (channel-major planes); each lane accumulates c for its halo row
//    over all halo columns x and its 6 shifts (84 accumulators);
//  * the horizontal box sum over the patch width is done in registers, the
//    vertical one across the lanes of the group (shuffles), and lane j_h
//    writes B for its tile row into the per-query window table Bw (every
//    (query, cell) entry is written by exactly one lane: deterministic);
//  * the 4-tap combination (positions and weights from disp_d exactly as
//    the output reports them) and the exact validity test give the score of
//    every window cell, which is written to the caller's workspace
//    (rows x candidates, candidate id order).
// A frame whose union of shifts is too wide for the LDS layout is scored
// directly instead (per candidate, canonical positions).
//
// A second kernel then streams each query row's scores once and keeps its
// top k (Sec. 3.2 top-L over the whole space-time window), so the
// correlation kernel carries no per-query selection state.
#include "snls_internal.h"

namespace snls {

namespace tile {

constexpr int TQW = 8;                  // tile width (queries)
constexpr int HROWS = 16;               // halo rows = lanes per group
constexpr int NGROUP = 64;              // groups per workgroup
constexpr int NTHREADS = HROWS * NGROUP;
constexpr int S = 6;                    // shift columns per task
constexpr int CC = 4;                   // channels per staging chunk (double-buffered)
constexpr int KR = 36;                  // K rows in LDS
constexpr int KP = 45;                  // K row pitch (odd: spreads the 16 rows of a group over the banks)
constexpr int QP = 21;                  // q row pitch (odd)
constexpr int NIT = 2;                  // staging items (4 columns of one row) per thread and chunk
constexpr int MAXBLK = 5;               // shift-column blocks: union width <= 30
constexpr int WSMAX = 9;                // window side of the common instances
constexpr int WSBIG = 15;               // ... and of the P = 7 instance for larger windows
// window-table pitch for windows up to WSM (shifts floor(disp_0) ..
// floor(disp_last) + 1) and the table of one query
constexpr int wpitch(int WSM) { return WSM + 2; }
constexpr int wtable(int WSM) { return wpitch(WSM) * wpitch(WSM); }

// Staging buffers (double-buffered chunks of CC channels).
constexpr int KST_F = (CC * KR * KP + 63) / 64 * 64;     // 6528 floats
constexpr int QST_F = (CC * HROWS * QP + 63) / 64 * 64;  // 1344


template <int PS, int WSM>
struct Smem {
  static constexpr int QN = (HROWS - PS + 1) * TQW;  // queries per tile
  float kst[2][KST_F];  // K union region chunks (double buffer)
  float qst[2][QST_F];  // q halo chunks
  float bw[QN * wtable(WSM)];  // per-query window of box sums
  int qlo_h[QN], qlo_w[QN];  // smallest integer shift of the query's window (table origin)
  float qf_h[QN], qf_w[QN];  // the offset itself
  int uni[4];                // min N_h, max N_h, min N_w, max N_w
};

}  // namespace tile

// Window cell offsets (d_h - r, d_w - r) of a 9 x 9 window by distance from
// the centre (then row, then column): the first k inside the window seed the
// threshold of the query frame.
__constant__ signed char kSpiral[81][2] = {
    {0, 0}, {-1, 0}, {0, -1}, {0, 1}, {1, 0}, {-1, -1}, {-1, 1}, {1, -1}, {1, 1},
    {-2, 0}, {0, -2}, {0, 2}, {2, 0}, {-2, -1}, {-2, 1}, {-1, -2}, {-1, 2}, {1, -2},
    {1, 2}, {2, -1}, {2, 1}, {-2, -2}, {-2, 2}, {2, -2}, {2, 2}, {-3, 0}, {0, -3},
    {0, 3}, {3, 0}, {-3, -1}, {-3, 1}, {-1, -3}, {-1, 3}, {1, -3}, {1, 3}, {3, -1},
    {3, 1}, {-3, -2}, {-3, 2}, {-2, -3}, {-2, 3}, {2, -3}, {2, 3}, {3, -2}, {3, 2},
    {-4, 0}, {0, -4}, {0, 4}, {4, 0}, {-4, -1}, {-4, 1}, {-1, -4}, {-1, 4}, {1, -4},
    {1, 4}, {4, -1}, {4, 1}, {-3, -3}, {-3, 3}, {3, -3}, {3, 3}, {-4, -2}, {-4, 2},
    {-2, -4}, {-2, 4}, {2, -4}, {2, 4}, {4, -2}, {4, 2}, {-4, -3}, {-4, 3}, {-3, -4},
    {-3, 4}, {3, -4}, {3, 4}, {4, -3}, {4, 3}, {-4, -4}, {-4, 4}, {4, -4}, {4, 4},
};

// Value of lane (i + N) of the same 16-lane row (DPP row_shl:N); lanes whose
// source lies past the end of the row read 0.
template <int N>
SNLS_DEV float row_shl(float v) {
  if constexpr (N == 0) return v;
  else return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + N, 0xf, 0xf, true));
}

// Box sums of width P <= 7 as a sum of power-of-two boxes (P = 4a + 2b + c):
// b2(i) = v(i) + v(i+1), b4(i) = b2(i) + b2(i+2), box(i) = b4(i) + b2(i+4a)
// + v(i+4a+2b) for the terms present.  At most 4 additions instead of P-1.
template <int P>
struct Pow2Box {
  static_assert(P >= 1 && P <= 7, "box width");
  static constexpr int O2 = (P & 4) ? 4 : 0;          // offset of the width-2 term
  static constexpr int O1 = O2 + ((P & 2) ? 2 : 0);   // offset of the width-1 term
};

// Sum of lanes i .. i+P-1 of the 16-lane row (a box sum down the halo rows).
template <int P>
SNLS_DEV float row_box(float v) {
  using B = Pow2Box<P>;
  if constexpr (P == 1) {
    return v;
  } else {
    const float b2 = v + row_shl<1>(v);
    float r;
    if constexpr ((P & 4) != 0) {
      r = b2 + row_shl<2>(b2);
      if constexpr ((P & 2) != 0) r += row_shl<B::O2>(b2);
    } else {
      r = b2;
    }
    if constexpr ((P & 1) != 0) r += row_shl<B::O1>(v);
    return r;
  }
}

// In-place horizontal box sums of one shift column: a[x] becomes
// a[x] + ... + a[x+P-1] for x < N (the array holds N + P - 1 values).
template <int P, int N, int L, int S, int I>
SNLS_DEV void row_box_regs(float (&a)[L][S]) {
  static_assert(L == N + P - 1, "array length");
  using B = Pow2Box<P>;
  if constexpr (P > 1) {
    float b2[L - 1];
#pragma unroll
    for (int x = 0; x < L - 1; ++x) b2[x] = a[x][I] + a[x + 1][I];
    float b4[(P & 4) ? L - 3 : 1];
    if constexpr ((P & 4) != 0) {
#pragma unroll
      for (int x = 0; x < L - 3; ++x) b4[x] = b2[x] + b2[x + 2];
    }
#pragma unroll
    for (int x = 0; x < N; ++x) {  // ascending x: a[x + O1] (O1 >= 1) is not yet overwritten
      float r;
      if constexpr ((P & 4) != 0) {
        r = b4[x];
        if constexpr ((P & 2) != 0) r += b2[x + B::O2];
      } else {
        r = b2[x];
      }
      if constexpr ((P & 1) != 0) r += a[x + B::O1][I];
      a[x][I] = r;
    }
  }
}

template <int P, int N, int L, int S, int I = 0>
SNLS_DEV void box_cols(float (&a)[L][S]) {
  if constexpr (I < S) {
    row_box_regs<P, N, L, S, I>(a);
    box_cols<P, N, L, S, I + 1>(a);
  }
}

// WSM: the largest window side of the instance (the window tables' size).
template <int PS, int WSM>
__global__ void __launch_bounds__(tile::NTHREADS) search_tile_scores_kernel(const float* __restrict__ q,
                                                                             const float* __restrict__ k,
                                                                             const float* __restrict__ flows, Geo g,
                                                                             int tiles_x, int tiles_y,
                                                                             float* __restrict__ scores, int pitch) {
  using namespace tile;
  constexpr int HW = TQW + PS - 1;
  constexpr int LO = -(PS / 2);
  constexpr int QC4 = (HW + 3) / 4;  // 4-column items per q row
  constexpr int NQIT = CC * HROWS * QC4;  // q items per chunk (a multiple of 64)
  static_assert(NQIT % 64 == 0 && NQIT <= NTHREADS, "q items fill whole waves of item slot 1");
  static_assert(CC * KR * ((KP + 3) / 4) <= 2 * NTHREADS - NQIT, "every K item has a slot");
  constexpr int QN = Smem<PS, WSM>::QN;
  constexpr int WP = wpitch(WSM), WIN = wtable(WSM);
  static_assert(sizeof(Smem<PS, WSM>) <= 160 * 1024, "the LDS of one CU");
  __shared__ Smem<PS, WSM> sm;

  const int tid = threadIdx.x;
  const int lane16 = tid & 15;
  const int grp = tid >> 4;

  // XCD-aware order: consecutive workgroups land on different XCDs, so give
  // each XCD a contiguous run of tiles (neighbouring tiles share K in L2).
  const long long nwg = (long long)gridDim.x;
  const long long xcd = blockIdx.x % 8, xq = nwg / 8, xrem = nwg % 8;
  const long long wg = xcd * xq + (xcd < xrem ? xcd : xrem) + blockIdx.x / 8;
  // The query frames (and heads, batch entries) of one tile are consecutive
  // workgroups, so the key frames they share stay in the XCD's L2.
  const int nimg = g.B * g.HD * g.T;
  const int img = (int)(wg % nimg);
  const int trem = (int)(wg / nimg);
  const int ty = trem / tiles_x, tx = trem % tiles_x;
  const int t = img % g.T;
  const int hd = (img / g.T) % g.HD;
  const int b = img / (g.T * g.HD);
  // Query stride S_Q: the tile is tqh x tqw queries (query-grid units) whose
  // patches fit the HROWS x HW halo; at S_Q = 1 that is TQH x TQW.
  const int s0 = g.s0;
  const int tqh = (HROWS - PS) / s0 + 1, tqw = (TQW - 1) / s0 + 1, qn = tqh * tqw;
  const int my0 = ty * tqh, mx0 = tx * tqw;  // tile origin (query grid)
  const int y0 = my0 * s0, x0 = mx0 * s0;    // tile origin (pixels)
  const int Y0 = y0 + LO, X0 = x0 + LO;      // halo origin
  // halo row of this lane as the patch origin of a query row (-1: none), and
  // the halo columns that are query patch origins
  const int jh_lane = (lane16 % s0 == 0 && lane16 / s0 < tqh) ? lane16 / s0 : -1;
  unsigned xmask = 0;
  for (int xq = 0; xq < TQW; xq += s0) xmask |= 1u << xq;
  const int ws = g.ws, r = g.r;

  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;

  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  constexpr unsigned OOB = 0x80000000u;  // buffer offset past any extent: reads 0
  const int HWi = (int)g.HW;
  const __amdgpu_buffer_rsrc_t q_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)qb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);

  // window offset of this thread's query (tid < qn) for frame step dt
  auto fetch_flow = [&](int dtt, float& fh, float& fw) {
    fh = 0.f;
    fw = 0.f;
    const int h = y0 + s0 * (tid / tqw), w = x0 + s0 * (tid % tqw);
    if (dtt != 0 && tid < qn && h < g.H && w < g.W) {
      const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dtt, g.wt)) * 2;
      const long long pix = (long long)h * g.W + w;
      fh = flows[base * g.HW + pix];
      fw = flows[(base + 1) * g.HW + pix];
    }
  };
  float fh_next = 0.f, fw_next = 0.f;
  bool first = true;

  auto frame_dt = [&](int s) { return s - g.wt; };
  for (int si = 0; si <= 2 * g.wt; ++si) {
    const int dt = frame_dt(si);
    const long long rowb = (((long long)b * g.HD + hd) * g.T + t) * g.nH;
    const int cbase = (dt + g.wt) * ws * ws;
    const int t2 = t + dt;
    if (t2 < 0 || t2 >= g.T) continue;
    const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
    const __amdgpu_buffer_rsrc_t k_rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)kb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);

    // ---- offsets of the tile's queries and the union of shifts ----
    // (thread-index arithmetic is redone per frame rather than kept live
    // across the frame's channel loops)
    int tidf = tid;
    asm volatile("" : "+v"(tidf));
    if (tidf < 4) sm.uni[tidf] = (tidf & 1) ? INT_MIN : INT_MAX;
    if (first) {
      fetch_flow(dt, fh_next, fw_next);
      first = false;
    }
    __syncthreads();
    {
      const int jh = tidf / tqw, jw = tidf % tqw;
      const bool inside = tidf < qn && y0 + s0 * jh < g.H && x0 + s0 * jw < g.W;
      const float fh = fh_next, fw = fw_next;
      // Integer shifts a query's window reads: floor(disp) .. floor(disp) + 1
      // for its first .. last cell (disp grows with the cell index).
      // Offsets that are not finite or absurdly large count as zero here;
      // their candidates fail the exact validity test below.
      const float fh_u = fabsf(fh) < kFarDisp ? fh : 0.f, fw_u = fabsf(fw) < kFarDisp ? fw : 0.f;
      const int lo_h = (int)floorf(cand_disp(fh_u, g.s1, 0, r));
      const int hi_h = (int)floorf(cand_disp(fh_u, g.s1, ws - 1, r)) + 1;
      const int lo_w = (int)floorf(cand_disp(fw_u, g.s1, 0, r));
      const int hi_w = (int)floorf(cand_disp(fw_u, g.s1, ws - 1, r)) + 1;
      if (tidf < qn) {
        sm.qlo_h[tidf] = lo_h;
        sm.qlo_w[tidf] = lo_w;
        sm.qf_h[tidf] = fh;
        sm.qf_w[tidf] = fw;
      }
      // union bounds: wave reductions, then one LDS atomic per wave
      if (tidf < ((QN + 63) & ~63)) {
        int a0 = inside ? lo_h : INT_MAX, a1 = inside ? hi_h : INT_MIN;
        int a2 = inside ? lo_w : INT_MAX, a3 = inside ? hi_w : INT_MIN;
        const int ln = tidf & 63;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const int src = (ln ^ off) << 2;
          a0 = min(a0, __builtin_amdgcn_ds_bpermute(src, a0));
          a1 = max(a1, __builtin_amdgcn_ds_bpermute(src, a1));
          a2 = min(a2, __builtin_amdgcn_ds_bpermute(src, a2));
          a3 = max(a3, __builtin_amdgcn_ds_bpermute(src, a3));
        }
        if (ln == 0) {
          atomicMin(&sm.uni[0], a0);
          atomicMax(&sm.uni[1], a1);
          atomicMin(&sm.uni[2], a2);
          atomicMax(&sm.uni[3], a3);
        }
      }
    }
    // next searched frame's offsets, in flight during this frame
    {
      int sn = si + 1;
      while (sn <= 2 * g.wt && (t + frame_dt(sn) < 0 || t + frame_dt(sn) >= g.T)) ++sn;
      if (sn <= 2 * g.wt) fetch_flow(frame_dt(sn), fh_next, fw_next);
    }
    __syncthreads();
    // (uniform values: kept in scalar registers)
    // Only shifts that a valid cell can read matter: a valid cell of a query
    // at row h has h + disp in [0, H-1], so its taps lie in rows
    // [-h, H - h]; over the tile's queries that is [-h_last, H - y0] (and
    // likewise for columns).  Clipping the union to that range bounds the
    // rounds of a tile whose offsets are spread far outside the frame.
    const int h_last = min(y0 + (tqh - 1) * s0, (g.nH - 1) * s0);
    const int w_last = min(x0 + (tqw - 1) * s0, (g.nW - 1) * s0);
    const int u0 = max(__builtin_amdgcn_readfirstlane(sm.uni[0]), -h_last);
    const int u1 = min(__builtin_amdgcn_readfirstlane(sm.uni[1]), g.H - y0);
    const int u2 = max(__builtin_amdgcn_readfirstlane(sm.uni[2]), -w_last);
    const int u3 = min(__builtin_amdgcn_readfirstlane(sm.uni[3]), g.W - x0);
    const int dmin_h = u0, UH = u1 - u0 + 1;
    const int dmin_w = u2, UW = u3 - u2 + 1;
    // no shift left: every cell of the frame is invalid (the 4-tap pass below
    // scores them so without reading the tables)
    const bool none = UH <= 0 || UW <= 0;
    const int nblk = none ? 0 : (UW + S - 1) / S;

    if (nblk <= MAXBLK) {
      // A task is (shift row, column block); a round covers as many shift
      // rows as the groups and the K rows of the LDS layout allow.  Whole
      // quads of rows go to whole waves -- a wave's 4 groups take 4
      // consecutive shift rows of one block, so their K reads hit
      // overlapping rows (broadcast) in distinct banks.  The rows past the
      // last whole quad (tail) go to single groups packed after them.  The
      // channels of a task are split into csplit parts (each part a group of
      // its own) as far as the 64 groups allow: the full quads first, then
      // the tail, which would otherwise keep whole waves busy for one row.
      const int span_max = KR - HROWS + 1;
      const int rows_per_round = none ? 1 : min(span_max, NGROUP / nblk);
      for (int rr0 = 0; rr0 < (none ? 0 : UH); rr0 += rows_per_round) {
        const int nrows = min(rows_per_round, UH - rr0);
        const int uf = nblk * (nrows >> 2);  // whole quads: waves per channel part
        const int tt = nblk * (nrows & 3);   // tail tasks
        const int csf = 16 * uf + tt <= NGROUP ? 4 : (8 * uf + tt <= NGROUP ? 2 : 1);
        const int gf = 4 * uf * csf;         // groups of the whole quads (a whole number of waves)
        const int cst = gf + 4 * tt <= NGROUP ? 4 : (gf + 2 * tt <= NGROUP ? 2 : 1);

        int part, blk, d_row;
        bool active;
        if (wave < gf / 4) {
          part = wave / uf;
          const int unit = wave - part * uf;
          blk = unit % nblk;
          d_row = (unit / nblk) * 4 + (grp & 3);
          active = true;
        } else {
          // tail: the cst parts of a task are consecutive groups of one wave
          // (lanes 16 or 32 apart), summed across the lanes before the
          // window tables are written
          const int e = grp - gf, rt = nrows & 3;
          const int task = e / cst;
          part = e - task * cst;
          blk = rt > 0 ? task / rt : nblk;
          d_row = (nrows & ~3) + (rt > 0 ? task - (task / rt) * rt : 0);
          active = rt > 0 && blk < nblk;
        }
        // channel parts are whole waves: gf is a multiple of 4 groups
        const int csplit = __builtin_amdgcn_readfirstlane(wave < gf / 4 ? csf : cst);
        const int dh_lo = dmin_h + rr0;
        const int krows = HROWS + nrows - 1;
        const int kcols = HW + nblk * S - 1;
        const int d_h = dh_lo + d_row;
        const int krow = lane16 + d_row;

        float acc[HW][S];
#pragma unroll
        for (int x = 0; x < HW; ++x)
#pragma unroll
          for (int i = 0; i < S; ++i) acc[x][i] = 0.f;

        // Staging through registers: a chunk (CC channels) of the round's K
        // region and of the q halo is cut into items of 4 consecutive
        // columns of one row; each thread owns up to NIT items, loads them
        // with one 16-byte buffer load each (the start column is clamped into
        // the frame, so no access leaves the row; values are realigned and
        // columns outside the frame zeroed in registers) and writes them to
        // LDS.  Rows outside the frame and channels past the head read 0
        // through an out-of-range offset.  Offsets stay below 2^31: the tiled
        // kernel requires Ch*H*W*4 < 2^31.
        const int ncol4 = (kcols + 3) >> 2;
        const int nkit = CC * krows * ncol4;  // K items (at most 2*NTHREADS - NQIT)
        // Item slot 0 of every thread is K item tid; slot 1 is q item tid for
        // the first NQIT threads (a whole number of waves, so the buffer a
        // wave reads is wave-uniform) and K item NTHREADS + tid - NQIT after.
        unsigned it_voff[NIT];  // byte offset of the item at channel 0 (OOB: nothing to read)
        int it_pack[NIT];       // LDS index | (shift + 3) << 13 | column mask << 16 | channel << 20 | on << 24
        const bool q_slot = wave < NQIT / 64;  // slot 1 holds a q item
#pragma unroll
        for (int n = 0; n < NIT; ++n) {
          const bool isq = n == 1 && q_slot;
          const int ee = n == 0 ? tid : (isq ? tid : NTHREADS + tid - NQIT);
          it_voff[n] = OOB;
          it_pack[n] = 0;
          if (isq || ee < nkit) {
            const int nc4 = isq ? QC4 : ncol4, nrow = isq ? HROWS : krows;
            const int c = ee / (nrow * nc4), rem = ee - c * (nrow * nc4);
            const int row = rem / nc4, c4 = rem - row * nc4;
            const int gy = Y0 + (isq ? 0 : dh_lo) + row;
            const int gx = (isq ? X0 : X0 + dmin_w) + 4 * c4;
            const int gxl = min(max(gx, 0), g.W - 4);
            int mask = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) mask |= (gx + j >= 0 && gx + j < g.W) ? (1 << j) : 0;
            if (gy >= 0 && gy < g.H && mask) it_voff[n] = (unsigned)((gy * g.W + gxl) * 4);
            const int ldsi = isq ? (c * HROWS + row) * QP + 4 * c4 : (c * KR + row) * KP + 4 * c4;
            it_pack[n] = ldsi | ((gx - gxl + 3) << 13) | (mask << 16) | (c << 20) | (1 << 24);
          }
        }
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        u32x4 stg[NIT];
        auto load_items = [&](int c0) {
#pragma unroll
          for (int n = 0; n < NIT; ++n) {
            const int c = (it_pack[n] >> 20) & 7;
            const unsigned off = (it_voff[n] != OOB && c0 + c < g.Ch) ? it_voff[n] + (unsigned)((c0 + c) * HWi * 4) : OOB;
            stg[n] = __builtin_amdgcn_raw_buffer_load_b128((n == 1 && q_slot) ? q_rs : k_rs, off, 0, 0);
          }
        };
        auto store_items = [&](int bsel) {
#pragma unroll
          for (int n = 0; n < NIT; ++n) {
            const int pk = it_pack[n];
            if (pk & (1 << 24)) {
              // bits 13..19 of the pack read 3 | 15 << 3 for an aligned item
              // with all four columns inside the frame: stored as loaded
              if (((pk >> 13) & 127) != (3 | (15 << 3))) {
                int pkb = pk;
                asm volatile("" : "+v"(pkb));  // selects from the pack here, not from masks kept in SGPRs
                const int sh = ((pkb >> 13) & 7) - 3, mask = (pkb >> 16) & 15;
                const unsigned v0 = stg[n].x, v1 = stg[n].y, v2 = stg[n].z, v3 = stg[n].w;
                unsigned o[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                  const int src = j + sh;  // in 0..3 for every column inside the frame
                  const unsigned val = src <= 0 ? v0 : (src == 1 ? v1 : (src == 2 ? v2 : v3));
                  o[j] = (mask >> j) & 1 ? val : 0u;
                }
                stg[n] = u32x4{o[0], o[1], o[2], o[3]};
              }
              float* dst = (n == 1 && q_slot) ? &sm.qst[bsel][pk & 8191] : &sm.kst[bsel][pk & 8191];
              dst[0] = __uint_as_float(stg[n].x);
              dst[1] = __uint_as_float(stg[n].y);
              dst[2] = __uint_as_float(stg[n].z);
              dst[3] = __uint_as_float(stg[n].w);
            }
          }
        };
        __syncthreads();  // buffers of the previous round / frame are free
        load_items(0);
        store_items(0);
        int bsel = 0;
        for (int c0 = 0; c0 < g.Ch; c0 += CC, bsel ^= 1) {
          __syncthreads();  // chunk c0 is in buffer bsel; buffer bsel^1 is no longer read
          const bool more = c0 + CC < g.Ch;
          if (more) load_items(c0 + CC);  // in flight during this chunk's products
          if (active) {
#pragma unroll 1
            for (int it = 0; it < CC / csplit; ++it) {  // CC is a multiple of csplit: same count for every part
              const int c = part + it * csplit;
              const float* qr = &sm.qst[bsel][(c * HROWS + lane16) * QP];
              const float* kr = &sm.kst[bsel][(c * KR + krow) * KP + blk * S];
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
          if (more) store_items(bsel ^ 1);
        }

        // horizontal box over the patch width, in place (registers)
        box_cols<PS, TQW, HW, S>(acc);
        // vertical box over the patch height, across the 16 lanes of the group
#pragma unroll
        for (int jw = 0; jw < TQW; ++jw)
#pragma unroll
          for (int i = 0; i < S; ++i) {
            float s = row_box<PS>(acc[jw][i]);
            asm volatile("" : "+v"(s));  // materialise the sum here: keeps the row moves short-lived
            acc[jw][i] = s;
          }
        // tail parts: sum over the groups of the wave (fixed order, the same
        // value in every part: (p0 + p1) + (p2 + p3))
        if (wave >= gf / 4 && csplit > 1) {
#pragma unroll
          for (int jw = 0; jw < TQW; ++jw)
#pragma unroll
            for (int i = 0; i < S; ++i) {
              float s = acc[jw][i];
              s += __shfl_xor(s, 16);
              if (csplit == 4) s += __shfl_xor(s, 32);
              acc[jw][i] = s;
            }
        }
        // window tables: the first channel part writes, the other parts of
        // the whole quads add in turn (the tail's part 0 writes the sum)
        for (int pp = 0; pp < csf; ++pp) {
          if (pp > 0) __syncthreads();
          int jl = jh_lane;
          unsigned xm = xmask;
          asm volatile("" : "+v"(jl), "+s"(xm));  // computed here, not kept live across the channel loop
          if (active && part == pp && (pp == 0 || wave < gf / 4) && jl >= 0) {
#pragma unroll
            for (int jw = 0; jw < TQW; ++jw) {  // halo column of the patch origin
              if (!((xm >> jw) & 1u)) continue;
              const int j = jl * tqw + __builtin_popcount(xm & ((1u << jw) - 1u));
              const int u = d_h - sm.qlo_h[j];
              const int vbase = dmin_w + blk * S - sm.qlo_w[j];
              if (u >= 0 && u < WP) {
#pragma unroll
                for (int i = 0; i < S; ++i) {
                  const int v = vbase + i;
                  if (v >= 0 && v < WP) {
                    float* cell = &sm.bw[j * WIN + u * WP + v];
                    *cell = pp == 0 ? acc[jw][i] : *cell + acc[jw][i];
                  }
                }
              }
            }
          }
        }
      }
      __syncthreads();
      // ---- 4-tap combination and exact validity ----
      // Score of window cell (dh, dw) of query j from its box-sum table:
      // bilinear taps at floor(disp), fraction disp - floor(disp).  One
      // thread takes a window row; what depends only on the row (its
      // displacement, validity, table row and the query's offsets) is set up
      // once for the row's cells.
      for (int e = tid; e < qn * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int mh = my0 + j / tqw, mw = mx0 + j % tqw;
        if (mh >= g.nH || mw >= g.nW) continue;
        const int h = mh * s0, w = mw * s0;
        float* srow = scores + ((rowb + mh) * g.nW + mw) * pitch + cbase + dh * ws;
        const float fw = sm.qf_w[j];
        const int lw = sm.qlo_w[j];
        const float disp_h = cand_disp(sm.qf_h[j], g.s1, dh, r);
        const bool okh = centre_ok(h, disp_h, g.H);
        const float fl_h = floorf(disp_h), ah = disp_h - fl_h;
        // table reads only matter for valid cells (row 0 / column 0 otherwise)
        const float* r0p = &sm.bw[j * WIN + (okh ? (int)fl_h - sm.qlo_h[j] : 0) * WP];
        const float* r1p = r0p + WP;
        for (int dw = 0; dw < ws; ++dw) {
          {
            const float disp_w = cand_disp(fw, g.s1, dw, r);
            const bool ok = okh && centre_ok(w, disp_w, g.W);
            const float fl_w = floorf(disp_w), aw = disp_w - fl_w;
            const int col = ok ? (int)fl_w - lw : 0;
            const float top = (1.f - aw) * r0p[col] + aw * r0p[col + 1];
            const float bot = (1.f - aw) * r1p[col] + aw * r1p[col + 1];
            const float dv = (1.f - ah) * top + ah * bot;
            srow[dw] = ok && dv == dv ? dv : -INFINITY;  // NaN scores as invalid
          }
        }
      }
    } else {
      // Union too wide for the LDS layout: score this frame directly.  The
      // workspace holds inner products for both distances (the top-k pass
      // forms the squared L2 distance from them and the norm terms), so the
      // direct scores are inner products too.
      Geo gp = g;
      gp.dist = SNLS_DIST_PROD;
      __syncthreads();
      for (int e = tid; e < qn * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int mh = my0 + j / tqw, mw = mx0 + j % tqw;
        if (mh >= g.nH || mw >= g.nW) continue;
        const int h = mh * s0, w = mw * s0;
        const float fh = sm.qf_h[j], fw = sm.qf_w[j];
        const float disp_h = cand_disp(fh, g.s1, dh, r);
        const bool okh = centre_ok(h, disp_h, g.H);
        for (int dw = 0; dw < ws; ++dw) {
          const float disp_w = cand_disp(fw, g.s1, dw, r);
          float d = -INFINITY;
          if (okh && centre_ok(w, disp_w, g.W)) d = score_candidate(q, k, gp, b, hd, t, h, w, t2, disp_h, disp_w);
          scores[((rowb + mh) * g.nW + mw) * pitch + cbase + dh * ws + dw] = d;
        }
      }
    }
    __syncthreads();
  }
}

// ---- top-k of the scored rows ----
//
// One thread per query row, reading its row of scores 32 at a time with
// 16-byte loads (rows are padded to a multiple of 32 candidates).  A thread
// first takes as threshold the worst of the k query-frame cells nearest the
// window centre (a lower bound of its k-th best: the k best of any k
// candidates rank no higher than the k best of all), so only candidates that
// rank before the threshold reach its register top-k list.  Candidates of
// frames outside the clip score as invalid (-inf), in id order.
namespace tk {
constexpr int ROWS = 256;  // query rows per workgroup (one per thread)
constexpr int CK = 32;     // candidates per pass
constexpr int CP = CK + 4; // private LDS row of a thread (16-byte aligned, spreads the banks)
}  // namespace tk

template <int KMAX>
__global__ void __launch_bounds__(tk::ROWS) tile_topk_kernel(const float* __restrict__ scores,
                                                             const float* __restrict__ gnorm,
                                                             const float* __restrict__ qnorm, int pitch,
                                                             const float* __restrict__ flows, Geo g,
                                                             float* __restrict__ dists, float* __restrict__ inds) {
  using namespace tk;
  __shared__ float4 pass_buf[ROWS * CP / 4];  // a thread's current 32 scores, read back by index
  const int tid = threadIdx.x;
  const long long row = (long long)blockIdx.x * ROWS + tid;
  if (row >= g.rows) return;
  const int ncell = g.ws * g.ws;
  // query of this row
  const int w = (int)(row % g.nW) * g.s0;
  const int h = (int)((row / g.nW) % g.nH) * g.s0;
  const int t = (int)((row / ((long long)g.nW * g.nH)) % g.T);
  const int b = (int)(row / ((long long)g.nW * g.nH * g.T * g.HD));
  const float* srow = scores + row * pitch;
  // ranking score of a candidate: the inner product, or minus the squared L2
  // distance |q|^2 - 2 <q, k~> + |k~|^2 from the norm terms (invalid: -inf)
  const bool l2 = g.dist == SNLS_DIST_L2;
  const float qn = l2 ? qnorm[row] : 0.f;
  const float* grow = l2 ? gnorm + row * pitch : nullptr;
  auto rank_score = [&](float ip, float gn) -> float {
    if (!l2) return ip;
    const float dd = qn - 2.f * ip + gn;
    return ip > -INFINITY && dd == dd ? -dd : -INFINITY;
  };
  // candidate ids of the frames inside the clip
  const int lo = (max(0, t - g.wt) - t + g.wt) * ncell, hi = (min(g.T - 1, t + g.wt) - t + g.wt + 1) * ncell;
  float ts = -INFINITY;  // threshold entry: candidates ranking after it are skipped
  int ti = 0x7fffffff;
  // (the spiral covers the central 9 x 9 cells: a bound needs k of them)
  if (g.k <= ncell && g.k <= 81) {
    ts = INFINITY;
    ti = -1;
    for (int i = 0, n = 0; n < g.k && i < 81; ++i) {
      const int dh = g.r + kSpiral[i][0], dw = g.r + kSpiral[i][1];
      if (dh < 0 || dh >= g.ws || dw < 0 || dw >= g.ws) continue;
      ++n;
      const int id = (g.wt * g.ws + dh) * g.ws + dw;  // query frame: always inside the clip
      const float d = rank_score(srow[id], l2 ? grow[id] : 0.f);
      if (ranks_before(ts, ti, d, id)) {
        ts = d;
        ti = id;
      }
    }
  }
  TopList<KMAX> lst;
  lst.init(g.k);
  float4* const mine = &pass_buf[tid * (CP / 4)];
  for (int c0 = 0; c0 < g.ncand; c0 += CK) {
    float4 v[CK / 4];
#pragma unroll
    for (int i = 0; i < CK / 4; ++i) {
      const int c = c0 + 4 * i;
      v[i] = c + 4 > lo && c < hi ? *reinterpret_cast<const float4*>(srow + c)
                                  : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
    if (l2) {
#pragma unroll
      for (int i = 0; i < CK / 4; ++i) {
        const int c = c0 + 4 * i;
        if (c + 4 > lo && c < hi) {
          const float4 gn = *reinterpret_cast<const float4*>(grow + c);
          v[i] = make_float4(rank_score(v[i].x, gn.x), rank_score(v[i].y, gn.y), rank_score(v[i].z, gn.z),
                             rank_score(v[i].w, gn.w));
        }
      }
    }
    // the tighter of the seed threshold and the list's k-th entry
    if (ranks_before(lst.thr_s(), lst.thr_id(), ts, ti)) {
      ts = lst.thr_s();
      ti = lst.thr_id();
    }
    unsigned mask = 0;
#pragma unroll
    for (int i = 0; i < CK / 4; ++i) {
      const float e[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + 4 * i + u;
        const float sc = c >= lo && c < hi ? e[u] : -INFINITY;
        if (c < g.ncand && (ranks_before(sc, c, ts, ti) || c == ti)) mask |= 1u << (4 * i + u);
      }
    }
    if (mask) {
#pragma unroll
      for (int i = 0; i < CK / 4; ++i) mine[i] = v[i];
      while (mask) {
        const int j = __ffs(mask) - 1;
        mask &= mask - 1;
        const int c = c0 + j;
        const float sc = c >= lo && c < hi ? reinterpret_cast<const float*>(mine)[j] : -INFINITY;
        lst.push(sc, c);
      }
    }
  }
  float* drow = dists + row * g.k;
  float* irow = inds + row * g.k * 3;
  const long long pix = (long long)h * g.W + w;
  const int first = KMAX - g.k;  // slot of the best entry
#pragma unroll
  for (int e = 0; e < KMAX; ++e) {
    if (e >= first) {
      const int i = e - first;
      // every candidate was ranked, so the k best are real candidates; the
      // clamp only keeps a placeholder id in bounds
      const int cid = min(max(lst.id[e], 0), g.ncand - 1);
      const int dw = cid % g.ws, dh = (cid / g.ws) % g.ws, dt = cid / ncell - g.wt;
      float fh = 0.f, fw = 0.f;
      if (dt != 0) {
        const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
        fh = flows[base * g.HW + pix];
        fw = flows[(base + 1) * g.HW + pix];
      }
      drow[i] = from_score(lst.s[e], g.dist);
      irow[3 * i + 0] = (float)(t + dt);
      irow[3 * i + 1] = cand_disp(fh, g.s1, dh, g.r);
      irow[3 * i + 2] = cand_disp(fw, g.s1, dw, g.r);
    }
  }
}

// ---- exact top-k, one wave per scored row (k <= 64, <= 64 * NV candidates) ----
//
// Lane l holds candidates l, l + 64, ... as 32-bit keys ordered like the
// ranking scores (empty slots 0, below every real candidate).  The k-th
// largest of the 64 lane maxima is a lower bound T of the row's k-th best
// (at least k lanes hold a candidate >= T), and on scored rows only a few
// more than k candidates reach it.  Those are compacted into one LDS slot
// per lane and sorted by (score descending, id ascending) with a bitonic
// network across the wave; 65 to 128 take two slots per lane and a
// 128-entry network.  When more than 128 reach T, the exact k-th key is
// found by bisection over the keys instead: every key above it plus the
// smallest ids among the keys equal to it make exactly k entries.
namespace wtk {
constexpr int WAVES = 4;  // rows per workgroup
}  // namespace wtk

// Bitonic sort of one value per lane, descending across lanes 0..63.
template <typename V, typename X>
SNLS_DEV V sort64_desc(V x, int lane, X xchg) {
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const V p = xchg(x, stride);
      const bool take_max = ((lane & stride) == 0) == ((lane & size) == 0);
      x = take_max ? (x > p ? x : p) : (x < p ? x : p);
    }
  return x;
}

template <int NV>
__global__ void __launch_bounds__(wtk::WAVES * 64) wave_topk_kernel(const float* __restrict__ scores,
                                                                    const float* __restrict__ gnorm,
                                                                    const float* __restrict__ qnorm, int pitch,
                                                                    const float* __restrict__ flows, Geo g,
                                                                    float* __restrict__ dists,
                                                                    float* __restrict__ inds) {
  __shared__ unsigned long long slot[wtk::WAVES][128];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long long row = (long long)blockIdx.x * wtk::WAVES + wv;
  if (row >= g.rows) return;  // whole wave
  const int ncell = g.ws * g.ws;
  const int w = (int)(row % g.nW) * g.s0;
  const int h = (int)((row / g.nW) % g.nH) * g.s0;
  const int t = (int)((row / ((long long)g.nW * g.nH)) % g.T);
  const int b = (int)(row / ((long long)g.nW * g.nH * g.T * g.HD));
  const float* srow = scores + row * pitch;
  const bool l2 = g.dist == SNLS_DIST_L2;
  const float qn = l2 ? qnorm[row] : 0.f;
  const float* grow = l2 ? gnorm + row * pitch : nullptr;
  // candidate ids of the frames inside the clip (the others score -inf)
  const int lo = (max(0, t - g.wt) - t + g.wt) * ncell, hi = (min(g.T - 1, t + g.wt) - t + g.wt + 1) * ncell;
  unsigned u[NV];
  unsigned umax = 0;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int c = lane + 64 * v;
    unsigned key = 0;
    if (c < g.ncand) {
      float sc = -INFINITY;
      if (c >= lo && c < hi) {
        const float ip = srow[c];
        if (l2) {
          const float dd = qn - 2.f * ip + grow[c];
          sc = ip > -INFINITY && dd == dd ? -dd : -INFINITY;
        } else {
          sc = ip == ip ? ip : -INFINITY;
        }
      }
      key = order_key(sc);
    }
    u[v] = key;
    umax = max(umax, key);
  }
  auto xchg32 = [](unsigned x, int m) { return (unsigned)__shfl_xor(x, m); };
  const unsigned smax = sort64_desc(umax, lane, xchg32);
  const unsigned top = (unsigned)__shfl(smax, 0);
  const unsigned T1 = (unsigned)__shfl(smax, g.k - 1);
  auto count_ge = [&](unsigned x) {
    int n = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) n += __popcll(__ballot(u[v] >= x));
    return n;
  };
  unsigned long long* sl = slot[wv];
  sl[lane] = 0ull;  // pads rank below every entry
  sl[lane + 64] = 0ull;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  auto entry = [&](unsigned key, int id) { return ((unsigned long long)key << 32) | (unsigned)(~id); };
  const int n1 = count_ge(T1);
  if (n1 <= 128) {
    int base = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const bool take = u[v] >= T1;
      const unsigned long long bal = __ballot(take);
      if (take) sl[base + lanes_below(bal)] = entry(u[v], lane + 64 * v);
      base += __popcll(bal);
    }
  } else {
    // exact k-th key: the largest x with count_ge(x) >= k
    unsigned klo = T1;
    unsigned long long khi = (unsigned long long)top + 1;
    while (khi - klo > 1) {
      const unsigned mid = (unsigned)(klo + (khi - klo) / 2);
      if (count_ge(mid) >= g.k) klo = mid;
      else khi = mid;
    }
    const int need = g.k - (klo < top ? count_ge(klo + 1) : 0);  // entries equal to the k-th key
    int base = 0, eqn = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const bool eq = u[v] == klo;
      const unsigned long long beq = __ballot(eq);
      const bool take = u[v] > klo || (eq && eqn + lanes_below(beq) < need);
      eqn += __popcll(beq);
      const unsigned long long bal = __ballot(take);
      if (take) sl[base + lanes_below(bal)] = entry(u[v], lane + 64 * v);
      base += __popcll(bal);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  unsigned long long best;
  if (n1 > 64 && n1 <= 128) {
    // up to 128 entries, two per lane (entry lane + 64 h): bitonic sort of
    // the 128, descending; the step across the halves is within the lane
    unsigned long long x0 = sl[lane], x1 = sl[lane + 64];
#pragma unroll
    for (int size = 2; size <= 128; size <<= 1)
#pragma unroll
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        if (stride == 64) {  // size 128: element i pairs with i + 64, larger first
          const unsigned long long hi = x0 > x1 ? x0 : x1, lo = x0 > x1 ? x1 : x0;
          x0 = hi;
          x1 = lo;
        } else {
          const unsigned long long p0 = shfl_xor64(x0, stride), p1 = shfl_xor64(x1, stride);
          // element i = lane + 64 h keeps the larger of the pair when the
          // pair's order within its size-block is descending and it is the
          // lower index, or ascending and it is the higher index
          const bool low = (lane & stride) == 0;
          const bool desc0 = (lane & size) == 0, desc1 = ((lane + 64) & size) == 0;
          x0 = (low == desc0) ? (x0 > p0 ? x0 : p0) : (x0 < p0 ? x0 : p0);
          x1 = (low == desc1) ? (x1 > p1 ? x1 : p1) : (x1 < p1 ? x1 : p1);
        }
      }
    best = x0;  // ranks 0..63 are the first halves
  } else {
    best = sort64_desc(sl[lane], lane, shfl_xor64);
  }
  if (lane >= g.k) return;
  // every candidate was ranked, so the k best are real candidates; the clamp
  // only keeps a placeholder id in bounds
  const int cid = min(max((int)~(unsigned)best, 0), g.ncand - 1);
  const int dw = cid % g.ws, dh = (cid / g.ws) % g.ws, dt = cid / ncell - g.wt;
  float fh = 0.f, fw = 0.f;
  if (dt != 0) {
    const long long pix = (long long)h * g.W + w;
    const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
    fh = flows[base * g.HW + pix];
    fw = flows[(base + 1) * g.HW + pix];
  }
  dists[row * g.k + lane] = from_score(key_score((unsigned)(best >> 32)), g.dist);
  float* irow = inds + (row * g.k + lane) * 3;
  irow[0] = (float)(t + dt);
  irow[1] = cand_disp(fh, g.s1, dh, g.r);
  irow[2] = cand_disp(fw, g.s1, dw, g.r);
}

// The tiled path handles any S_Q, P <= 7, Ws <= 9 with the inner product
// (S_K <= 1) or the squared L2 distance (S_K = 1).
bool tile_supported(const Geo& g) {
  const bool dist_ok = g.s1 > 0.f && g.s1 <= 1.0f;  // both distances (L2: norm terms per cell unless S_K = 1)
  // windows above 9 only at P = 7: its 80-query tile keeps 15 x 15 windows'
  // tables within the LDS (smaller patches make taller tiles); their L2 norm
  // terms are formed cell by cell
  const bool ws_ok = g.ws <= tile::WSMAX || (g.ws <= tile::WSBIG && g.ps == 7);
  return dist_ok && g.ps <= 7 && ws_ok && g.W >= 4 && g.k >= 1 &&
         (long long)g.Ch * g.HW * 4 < (1LL << 31);
}

// Workspace rows hold the scores of one query row, padded to a multiple of
// 32 candidates: each 32-candidate pass of the top-k reads one whole
// 128-byte line (480x854 top-k 1.43 -> 1.16 ms against 16-byte padding).
static int tile_ws_pitch(const Geo& g) { return (g.ncand + 31) & ~31; }
static size_t tile_plane_bytes(const Geo& g) {
  return ((size_t)g.rows * (size_t)tile_ws_pitch(g) * sizeof(float) + 255) & ~(size_t)255;
}
size_t tile_ws_bytes(const Geo& g) {
  size_t b = tile_plane_bytes(g);                             // inner-product scores
  if (g.dist == SNLS_DIST_L2)  // key and query norm terms, key pair planes
    b += tile_plane_bytes(g) + (((size_t)g.rows * sizeof(float) + 255) & ~(size_t)255) + l2_planes_bytes(g);
  return b;
}

// Top-k of the scored rows (any scores kernel of the tiled family).
static snls_status launch_tile_topk(const float* scores, const float* gnorm, const float* qnorm, int pitch,
                                    const float* flows, const Geo& g, float* dists, float* inds, hipStream_t s) {
  // Large k: the thread-per-row list insertions diverge on nearly every
  // candidate, the wave-per-row selection does not.
  const int nv = (g.ncand + 63) / 64;
  if (g.k > 16 && g.k <= 64 && nv <= 32) {
    const unsigned wblocks = (unsigned)((g.rows + wtk::WAVES - 1) / wtk::WAVES);
#define SNLS_WTK(N)                                                                                               \
  hipLaunchKernelGGL(wave_topk_kernel<N>, dim3(wblocks), dim3(wtk::WAVES * 64), 0, s, scores, gnorm, qnorm, pitch, \
                     flows, g, dists, inds)
    if (nv <= 4) SNLS_WTK(4);
    else if (nv <= 8) SNLS_WTK(8);
    else if (nv <= 12) SNLS_WTK(12);
    else if (nv <= 16) SNLS_WTK(16);
    else if (nv <= 20) SNLS_WTK(20);
    else if (nv <= 25) SNLS_WTK(25);
    else SNLS_WTK(32);
#undef SNLS_WTK
    return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
  }
  const unsigned tblocks = (unsigned)((g.rows + tk::ROWS - 1) / tk::ROWS);
  if (g.k <= 12)
    hipLaunchKernelGGL(tile_topk_kernel<12>, dim3(tblocks), dim3(tk::ROWS), 0, s, scores, gnorm, qnorm, pitch, flows,
                       g, dists, inds);
  else if (g.k <= 16)
    hipLaunchKernelGGL(tile_topk_kernel<16>, dim3(tblocks), dim3(tk::ROWS), 0, s, scores, gnorm, qnorm, pitch, flows,
                       g, dists, inds);
  else if (g.k <= 32)
    hipLaunchKernelGGL(tile_topk_kernel<32>, dim3(tblocks), dim3(tk::ROWS), 0, s, scores, gnorm, qnorm, pitch, flows,
                       g, dists, inds);
  else if (g.k <= 64)
    hipLaunchKernelGGL(tile_topk_kernel<64>, dim3(tblocks), dim3(tk::ROWS), 0, s, scores, gnorm, qnorm, pitch, flows,
                       g, dists, inds);
  else
    hipLaunchKernelGGL(tile_topk_kernel<128>, dim3(tblocks), dim3(tk::ROWS), 0, s, scores, gnorm, qnorm, pitch, flows,
                       g, dists, inds);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_search_p1(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                             float* inds, float* scores, hipStream_t s) {
  const int pitch = tile_ws_pitch(g);
  const snls_status st = launch_search_p1_scores(q, k, flows, g, scores, pitch, s);
  if (st != SNLS_OK) return st;
  return launch_tile_topk(scores, nullptr, nullptr, pitch, flows, g, dists, inds, s);
}

snls_status launch_search_tile(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                               float* inds, float* scores, hipStream_t s) {
  // tile of tqh x tqw queries (the kernel derives the same from S_Q)
  const int tqh = (tile::HROWS - g.ps) / g.s0 + 1, tqw = (tile::TQW - 1) / g.s0 + 1;
  const int tiles_x = (g.nW + tqw - 1) / tqw;
  const int tiles_y = (g.nH + tqh - 1) / tqh;
  const long long nwg = (long long)tiles_x * tiles_y * g.B * g.HD * g.T;
  if (nwg == 0) return SNLS_OK;
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  dim3 grid((unsigned)nwg), block(tile::NTHREADS);
  switch (g.ws > tile::WSMAX ? 0 : g.ps) {
    case 0:  // P = 7 with a window above 9 (tile_supported)
      hipLaunchKernelGGL((search_tile_scores_kernel<7, tile::WSBIG>), grid, block, 0, s, q, k, flows, g, tiles_x,
                         tiles_y, scores, tile_ws_pitch(g));
      break;
#define SNLS_TILE_CASE(P)                                                                                       \
  case P:                                                                                                       \
    hipLaunchKernelGGL((search_tile_scores_kernel<P, tile::WSMAX>), grid, block, 0, s, q, k, flows, g, tiles_x, \
                       tiles_y, scores, tile_ws_pitch(g));                                                      \
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
  const int pitch = tile_ws_pitch(g);
  float* gnorm = nullptr;
  float* qnorm = nullptr;
  if (g.dist == SNLS_DIST_L2) {
    gnorm = reinterpret_cast<float*>(reinterpret_cast<char*>(scores) + tile_plane_bytes(g));
    qnorm = reinterpret_cast<float*>(reinterpret_cast<char*>(gnorm) + tile_plane_bytes(g));
    float* planes = reinterpret_cast<float*>(reinterpret_cast<char*>(qnorm) +
                                             (((size_t)g.rows * sizeof(float) + 255) & ~(size_t)255));
    const snls_status st = launch_l2_norms(q, k, flows, g, gnorm, pitch, qnorm, planes, s);
    if (st != SNLS_OK) return st;
  }
  return launch_tile_topk(scores, gnorm, qnorm, pitch, flows, g, dists, inds, s);
}

}  // namespace snls

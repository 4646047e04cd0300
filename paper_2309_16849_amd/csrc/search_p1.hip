// search_p1.hip -- the shifted search for single-pixel patches (P = 1), any
// query stride, key stride 1, inner product (Sec. 3.2).
//
// With P = 1 a candidate's score is the bilinear combination of four pixel
// correlations c(y, x) = <q(query), K(y, x)>.  Window row d_h reads its taps
// from key rows Y(d_h) = h + floor(disp_h) and Y(d_h) + 1, and from the ws + 2
// columns starting at floor(disp_w of cell 0) (the cells' floors are
// nondecreasing and, for key stride 1, each lies within one of its ideal
// column).  Y(d_h + 1) is Y(d_h) + 1 except when rounding of the offset
// lands on an integer, so the 16 threads of a query each accumulate the
// correlations of ONE key row -- thread d_h row Y(d_h), thread ws the row
// below the last -- over the head's channels from an LDS copy of the key
// region the tile's windows span, and a window row takes its second row from
// the next lane (DPP).  A row whose next key row is not Y + 1 is scored
// directly.
//
// Two kernels use these scores:
//  * search_p1_topk_kernel (k <= 32): one workgroup loops over the frames of
//    the window and keeps each query's top k itself (no score workspace);
//  * search_p1_scores_kernel (larger k): one workgroup per frame writes the
//    scores to the workspace rows for the streaming top-k kernel.
#include "snls_internal.h"

namespace snls {

namespace p1 {
// TQH x TQW queries per workgroup (query-grid units).  4 x 8 queries make a
// 512-thread workgroup whose LDS (about 72 KB) and registers (at most 128
// VGPRs) let two workgroups share a CU, so one's barriers and selection
// overlap the other's staging and products.
constexpr int TQH = 4, TQW = 8;
constexpr int NQ = TQH * TQW;
constexpr int WSM = 15;                // largest window side
constexpr int NR = 16;                 // thread slots per query (key rows): one 16-lane DPP row
constexpr int NT = NQ * NR;            // 512
constexpr int NC = WSM + 2;            // correlation columns per key row
constexpr int CC = 4;                  // channels per staging chunk (double-buffered)
constexpr int RH = 40, RW = 48;        // key region of the tile
constexpr int RP = RW + 1;             // row pitch (odd)
constexpr int NRI = (RH + NT / 64 - 1) / (NT / 64);  // region rows per thread (lane = column)
constexpr int CHUNK = CC * RH * RP;
constexpr int QR = WSM + 2;            // per-query block (when the tile's region is too wide): rows ..
constexpr int QB = QR * NC;            // .. x NC columns, one channel at a time
constexpr int LS = 32;                 // list slots per query in the fused selection (2 per lane)
constexpr int WPE = 4;                 // waves per SIMD the registers are budgeted for (128 VGPRs)
static_assert(NQ * QB <= 2 * CHUNK, "per-query blocks fit in the two staging buffers");
static_assert(RW <= 64, "a region row is staged by one wave");
static_assert(NQ * WSM * WSM <= 2 * CHUNK, "the tile's scores of one frame fit in the staging buffers");
}  // namespace p1

// Value of lane i + 1 of the same 16-lane row (lane 15 reads 0).
SNLS_DEV float next_lane(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x101, 0xf, 0xf, true));
}
SNLS_DEV int next_lane(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x101, 0xf, 0xf, true); }

// ---- 16-lane group operations (the 16 threads of a query are one DPP row) ----

// DPP row operation CTRL on a 32-bit value (every lane of the row is active).
template <int CTRL>
SNLS_DEV unsigned dpp_row(unsigned v) {
  return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xf, 0xf, false);
}
// Value of lane i ^ M of the group (M in {1, 2, 4, 8, 15}; l = i) through
// DPP, not the LDS crossbar: quad permutes for 1 and 2, a row rotation by 8,
// for 4 a rotation by 4 (lane i - 4, bit 2 of i set) or by 12 (lane i + 4),
// the row mirror for 15.  A rotation by N gives lane i the value of lane
// (i - N) mod 16.
template <int M>
SNLS_DEV unsigned grp_xor(unsigned x, int l) {
  static_assert(M == 1 || M == 2 || M == 4 || M == 8 || M == 15, "partner distance");
  if constexpr (M == 1) return dpp_row<0xB1>(x);  // quad_perm [1,0,3,2]
  else if constexpr (M == 2) return dpp_row<0x4E>(x);  // quad_perm [2,3,0,1]
  else if constexpr (M == 8) return dpp_row<0x128>(x);  // row_ror:8
  else if constexpr (M == 15) return dpp_row<0x140>(x);  // row_mirror
  else {
    // both rotations run with every lane of the row active (a DPP read from
    // a lane switched off by a branch returns 0), then one is selected
    unsigned a = dpp_row<0x124>(x), b = dpp_row<0x12C>(x);  // row_ror:4 / row_ror:12
    asm volatile("" : "+v"(a), "+v"(b));
    return (l & 4) ? a : b;
  }
}
template <int M>
SNLS_DEV unsigned long long grp_xor64(unsigned long long x, int l) {
  return ((unsigned long long)grp_xor<M>((unsigned)(x >> 32), l) << 32) | grp_xor<M>((unsigned)x, l);
}
// Sum and maximum over the group (every lane gets the result): rotations by
// 8, 4, 2 and 1 lanes -- after the step by 8 a lane's value depends only on
// its lane mod 8, so the rotation by 4 reads its xor-4 partner's value, and
// so on.
SNLS_DEV int grp_sum(int x) {
  x += (int)dpp_row<0x128>((unsigned)x);
  x += (int)dpp_row<0x124>((unsigned)x);
  x += (int)dpp_row<0x122>((unsigned)x);
  x += (int)dpp_row<0x121>((unsigned)x);
  return x;
}
SNLS_DEV unsigned grp_max(unsigned x) {
  x = max(x, dpp_row<0x128>(x));
  x = max(x, dpp_row<0x124>(x));
  x = max(x, dpp_row<0x122>(x));
  x = max(x, dpp_row<0x121>(x));
  return x;
}
// Value of lane i - N of the row (0 for i < N).
template <int N>
SNLS_DEV int row_shr(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x110 + N, 0xf, 0xf, true);
}
// Exclusive prefix sum over the lanes of the group.
SNLS_DEV int grp_excl_scan(int x) {
  int s = x;
  s += row_shr<1>(s);
  s += row_shr<2>(s);
  s += row_shr<4>(s);
  s += row_shr<8>(s);
  return s - x;
}

// Slot 2 dh - 1 of the list (lane dh - 1's second entry) and the flag of
// the lane before; lane 0 of the group gets 0 and true (no slot before it).
SNLS_DEV unsigned long long prev_lane64(unsigned long long x) {
  const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)x, 0x111, 0xf, 0xf, true);
  const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)(x >> 32), 0x111, 0xf, 0xf, true);
  return ((unsigned long long)hi << 32) | lo;
}
SNLS_DEV bool prev_lane_flag(bool f) { return __builtin_amdgcn_update_dpp(1, f ? 1 : 0, 0x111, 0xf, 0xf, false) != 0; }

// Inverse of order_key.
SNLS_DEV unsigned order_key_inv(unsigned u) { return (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u; }

// Survivors of a frame up to this many are inserted one by one; more are
// sorted and merged.
constexpr int kInsertMax = 20;

// One compare-exchange stage of a bitonic network over the group's 32
// entries, element e = 2 * lane + half, ending in descending order.
template <int SIZE, int STRIDE>
SNLS_DEV void bitonic_stage(unsigned long long& x0, unsigned long long& x1, int l) {
  const bool desc = ((2 * l) & SIZE) == 0;
  if constexpr (STRIDE == 1) {
    const unsigned long long hi = x0 > x1 ? x0 : x1, lo = x0 > x1 ? x1 : x0;
    x0 = desc ? hi : lo;
    x1 = desc ? lo : hi;
  } else {
    constexpr int LM = STRIDE / 2;  // partner lane distance
    const unsigned long long p0 = grp_xor64<LM>(x0, l), p1 = grp_xor64<LM>(x1, l);
    const bool keep_max = ((l & LM) == 0) == desc;
    x0 = keep_max ? (x0 > p0 ? x0 : p0) : (x0 < p0 ? x0 : p0);
    x1 = keep_max ? (x1 > p1 ? x1 : p1) : (x1 < p1 ? x1 : p1);
  }
}

// Sort the group's 32 entries in descending order.  The lane index is made
// opaque so that each stage forms its direction flags from it instead of a
// caller's loop keeping every stage's lane masks live.
SNLS_DEV void bitonic_sort32(unsigned long long& x0, unsigned long long& x1, int l) {
  asm volatile("" : "+v"(l));
  bitonic_stage<2, 1>(x0, x1, l);
  bitonic_stage<4, 2>(x0, x1, l);
  bitonic_stage<4, 1>(x0, x1, l);
  bitonic_stage<8, 4>(x0, x1, l);
  bitonic_stage<8, 2>(x0, x1, l);
  bitonic_stage<8, 1>(x0, x1, l);
  bitonic_stage<16, 8>(x0, x1, l);
  bitonic_stage<16, 4>(x0, x1, l);
  bitonic_stage<16, 2>(x0, x1, l);
  bitonic_stage<16, 1>(x0, x1, l);
  bitonic_stage<32, 16>(x0, x1, l);
  bitonic_stage<32, 8>(x0, x1, l);
  bitonic_stage<32, 4>(x0, x1, l);
  bitonic_stage<32, 2>(x0, x1, l);
  bitonic_stage<32, 1>(x0, x1, l);
}

// The 32 best of two descending lists of 32 (a: the list, s: sorted
// survivors), in descending order: element e takes max(a[e], s[31 - e]),
// a bitonic sequence, then a bitonic merge.
SNLS_DEV void merge_top32(unsigned long long& a0, unsigned long long& a1, unsigned long long s0,
                          unsigned long long s1, int l) {
  asm volatile("" : "+v"(l));  // as in bitonic_sort32
  // s[31 - e] for e = 2l is s1 of lane 15 - l, for e = 2l + 1 it is s0
  const unsigned long long r0 = grp_xor64<15>(s1, l), r1 = grp_xor64<15>(s0, l);
  a0 = a0 > r0 ? a0 : r0;
  a1 = a1 > r1 ? a1 : r1;
  bitonic_stage<64, 16>(a0, a1, l);
  bitonic_stage<64, 8>(a0, a1, l);
  bitonic_stage<64, 4>(a0, a1, l);
  bitonic_stage<64, 2>(a0, a1, l);
  bitonic_stage<64, 1>(a0, a1, l);
}

// Bit d_w set where pred(d_w) holds, for the WSM columns of a window row;
// built by shifts, so no per-column constants are held in registers.
template <class Pred>
SNLS_DEV unsigned col_mask(Pred pred) {
  unsigned m = 0;
#pragma unroll
  for (int dw = p1::WSM - 1; dw >= 0; --dw) m = m + m + (pred(dw) ? 1u : 0u);  // one add with carry-in
  return m;
}

// ---- scores of one frame ----

// Score of a cell that does not exist (d_w >= ws, a thread with d_h >= ws, a
// query outside the grid): the NaN whose order key is 0, so that comparisons
// and order keys drop it without per-column masks.
SNLS_DEV float no_cell() { return __uint_as_float(0xffffffffu); }

// Number of real cells in the calling thread's window row: ws, or 0 for
// threads with d_h >= ws and queries outside the grid.  The thread index is
// opaque, so the per-column compares against it stay inside a caller's frame
// loop instead of being hoisted as live lane masks.
template <int WSF>
SNLS_DEV int p1_row_cells(const Geo& g, int ty, int tx) {
  using namespace p1;
  int tid = threadIdx.x, ws = WSF > 0 ? WSF : g.ws;
  asm volatile("" : "+v"(tid));
  if constexpr (WSF == 0) asm volatile("" : "+s"(ws));
  const int j = tid / NR, dh = tid % NR;
  const int mh = ty * TQH + j / TQW, mw = tx * TQW + j % TQW;
  return (mh < g.nH && mw < g.nW && dh < ws) ? ws : 0;
}

struct P1Smem {
  // key region chunks (double buffer), pixel-major with the chunk's CC
  // channels of a pixel in one 16-byte slot; per-query blocks (one channel,
  // plane layout) use both buffers
  alignas(16) float reg[2][p1::CHUNK];
  alignas(16) float qs[2][p1::NQ][p1::CC];  // query values of a chunk
  int ubox[4];                  // key rows and columns the tile's windows span
  int y0q[p1::NQ], x0q[p1::NQ];  // first key row and column of each query's block
};

// Scores of the window row of thread (j = tid / 16, d_h = tid % 16) for frame
// step dt of query tile (ty, tx) of image (b, hd, t): sc[d_w] for d_w < ws,
// -inf for invalid cells and NaN similarities, no_cell() where there is no
// cell (d_w >= ws; every d_w of threads with d_h >= ws and of queries outside
// the grid).  Workgroup barriers inside: every
// thread calls it; its staging buffers are free again at the caller's next
// barrier.
template <int WSF>
SNLS_DEV void p1_frame_scores(P1Smem& sm, const float* __restrict__ q, const float* __restrict__ k,
                              const float* __restrict__ flows, const Geo& g, int b, int hd, int t, int dt, int ty,
                              int tx, float (&sc)[p1::WSM]) {
  using namespace p1;
  // The thread index is made opaque here so that what derives from it is
  // recomputed per frame rather than hoisted out of a caller's frame loop
  // and kept live (spilled) across the selection.
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  // The window side and radius likewise: the per-column values derived from
  // them (offsets d - r, column compares) are formed where they are used
  // instead of being held in registers across the caller's loop; a window
  // side fixed at compile time (WSF > 0) makes them immediates instead.  The
  // key stride is 1 on this route, so a cell's offset is F + (d - r).
  int ws = WSF > 0 ? WSF : g.ws, r = WSF > 0 ? WSF / 2 : g.r;
  if constexpr (WSF == 0) asm volatile("" : "+s"(ws), "+s"(r));
  const int j = tid / NR, dh = tid % NR;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index (uniform)
  const int t2 = t + dt;
  const int mh = ty * TQH + j / TQW, mw = tx * TQW + j % TQW;  // query-grid position
  const bool inside = mh < g.nH && mw < g.nW;
  const bool rowtask = inside && dh <= ws;  // thread accumulates a key row
  const int h = mh * g.s0, w = mw * g.s0;

  float fh = 0.f, fw = 0.f;
  if (dt != 0 && inside) {
    const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
    const long long pix = (long long)h * g.W + w;
    fh = flows[base * g.HW + pix];
    fw = flows[(base + 1) * g.HW + pix];
  }
  // this thread's key row and the first column of the query's rows; offsets
  // that are not finite or absurdly large are placed at 0 for the region
  // (their cells fail the exact validity test)
  const int drow = min(dh, ws - 1);
  const float disp_h = cand_disp(fh, 1.f, drow, r);
  const float disp_w0 = cand_disp(fw, 1.f, 0, r);
  const bool sane = fabsf(fh) < kFarDisp && fabsf(fw) < kFarDisp;
  const int below = dh == ws ? 1 : 0;  // the row under the last window row
  const int y0 = (sane ? h + (int)floorf(disp_h) : h) + below;
  const int x0 = sane ? w + (int)floorf(disp_w0) : w;
  if (tid < 4) sm.ubox[tid] = (tid & 1) ? INT_MIN : INT_MAX;
  if (dh == 0) {
    sm.y0q[j] = y0;
    sm.x0q[j] = x0;
  }
  __syncthreads();
  {
    // union bounds: a query's key rows grow with d_h (its first row at d_h =
    // 0, its last at d_h = ws) and all its rows start at one column, so a
    // wave reads the bounds from its queries' lanes; one LDS atomic per wave
    int a0 = INT_MAX, a1 = INT_MIN, a2 = INT_MAX, a3 = INT_MIN;
#pragma unroll
    for (int qq = 0; qq < 64 / NR; ++qq) {
      const int jq = wv * (64 / NR) + qq;  // the query of lanes NR qq .. NR qq + NR - 1
      if (ty * TQH + jq / TQW < g.nH && tx * TQW + jq % TQW < g.nW) {
        a0 = min(a0, __builtin_amdgcn_readlane(y0, NR * qq));
        a1 = max(a1, __builtin_amdgcn_readlane(y0, NR * qq + ws));
        a2 = min(a2, __builtin_amdgcn_readlane(x0, NR * qq));
        a3 = max(a3, __builtin_amdgcn_readlane(x0, NR * qq));
      }
    }
    if ((tid & 63) == 0 && a0 <= a1) {
      atomicMin(&sm.ubox[0], a0);
      atomicMax(&sm.ubox[1], a1);
      atomicMin(&sm.ubox[2], a2);
      atomicMax(&sm.ubox[3], a3);
    }
  }
  __syncthreads();
  const int ry0 = sm.ubox[0], rx0 = sm.ubox[2];
  const int rh = sm.ubox[1] - ry0 + 1, rw = sm.ubox[3] - rx0 + NC;
  // The tile's key region is staged CC channels at a time when it fits;
  // otherwise (windows far apart) each query's own block of rows and
  // columns is staged, one channel at a time.
  const bool staged = sm.ubox[1] >= sm.ubox[0] && rh <= RH && rw <= RW;

  const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;
  auto kval = [&](int c, int y, int x) -> float {
    return (y >= 0 && y < g.H && x >= 0 && x < g.W) ? kb[(long long)c * g.HW + (long long)y * g.W + x] : 0.f;
  };
  // Region staging through registers: lane = column, the NT / 64 waves take the
  // rows (NRI rows each); a chunk's loads are issued before the products of
  // the previous chunk and written to LDS after them.
  const int xx = tid & 63;
  // Branch-free region loads: a raw buffer load at an offset past the
  // buffer's extent reads 0 (pixels outside the frame, channels past the
  // head).  Offsets stay below 2^31: p1_supported requires Ch*H*W*4 < 2^31.
  constexpr unsigned OOB = 0x80000000u;
  const __amdgpu_buffer_rsrc_t k_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)kb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);
  unsigned roff[NRI];  // byte offset of this thread's region pixels in channel 0 (OOB: none)
  const int x = rx0 + xx;
  const bool colok = staged && xx < rw && x >= 0 && x < g.W;
#pragma unroll
  for (int i = 0; i < NRI; ++i) {
    const int yy = wv + (NT / 64) * i, y = ry0 + yy;  // uniform: the row test is scalar
    roff[i] = (yy < rh && y >= 0 && y < g.H && colok) ? (unsigned)((y * g.W + x) * 4) : OOB;
  }
  // this thread's q staging item (tid < CC * NQ): channel tid / NQ of query
  // tid % NQ, as a byte offset in channel 0 (OOB: outside the frame)
  const __amdgpu_buffer_rsrc_t q_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)qb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);
  unsigned qoff = OOB;
  if (tid < CC * NQ) {
    const int c = tid / NQ, jj = tid % NQ;
    const int qh = (ty * TQH + jj / TQW) * g.s0, qw = (tx * TQW + jj % TQW) * g.s0;
    if (qh < g.H && qw < g.W) qoff = (unsigned)(((long long)c * g.HW + (long long)qh * g.W + qw) * 4);
  }
  float stg[CC][NRI];
  float qstg = 0.f;
  // The channel offset goes into the loads' scalar offset: a channel past
  // the head lands past the buffer's extent and reads 0 (p1_supported keeps
  // (Ch + CC) * H * W * 4 below 2^31, so no offset wraps).
  const int hwb = (int)g.HW * 4;
  auto load_chunk = [&](int c0) {
#pragma unroll
    for (int c = 0; c < CC; ++c)
#pragma unroll
      for (int i = 0; i < NRI; ++i)
        stg[c][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(k_rs, roff[i], (c0 + c) * hwb, 0));
    if (tid < CC * NQ)
      qstg = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(q_rs, qoff, c0 * hwb, 0));
  };
  auto store_chunk = [&](int buf) {
    // rows past the region and columns up to the pitch receive zeros that are never read
    if (xx < RP) {
      float4* r4 = reinterpret_cast<float4*>(sm.reg[buf]);
#pragma unroll
      for (int i = 0; i < NRI; ++i)
        r4[(wv + (NT / 64) * i) * RP + xx] = make_float4(stg[0][i], stg[1][i], stg[2][i], stg[3][i]);
    }
    if (tid < CC * NQ) sm.qs[buf][tid % NQ][tid / NQ] = qstg;
  };
  // Per-query blocks (windows far apart): one channel at a time.
  auto stage_blocks = [&](int c0) {
    for (int e = tid; e < NQ * QB; e += NT) {  // both buffers: no double buffering
      const int jj = e / QB, rem = e - jj * QB;
      const int yy = rem / NC, x = rem - yy * NC;
      (&sm.reg[0][0])[e] = kval(c0, sm.y0q[jj] + yy, sm.x0q[jj] + x);
    }
    if (tid < NQ) {
      const int qh = (ty * TQH + tid / TQW) * g.s0, qw = (tx * TQW + tid % TQW) * g.s0;
      sm.qs[0][tid][0] = (qh < g.H && qw < g.W) ? qb[(long long)c0 * g.HW + (long long)qh * g.W + qw] : 0.f;
    }
  };
  // this thread's row in the staging buffer
  const int toff = staged ? (y0 - ry0) * RP + (x0 - rx0) : j * QB + (y0 - sm.y0q[j]) * NC;

  float cr[NC];  // correlations of key row y0, columns x0 ..
#pragma unroll
  for (int x = 0; x < NC; ++x) cr[x] = 0.f;
  // Two separate loops (the branch is uniform), so that the accumulators
  // are not merged from two paths on every chunk.
  if (staged) {
    load_chunk(0);
    store_chunk(0);
    int buf = 0;
    for (int c0 = 0; c0 < g.Ch; c0 += CC, buf ^= 1) {
      const bool more = c0 + CC < g.Ch;
      __syncthreads();                 // chunk c0 is staged in buf; buf^1 is free
      if (more) load_chunk(c0 + CC);  // in flight during this chunk's products
      if (rowtask) {
        // channels past the head were staged as zeros
        static_assert(CC == 4, "one 16-byte slot per pixel");
        const float4 q4 = *reinterpret_cast<const float4*>(sm.qs[buf][j]);
        const float4* r4 = reinterpret_cast<const float4*>(sm.reg[buf]) + toff;
#pragma unroll
        for (int x = 0; x < NC; ++x) {
          const float4 kv = r4[x];
          cr[x] = fmaf(q4.x, kv.x, cr[x]);
          cr[x] = fmaf(q4.y, kv.y, cr[x]);
          cr[x] = fmaf(q4.z, kv.z, cr[x]);
          cr[x] = fmaf(q4.w, kv.w, cr[x]);
        }
      }
      if (more) store_chunk(buf ^ 1);
    }
  } else {
    for (int c0 = 0; c0 < g.Ch; ++c0) {
      __syncthreads();  // the previous channel is no longer read
      stage_blocks(c0);
      __syncthreads();
      if (rowtask) {
        const float qv = sm.qs[0][j][0];
        const float* r0 = &sm.reg[0][0] + toff;
#pragma unroll
        for (int x = 0; x < NC; ++x) cr[x] = fmaf(qv, r0[x], cr[x]);
      }
    }
  }
  const int ynext = next_lane(y0);
  const bool okh = inside && dh < ws && centre_ok(h, disp_h, g.H) && sane;
#pragma unroll
  for (int dw = 0; dw < WSM; ++dw) sc[dw] = -INFINITY;
  // Common case: offsets below 64 px whose fractions lie at least 1e-3 from
  // an integer (or are integers): F + (d - r) never rounds across an
  // integer, so every window row's next key row is Y + 1, cell d_w's taps
  // are columns d_w and d_w + 1, and its floor is floor(disp_w0) + d_w.
  const float afh = fabsf(fh), afw = fabsf(fw);
  const float frh = afh - floorf(afh), frw = afw - floorf(afw);
  const bool fast = sane && afh < 64.f && afw < 64.f && (frh == 0.f || (frh >= 1e-3f && frh <= 1.f - 1e-3f)) &&
                    (frw == 0.f || (frw >= 1e-3f && frw <= 1.f - 1e-3f));
  if (fast) {
    // each row interpolates its own correlations along the columns, the
    // next row's come from the next lane (every lane of the query takes part)
    const float fl0 = floorf(disp_w0);
    const float ah = disp_h - floorf(disp_h);
    // Valid cells: centre column w + disp_w in [0, W-1], i.e. d_w - r in
    // [-w - F, W-1-w - F].  Here the rounded offsets stay between the same
    // integers as the exact ones, and the bounds below are computed with an
    // error far below the fractions' 1e-3 distance from an integer, so their
    // ceiling and floor give the exact range of d_w.
    const int dlo = okh ? max(0, (int)ceilf((float)(r - w) - fw)) : WSM;
    const int dhi = min(ws - 1, (int)floorf((float)(g.W - 1 - w + r) - fw));
    float top[WSM];
#pragma unroll
    for (int dw = 0; dw < WSM; ++dw) {
      const float disp_w = cand_disp(fw, 1.f, dw, r);
      const float aw = disp_w - (fl0 + (float)dw);
      top[dw] = fmaf(aw, cr[dw + 1] - cr[dw], cr[dw]);
    }
#pragma unroll
    for (int dw = 0; dw < WSM; ++dw) {
      const float bot = next_lane(top[dw]);
      const float dv = fmaf(ah, bot - top[dw], top[dw]);
      sc[dw] = dw >= dlo && dw <= dhi ? fmaxf(dv, -INFINITY) : -INFINITY;  // NaN scores as invalid
    }
  } else {
    // the key row below from the next lane (every lane takes part)
    float cn[NC];
#pragma unroll
    for (int x = 0; x < NC; ++x) cn[x] = next_lane(cr[x]);
    if (okh && ynext != y0 + 1) {
      // rounding moved the next window row by two key rows: score directly
      // (one call site; the score lands in its register by selects)
#pragma unroll 1
      for (int dw = 0; dw < ws; ++dw) {
        const float disp_w = cand_disp(fw, 1.f, dw, r);
        const float d = centre_ok(w, disp_w, g.W)
                            ? fmaxf(score_candidate(q, k, g, b, hd, t, h, w, t2, disp_h, disp_w), -INFINITY)
                            : -INFINITY;
#pragma unroll
        for (int i = 0; i < WSM; ++i) sc[i] = i == dw ? d : sc[i];
      }
    } else if (okh) {
      // taps from each cell's own displacement
      const float ah = disp_h - floorf(disp_h);
      const int fl0 = (int)floorf(disp_w0);
#pragma unroll
      for (int dw = 0; dw < WSM; ++dw) {
        if (dw < ws) {
          const float disp_w = cand_disp(fw, 1.f, dw, r);
          const bool ok = centre_ok(w, disp_w, g.W);
          const float flw = floorf(disp_w);
          const float aw = disp_w - flw;
          // column of the cell's first tap: dw - 1, dw or dw + 1 (rounding of disp)
          const int dc = ok ? (int)flw - fl0 - dw : 0;
          const float a0 = dc < 0 ? cr[dw > 0 ? dw - 1 : 0] : (dc > 0 ? cr[dw + 1] : cr[dw]);
          const float a1 = dc < 0 ? cr[dw] : (dc > 0 ? cr[dw + 2] : cr[dw + 1]);
          const float b0 = dc < 0 ? cn[dw > 0 ? dw - 1 : 0] : (dc > 0 ? cn[dw + 1] : cn[dw]);
          const float b1 = dc < 0 ? cn[dw] : (dc > 0 ? cn[dw + 2] : cn[dw + 1]);
          const float top = (1.f - aw) * a0 + aw * a1;
          const float bot = (1.f - aw) * b0 + aw * b1;
          const float dv = (1.f - ah) * top + ah * bot;
          sc[dw] = ok ? fmaxf(dv, -INFINITY) : -INFINITY;  // NaN scores as invalid
        }
      }
    }
  }
  const int nreal = p1_row_cells<WSF>(g, ty, tx);
#pragma unroll
  for (int dw = 0; dw < WSM; ++dw) sc[dw] = dw < nreal ? sc[dw] : no_cell();
}

// ---- scores to the workspace (k > 32) ----

__global__ void __launch_bounds__(p1::NT, p1::WPE) search_p1_scores_kernel(const float* __restrict__ q,
                                                               const float* __restrict__ k,
                                                               const float* __restrict__ flows, Geo g, int tiles_x,
                                                               float* __restrict__ scores, int pitch) {
  using namespace p1;
  __shared__ P1Smem sm;
  const int tid = threadIdx.x, j = tid / NR, dh = tid % NR;
  const int dt = (int)blockIdx.z - g.wt;
  const int img = (int)blockIdx.y;  // (b, hd, t)
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  const int t2 = t + dt;
  if (t2 < 0 || t2 >= g.T) return;  // whole workgroup: frame outside the clip
  const int ty = (int)blockIdx.x / tiles_x, tx = (int)blockIdx.x % tiles_x;
  float sc[WSM];
  p1_frame_scores<0>(sm, q, k, flows, g, b, hd, t, dt, ty, tx, sc);
  // The scores of the tile's queries for this frame go through LDS (the
  // staging buffers are free once every thread is past the channel loop):
  // query j's ws^2 scores at sbuf[j * ws^2 ..], then copied to the workspace
  // rows with consecutive threads on consecutive addresses.
  const int nc2 = g.ws * g.ws;
  float* sbuf = &sm.reg[0][0];
  __syncthreads();
  if (dh < g.ws) {
#pragma unroll
    for (int dw = 0; dw < WSM; ++dw)
      if (dw < g.ws) sbuf[j * nc2 + dh * g.ws + dw] = sc[dw];
  }
  __syncthreads();
  // copy out: one wave per query row of the tile at a time
  const int lane = tid & 63;
  for (int jj = tid >> 6; jj < NQ; jj += NT / 64) {
    const int qh = ty * TQH + jj / TQW, qw = tx * TQW + jj % TQW;
    if (qh >= g.nH || qw >= g.nW) continue;
    const long long qrow = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + qh) * g.nW + qw;
    float* srow = scores + qrow * pitch + (dt + g.wt) * nc2;
    for (int e = lane; e < nc2; e += 64) srow[e] = sbuf[jj * nc2 + e];
  }
}

// ---- fused search and top-k (k <= 32) ----
//
// One workgroup = TQH x TQW queries of one (b, head, t), looping over the frames
// of the window, the query frame first and then the nearest frames (good
// thresholds early).  The 16 threads of a query (one 16-lane DPP row) hold
// its running list of the 32 best candidates so far, 2 per lane, best first,
// as 64-bit entries (order key of the score << 32 | ~id: larger is better,
// equal scores go to the smaller id, 0 is an empty slot).  After a frame's
// scores, the cells that rank before the list's k-th entry are compacted
// into the query's 32 LDS slots, sorted with a 32-entry bitonic network and
// merged with the list.  When more than 32 cells of a frame pass, a
// threshold with between k and 32 of the frame's cells above it is found
// first by bisection over their order keys (cells at or below it have k
// better cells in the frame alone); if ties at one key prevent that, the
// cells above the tie plus the tied ones of smallest id make the frame's
// top k.  Frames outside the clip contribute invalid candidates (-inf) in
// id order, which matter only while fewer than k better entries are known.
template <int WSF>
__global__ void __launch_bounds__(p1::NT, p1::WPE) search_p1_topk_kernel(const float* __restrict__ q,
                                                             const float* __restrict__ k,
                                                             const float* __restrict__ flows, Geo g, int tiles_x,
                                                             float* __restrict__ dists, float* __restrict__ inds) {
  using namespace p1;
  __shared__ P1Smem sm;
  // a frame's selected cells per query; the odd row pitch (LS + 1 entries)
  // puts the four queries of a wave on different banks for the same slot
  __shared__ unsigned long long surv[NQ][LS + 1];

  const int tid = threadIdx.x, j = tid / NR, dh = tid % NR;
  const int img = (int)blockIdx.y;  // (b, hd, t)
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  // Consecutive workgroups land on different XCDs (8 per device): give each
  // XCD a contiguous run of tiles, whose key regions overlap in its L2.
  const int ntile = (int)gridDim.x;
  const int xcd = (int)blockIdx.x % 8, xq = ntile / 8, xrem = ntile % 8;
  const int tile = xcd * xq + min(xcd, xrem) + (int)blockIdx.x / 8;
  const int ty = tile / tiles_x, tx = tile % tiles_x;
  const int mh = ty * TQH + j / TQW, mw = tx * TQW + j % TQW;
  const bool inside = mh < g.nH && mw < g.nW;  // the same for the query's 16 lanes
  const int gb = (tid & 63) & ~15;             // the group's first lane in the wave
  const int wsk = WSF > 0 ? WSF : g.ws;  // window side (a constant when WSF > 0)
  const int ncell = wsk * wsk;
  const int k1 = g.k - 1;

  unsigned long long L0 = 0ull, L1 = 0ull;  // list slots 2 dh and 2 dh + 1
  for (int fi = 0; fi <= 2 * g.wt; ++fi) {
    const int dt = (fi & 1) ? -((fi + 1) >> 1) : (fi >> 1);  // 0, -1, +1, -2, +2, ...
    const int t2 = t + dt;
    const int cbase = (dt + g.wt) * ncell;
    float sc[WSM];
    if (t2 >= 0 && t2 < g.T) {
      p1_frame_scores<WSF>(sm, q, k, flows, g, b, hd, t, dt, ty, tx, sc);
    } else {
      const int nreal = p1_row_cells<WSF>(g, ty, tx);  // frame outside the clip: invalid cells
#pragma unroll
      for (int dw = 0; dw < WSM; ++dw) sc[dw] = dw < nreal ? -INFINITY : no_cell();
    }
    if (!inside) continue;
    // threshold: the list's k-th entry
    const unsigned long long tsel = (k1 & 1) ? L1 : L0;
    const unsigned thi = (unsigned)__shfl((int)(unsigned)(tsel >> 32), gb + (k1 >> 1));
    const unsigned tlo = (unsigned)__shfl((int)(unsigned)tsel, gb + (k1 >> 1));
    // a cell ranks before T = (thi, tlo) iff its key exceeds thi, or equals
    // it and its id is smaller; this frame's ids all lie on one side of T's
    const bool empty = thi == 0u && tlo == 0u;
    const unsigned tid_t = ~tlo;
    const bool eq_wins = tid_t >= (unsigned)(cbase + ncell);
    const unsigned thr = empty ? 0u : thi + (eq_wins ? 0u : 1u);
    // pre-filter in floats: key >= thr implies sc >= score of thr (the float
    // order only merges -0 and +0, which lets a few more cells through to
    // the exact merge); no cell passes when thr is above +inf's key
    const float thrf = empty ? -INFINITY : key_score(thr);
    // The cells passing the float test are taken: a superset of those whose
    // key reaches thr (the extra ones, -0 cells against a threshold of +0,
    // are real candidates ranking after the list's k-th entry, so they
    // cannot enter the k best); no_cell() fails every compare.
    unsigned sel = col_mask([&](int dw) { return sc[dw] >= thrf; });
    int nsel = grp_sum(__builtin_popcount(sel));
    if (nsel == 0) continue;
    auto ukey = [&](int dw) -> unsigned { return order_key(sc[dw]); };  // 0: no cell
    if (nsel > LS) {
      // More than 32 cells rank before the list's k-th entry: keep the
      // frame's best only, above a threshold with between k and 32 cells
      // over it (a cell at or below it has k better cells in the frame).
      // Bisection over the scores' values first, over their order keys
      // when the values do not separate (ties, -inf cells, huge ranges).
      bool found = false;
      float fmx = -INFINITY, fmn = INFINITY;  // over the cells above -inf (no_cell() fails both tests)
#pragma unroll
      for (int dw = 0; dw < WSM; ++dw) {
        const float v = sc[dw];
        fmx = v > fmx ? v : fmx;
        fmn = v > -INFINITY && v < fmn ? v : fmn;
      }
      fmx = __uint_as_float(order_key_inv(grp_max(order_key(fmx))));
      fmn = -__uint_as_float(order_key_inv(grp_max(order_key(-fmn))));
      float flo = thrf > fmn ? thrf : fmn, fhi = fmx;  // keep cnt(> fhi) = 0 < k
      float fth = 0.f;
      if (isfinite(flo) && isfinite(fhi)) {
        // cnt(> flo) > 32 must hold to start: below the smallest finite score
        if (!(thrf > fmn)) flo = nextafterf(fmn, -INFINITY);
        int clo = 0;
#pragma unroll
        for (int dw = 0; dw < WSM; ++dw) clo += sc[dw] > flo ? 1 : 0;
        clo = grp_sum(clo);
        if (clo > LS) {
          for (int it = 0; it < 24; ++it) {
            const float mid = flo + 0.5f * (fhi - flo);
            if (!(mid > flo && mid < fhi)) break;  // adjacent values (or overflow): no split
            int c = 0;
#pragma unroll
            for (int dw = 0; dw < WSM; ++dw) c += sc[dw] > mid ? 1 : 0;
            c = grp_sum(c);
            if (c > LS) {
              flo = mid;
            } else if (c < g.k) {
              fhi = mid;
            } else {
              fth = mid;
              found = true;
              break;
            }
          }
        }
      }
      sel = 0;
      if (found) {
        sel = col_mask([&](int dw) { return sc[dw] > fth; });
      } else {
        // order keys: cnt(> lo) > 32 and cnt(> hi) < k
        unsigned lo = 0u, hi = 0u;
#pragma unroll
        for (int dw = 0; dw < WSM; ++dw) hi = max(hi, ukey(dw));
        hi = grp_max(hi);
        bool kfound = false;
        while (hi - lo > 1u) {
          const unsigned mid = lo + ((hi - lo) >> 1);
          int c = 0;
#pragma unroll
          for (int dw = 0; dw < WSM; ++dw) c += ukey(dw) > mid ? 1 : 0;
          c = grp_sum(c);
          if (c > LS) {
            lo = mid;
          } else if (c < g.k) {
            hi = mid;
          } else {
            lo = mid;
            kfound = true;
            break;
          }
        }
        if (kfound) {
          sel = col_mask([&](int dw) { return ukey(dw) > lo; });
        } else {
          // every key above lo equals hi: the cells above hi plus the tied
          // ones of smallest id (lane order, then column order) make k
          sel = col_mask([&](int dw) { return ukey(dw) > hi; });
          unsigned eq = col_mask([&](int dw) { return ukey(dw) == hi; });
          const int need = g.k - grp_sum(__builtin_popcount(sel));
          int take = need - grp_excl_scan(__builtin_popcount(eq));
          take = min(max(take, 0), __builtin_popcount(eq));
          for (int i = 0; i < take; ++i) {
            const unsigned lowbit = eq & (0u - eq);
            sel |= lowbit;
            eq ^= lowbit;
          }
        }
      }
      nsel = grp_sum(__builtin_popcount(sel));
    }
    if (nsel == 0) continue;
    // compaction into the query's slots (at most 32), id order
    int off = grp_excl_scan(__builtin_popcount(sel));
    const int ntot = min(nsel, LS);
    const unsigned idb = (unsigned)(cbase + dh * wsk);
#pragma unroll
    for (int dw = 0; dw < WSM; ++dw) {
      if ((sel >> dw) & 1u) {
        if (off < LS) surv[j][off] = ((unsigned long long)ukey(dw) << 32) | (unsigned)~(idb + (unsigned)dw);
        ++off;
      }
    }
    wave_lds_sync();
    // One choice for the whole wave: its groups would otherwise run both
    // paths one after the other.  The sort path takes any count up to 32.
    if (__builtin_amdgcn_ballot_w64(ntot > kInsertMax) == 0) {
      // few cells: insert them one at a time (the entries above a cell are
      // a prefix of the sorted list; the ones after it move down one slot)
      for (int i = 0; i < ntot; ++i) {
        const unsigned long long e = surv[j][i];
        const bool gt0 = L0 > e, gt1 = L1 > e;
        const unsigned long long p1v = prev_lane64(L1);  // slot 2 dh - 1
        const bool pgt1 = prev_lane_flag(gt1);            // lane 0: no slot before it
        const unsigned long long n0 = gt0 ? L0 : (pgt1 ? e : p1v);
        const unsigned long long n1 = gt1 ? L1 : (gt0 ? e : L0);
        L0 = n0;
        L1 = n1;
      }
      wave_lds_sync();  // read before the next frame's compaction writes
    } else {
      unsigned long long s0 = 2 * dh < ntot ? surv[j][2 * dh] : 0ull;
      unsigned long long s1 = 2 * dh + 1 < ntot ? surv[j][2 * dh + 1] : 0ull;
      wave_lds_sync();  // read before the next frame's compaction writes
      bitonic_sort32(s0, s1, dh);
      merge_top32(L0, L1, s0, s1, dh);
    }
  }
  if (!inside) return;
  // write the k best: list slots 2 dh, 2 dh + 1
  const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
  const int h = mh * g.s0, w = mw * g.s0;
  const long long pix = (long long)h * g.W + w;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int slot = 2 * dh + e;
    if (slot > k1) continue;
    const unsigned long long x = e ? L1 : L0;
    // every candidate was ranked, so the k best are real candidates; the
    // clamp only keeps a placeholder id in bounds
    const int cid = min(max((int)~(unsigned)x, 0), g.ncand - 1);
    const int dw = cid % wsk, dhh = (cid / wsk) % wsk, dtt = cid / ncell - g.wt;
    float fh = 0.f, fw = 0.f;
    if (dtt != 0) {
      const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dtt, g.wt)) * 2;
      fh = flows[base * g.HW + pix];
      fw = flows[(base + 1) * g.HW + pix];
    }
    dists[row * g.k + slot] = key_score((unsigned)(x >> 32));
    float* ir = inds + (row * g.k + slot) * 3;
    ir[0] = (float)(t + dtt);
    ir[1] = cand_disp(fh, g.s1, dhh, g.r);
    ir[2] = cand_disp(fw, g.s1, dw, g.r);
  }
}

// P = 1, key stride 1, inner product, ws <= 15 (any query stride).
bool p1_supported(const Geo& g) {
  // grid limits of both kernels: tiles in x, images (b, head, t) in y,
  // frame steps in z; larger problems take another route
  const long long ntile = (long long)((g.nW + p1::TQW - 1) / p1::TQW) * ((g.nH + p1::TQH - 1) / p1::TQH);
  return g.ps == 1 && g.s1 == 1.0f && g.dist == SNLS_DIST_PROD && g.ws <= p1::WSM && g.k >= 1 &&
         (long long)(g.Ch + p1::CC) * g.HW * 4 < (1LL << 31) && ntile <= 0x7fffffffLL &&
         (long long)g.B * g.HD * g.T <= 65535 && 2 * g.wt + 1 <= 65535;
}

// The fused kernel keeps at most 32 entries per query.
bool p1_fused(const Geo& g) { return p1_supported(g) && g.k <= p1::LS; }

snls_status launch_search_p1_scores(const float* q, const float* k, const float* flows, const Geo& g, float* scores,
                                    int pitch, hipStream_t s) {
  const int tiles_x = (g.nW + p1::TQW - 1) / p1::TQW, tiles_y = (g.nH + p1::TQH - 1) / p1::TQH;
  const long long ntile = (long long)tiles_x * tiles_y;
  if (ntile == 0 || g.rows == 0) return SNLS_OK;
  if (ntile > 0x7fffffffLL || (long long)g.B * g.HD * g.T > 65535 || 2 * g.wt + 1 > 65535) return SNLS_ERR_UNSUPPORTED;
  dim3 grid((unsigned)ntile, (unsigned)(g.B * g.HD * g.T), (unsigned)(2 * g.wt + 1));
  hipLaunchKernelGGL(search_p1_scores_kernel, grid, dim3(p1::NT), 0, s, q, k, flows, g, tiles_x, scores, pitch);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_search_p1_topk(const float* q, const float* k, const float* flows, const Geo& g, float* dists,
                                  float* inds, hipStream_t s) {
  const int tiles_x = (g.nW + p1::TQW - 1) / p1::TQW, tiles_y = (g.nH + p1::TQH - 1) / p1::TQH;
  const long long ntile = (long long)tiles_x * tiles_y;
  if (ntile == 0 || g.rows == 0) return SNLS_OK;
  if (ntile > 0x7fffffffLL || (long long)g.B * g.HD * g.T > 65535) return SNLS_ERR_UNSUPPORTED;
  dim3 grid((unsigned)ntile, (unsigned)(g.B * g.HD * g.T));
  // 15 x 15 and 9 x 9 windows get their own instances (window side and
  // radius as immediates)
  if (g.ws == p1::WSM)
    hipLaunchKernelGGL(search_p1_topk_kernel<p1::WSM>, grid, dim3(p1::NT), 0, s, q, k, flows, g, tiles_x, dists, inds);
  else if (g.ws == 9)
    hipLaunchKernelGGL(search_p1_topk_kernel<9>, grid, dim3(p1::NT), 0, s, q, k, flows, g, tiles_x, dists, inds);
  else
    hipLaunchKernelGGL(search_p1_topk_kernel<0>, grid, dim3(p1::NT), 0, s, q, k, flows, g, tiles_x, dists, inds);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

// Patch-similarity scores of the tiled route on the matrix cores (P = 7,
// S_Q = 1, 64 channels per head, windows up to 9).
//
// The tiled route scores a query's window cell from box sums B_D(j) =
// sum over the patch of pixel correlations c_D(x) = <q(x), K(x + D)> at
// integer shifts D (Sec. 3.2's patch similarity with bilinear key reads,
// regrouped: the 4-tap combination of the box sums is exact).  The pixel
// correlations of one halo row y against one key row are all the products
// of two 64-channel vectors over 16 halo columns and 32 or 48 key columns:
// a dense contraction over the channels, which this kernel runs as
// v_mfma_f32_16x16x4f32 products (fp32 operands and accumulation; 4
// channels per instruction).  The correlations a window needs lie on a band
// (key column = halo column + shift column) of those products; the band is
// cut out and box-summed on the vector units.
//
// A workgroup takes a 10 x 10 query tile (16 x 16 halo) of one query frame
// and loops over the frames of its window.  Wave y (16 waves) is halo row
// y: its MFMA A operand -- q at the 16 halo columns of row y for all 64
// channels -- stays in 16 registers for the whole workgroup.  The integer
// shifts the tile's windows cover (the union) are walked in rounds of up
// to 6 (or 4) shift rows; per round the key rows those shifts reach are
// staged through LDS 8 channels at a time (double-buffered), and wave y
// accumulates for every shift row i of the round the 16 x 16*NB products
// with key row y + i.  The band of each product tile is written to the
// wave's scratch rows as [halo column][shift column], where a column sum
// over 7 halo columns is the horizontal box; the 7-row vertical box is then
// summed across the waves from LDS and stored into each query's window
// table (integer shifts floor(disp_0) .. floor(disp_last) + 1), from which
// every window cell takes its 4-tap score as on the vector-unit kernel.
// All sums run in a fixed order: results are bit-identical between runs.
#include "snls_internal.h"

namespace snls {

namespace tmf {
constexpr int TQ = 10;               // query rows and columns of a tile
constexpr int PS = 7, LO = -3;       // patch side and first offset
constexpr int HR = TQ + PS - 1;      // halo rows: one wave each
constexpr int HC = TQ + PS - 1;      // halo columns: the MFMA's 16 rows
constexpr int NTHREADS = 64 * HR;
constexpr int CH = 64;               // channels per head
constexpr int NSTEP = CH / 4;        // MFMA steps of 4 channels
constexpr int CC = 8;                // channels per staging chunk
constexpr int NCHUNK = CH / CC;
constexpr int QN = TQ * TQ;
constexpr int WSM = 9;               // largest window side
constexpr int WP = WSM + 2, WIN = WP * WP;  // window table pitch and size
constexpr int UWMAX = 25;            // shift columns (15 + UW key columns in 2 or 3 blocks of 16)
constexpr int POOL = 28160;          // floats: staging, or scratch + box-sum rows
static_assert(HC == 16, "the halo columns are the 16 rows of the MFMA tile");
}  // namespace tmf

struct SmemMF {
  float pool[tmf::POOL];        // staging buffers, then the round's scratch and horizontal box sums
  float bw[tmf::QN * tmf::WIN];  // per-query window of box sums
  int qlo_h[tmf::QN], qlo_w[tmf::QN];  // smallest integer shift of the query's window (table origin)
  float qf_h[tmf::QN], qf_w[tmf::QN];  // the offset itself
  int uni[4];                   // min N_h, max N_h, min N_w, max N_w
};

typedef float mf_v4 __attribute__((ext_vector_type(4)));

// Box of 7 as power-of-two boxes: (v0 + v1) + (v2 + v3) + (v4 + v5) + v6.
SNLS_DEV float box7(float v0, float v1, float v2, float v3, float v4, float v5, float v6) {
  const float b20 = v0 + v1, b22 = v2 + v3, b24 = v4 + v5;
  return (b20 + b22) + b24 + v6;
}

// Layout constants of the two key-column widths: NB = 2 blocks of 16 key
// columns (up to 17 shift columns), NB = 3 (up to 25).
template <int NB>
struct MfLayout {
  static constexpr int RMAX = NB == 2 ? 6 : 4;   // shift rows per round (accumulators: RMAX x NB x 4)
  static constexpr int KC = 16 * NB;             // key columns staged per row
  static constexpr int SP = NB == 2 ? 17 : 25;   // shift columns of the box-sum rows
  // scratch row pitch of a product tile ([halo column][key column], key
  // columns below 15 + SP): 4 XP = 16 or 48 mod 64, so the 4 row groups of
  // a tile's store land on disjoint banks
  static constexpr int XP = NB == 2 ? 36 : 44;
  static constexpr int KROWS = tmf::HR - 1 + RMAX;   // key rows of a round at most
  // channel plane of a staged chunk: = 16 mod 64 floats, so the 4 channels
  // of an MFMA step (lanes 16 apart) sit 16 banks apart
  static constexpr int PLANE = KROWS * KC + ((16 - (KROWS * KC) % 64 + 64) % 64);
};

// One frame's correlation rounds, filling the window tables.
template <int NB>
SNLS_DEV void mf_frame(SmemMF& sm, __amdgpu_buffer_rsrc_t q_rs, unsigned qoff, __amdgpu_buffer_rsrc_t k_rs,
                       const Geo& g, int Y0, int X0, int dmin_h, int dmin_w, int UH, int UW, int tid, int wave) {
  using namespace tmf;
  using L = MfLayout<NB>;
  constexpr int RMAX = L::RMAX, KC = L::KC, SP = L::SP, PLANE = L::PLANE;
  constexpr int NC4 = KC / 4;  // 4-column staging items per row
  static_assert(2 * CC * PLANE <= POOL, "staging buffers");
  static_assert(HR * HC * L::XP + RMAX * HR * TQ * SP <= POOL, "scratch and box-sum rows");
  static_assert(15 + SP <= L::XP, "scratch columns");
  static_assert(CC * PLANE <= 8192, "LDS index field of the staging items");
  constexpr unsigned OOB = 0x80000000u;
  const int lane = tid & 63, jl = lane & 15, kq = lane >> 4;
  const int nround = (UH + RMAX - 1) / RMAX;
  const int rbase = UH / nround, rext = UH - rbase * nround;
  const int HWi = (int)g.HW;
  int i0 = 0;
  for (int rd = 0; rd < nround; ++rd) {
    const int R = rbase + (rd < rext ? 1 : 0);
    const int krows = HR - 1 + R;  // key rows y + i of the round, y < 16, i < R
    const int nitem = CC * krows * NC4;
    // Staging items: 4 consecutive key columns of one row and channel, one
    // 16-byte buffer load each (start column clamped into the frame, values
    // realigned and columns outside the frame zeroed in registers; rows
    // outside the frame and channels past the head read 0 through an
    // out-of-range offset).
    unsigned it_voff[2];
    int it_pack[2];  // LDS index | (shift + 3) << 13 | column mask << 16 | channel << 20 | on << 24
#pragma unroll
    for (int n = 0; n < 2; ++n) {
      const int e = tid + NTHREADS * n;
      it_voff[n] = OOB;
      it_pack[n] = 0;
      if (e < nitem) {
        const int c = e / (krows * NC4), rem = e - c * (krows * NC4);
        const int row = rem / NC4, c4 = rem - row * NC4;
        const int gy = Y0 + dmin_h + i0 + row;
        const int gx = X0 + dmin_w + 4 * c4;
        const int gxl = min(max(gx, 0), g.W - 4);
        int mask = 0;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) mask |= (gx + q4 >= 0 && gx + q4 < g.W) ? (1 << q4) : 0;
        if (gy >= 0 && gy < g.H && mask) it_voff[n] = (unsigned)((gy * g.W + gxl) * 4);
        const int ldsi = c * PLANE + row * KC + 4 * c4;
        it_pack[n] = ldsi | ((gx - gxl + 3) << 13) | (mask << 16) | (c << 20) | (1 << 24);
      }
    }
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 stg[2];
    // A operand of a chunk (2 steps): lane (kq, j) takes q at channel c0 +
    // 4 s + kq, halo row `wave`, halo column j; loaded with the chunk's K items
    float anext[CC / 4], acur[CC / 4];
    auto load_items = [&](int c0) {
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        const int c = (it_pack[n] >> 20) & 7;
        const unsigned off =
            (it_voff[n] != OOB && c0 + c < g.Ch) ? it_voff[n] + (unsigned)((c0 + c) * HWi * 4) : OOB;
        stg[n] = __builtin_amdgcn_raw_buffer_load_b128(k_rs, off, 0, 0);
      }
#pragma unroll
      for (int s = 0; s < CC / 4; ++s)
        anext[s] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(q_rs, qoff != OOB ? qoff + (unsigned)((c0 + 4 * s) * HWi * 4) : OOB, 0, 0));
    };
    auto store_items = [&](int bsel) {
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        const int pk = it_pack[n];
        if (pk & (1 << 24)) {
          if (((pk >> 13) & 127) != (3 | (15 << 3))) {  // not an aligned item with all columns inside
            int pkb = pk;
            asm volatile("" : "+v"(pkb));
            const int sh = ((pkb >> 13) & 7) - 3, mask = (pkb >> 16) & 15;
            const unsigned v0 = stg[n].x, v1 = stg[n].y, v2 = stg[n].z, v3 = stg[n].w;
            unsigned o[4];
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
              const int src = q4 + sh;
              const unsigned val = src <= 0 ? v0 : (src == 1 ? v1 : (src == 2 ? v2 : v3));
              o[q4] = (mask >> q4) & 1 ? val : 0u;
            }
            stg[n] = u32x4{o[0], o[1], o[2], o[3]};
          }
          float* dst = &sm.pool[bsel * CC * PLANE + (pk & 8191)];
          *reinterpret_cast<u32x4*>(dst) = stg[n];
        }
      }
    };

    mf_v4 acc[RMAX][NB];
#pragma unroll
    for (int i = 0; i < RMAX; ++i)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[i][nb] = mf_v4{0.f, 0.f, 0.f, 0.f};

    __syncthreads();  // the pool is free (previous round or frame)
    load_items(0);
    store_items(0);
#pragma unroll
    for (int cc = 0; cc < NCHUNK; ++cc) {
      const int bsel = cc & 1;
#pragma unroll
      for (int s = 0; s < CC / 4; ++s) acur[s] = anext[s];
      __syncthreads();  // chunk cc is in buffer bsel; the other buffer is no longer read
      if (cc + 1 < NCHUNK) load_items((cc + 1) * CC);  // in flight during this chunk's products
      // lane (kq, jl) supplies key column 16 nb + jl, channel 4 s + kq of key row wave + i
      const float* kcol = &sm.pool[bsel * CC * PLANE + kq * PLANE + wave * KC + jl];
#pragma unroll
      for (int s = 0; s < CC / 4; ++s) {
        const float a = acur[s];
        // all RMAX tiles, also past the round's R rows (stale rows of the
        // buffer, never extracted): no branch between the loads and products
#pragma unroll
        for (int i = 0; i < RMAX; ++i)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const float bv = kcol[4 * s * PLANE + i * KC + nb * 16];
            acc[i][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv, acc[i][nb], 0, 0, 0);
          }
      }
      if (cc + 1 < NCHUNK) store_items(bsel ^ 1);
    }
    __syncthreads();  // the staging buffers are no longer read

    // Band of each tile: D[x][c] (halo column x, key column c) goes to the
    // wave's scratch rows; the horizontal box of query column x0 at shift
    // column e is then the sum of D[x][x + e] over x = x0 .. x0 + 6, taken
    // by lane (e, half) for x0 = 5 half .. 5 half + 4 into the round's
    // box-sum rows [i][halo row][x0][e].
    constexpr int XP = L::XP;
    float* scr = &sm.pool[wave * HC * XP];
    float* hrows = &sm.pool[HR * HC * XP];
    const int ed = lane & 31, xs = 5 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < RMAX; ++i) {
      if (i < R) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (16 * nb + 16 <= XP || jl < XP - 16 * nb) scr[(4 * kq + v) * XP + 16 * nb + jl] = acc[i][nb][v];
        if (ed < UW) {
          float sv[11];
#pragma unroll
          for (int a = 0; a < 11; ++a) sv[a] = scr[(xs + a) * (XP + 1) + ed];
          float* hp = hrows + ((i * HR + wave) * TQ + xs) * SP + ed;
#pragma unroll
          for (int t = 0; t < 5; ++t)
            hp[t * SP] = box7(sv[t], sv[t + 1], sv[t + 2], sv[t + 3], sv[t + 4], sv[t + 5], sv[t + 6]);
        }
      }
    }
    __syncthreads();  // the round's horizontal boxes are complete

    // vertical box over 7 halo rows into the window tables: thread = (query,
    // table column), looping over the round's shift rows
    for (int e2 = tid; e2 < QN * WP; e2 += NTHREADS) {
      const int jq = e2 / WP, v = e2 - (e2 / WP) * WP;
      const int ee = sm.qlo_w[jq] + v - dmin_w;  // shift column of table column v
      if (ee < 0 || ee >= UW) continue;
      const int u0r = i0 + dmin_h - sm.qlo_h[jq];  // table row of the round's first shift row
      const int jh = jq / TQ, jw = jq - (jq / TQ) * TQ;
      const float* hp = hrows + (jh * TQ + jw) * SP + ee;
      constexpr int st = TQ * SP;
      float* tb = &sm.bw[jq * WIN + v];
      for (int ir = 0; ir < R; ++ir) {
        const int u = u0r + ir;
        if (u < 0 || u >= WP) continue;
        const float* h2 = hp + ir * (HR * st);
        tb[u * WP] = box7(h2[0], h2[st], h2[2 * st], h2[3 * st], h2[4 * st], h2[5 * st], h2[6 * st]);
      }
    }
    i0 += R;
  }
}

__global__ void __launch_bounds__(tmf::NTHREADS) search_mfma_scores_kernel(const float* __restrict__ q,
                                                                          const float* __restrict__ k,
                                                                          const float* __restrict__ flows, Geo g,
                                                                          int tiles_x, float* __restrict__ scores,
                                                                          int pitch) {
  using namespace tmf;
  __shared__ SmemMF sm;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;

  // XCD-aware order: consecutive workgroups land on different XCDs (8 per
  // device), so each XCD gets a contiguous run; the query frames of one tile
  // are consecutive there (the key frames they share stay in its L2).
  const long long nwg = (long long)gridDim.x;
  const long long xcd = blockIdx.x % 8, xq = nwg / 8, xrem = nwg % 8;
  const long long wg = xcd * xq + (xcd < xrem ? xcd : xrem) + blockIdx.x / 8;
  const int nimg = g.B * g.HD * g.T;
  const int img = (int)(wg % nimg);
  const int trem = (int)(wg / nimg);
  const int ty = trem / tiles_x, tx = trem % tiles_x;
  const int t = img % g.T;
  const int hd = (img / g.T) % g.HD;
  const int b = img / (g.T * g.HD);
  const int y0 = ty * TQ, x0 = tx * TQ;  // tile origin (S_Q = 1: pixels)
  const int Y0 = y0 + LO, X0 = x0 + LO;  // halo origin
  const int ws = g.ws, r = g.r;
  constexpr unsigned OOB = 0x80000000u;

  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;
  const __amdgpu_buffer_rsrc_t q_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)qb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);
  // byte offset of this lane's A-operand pixel (halo row `wave`, column
  // lane % 16) in channel lane / 16; OOB outside the frame (reads 0)
  unsigned qoff;
  {
    const int gy = Y0 + wave, gx = X0 + (lane & 15);
    const bool in = gy >= 0 && gy < g.H && gx >= 0 && gx < g.W;
    qoff = in ? (unsigned)((((lane >> 4) * (int)g.HW) + gy * g.W + gx) * 4) : OOB;
  }

  auto fetch_flow = [&](int dtt, float& fh, float& fw) {
    fh = 0.f;
    fw = 0.f;
    const int h = y0 + tid / TQ, w = x0 + tid % TQ;
    if (dtt != 0 && tid < QN && h < g.H && w < g.W) {
      const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dtt, g.wt)) * 2;
      const long long pix = (long long)h * g.W + w;
      fh = flows[base * g.HW + pix];
      fw = flows[(base + 1) * g.HW + pix];
    }
  };
  float fh_next = 0.f, fw_next = 0.f;
  bool first = true;
  const long long rowb = (((long long)b * g.HD + hd) * g.T + t) * g.nH;

  for (int si = 0; si <= 2 * g.wt; ++si) {
    const int dt = si - g.wt;
    const int cbase = (dt + g.wt) * ws * ws;
    const int t2 = t + dt;
    if (t2 < 0 || t2 >= g.T) continue;
    const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
    const __amdgpu_buffer_rsrc_t k_rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)kb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);

    // ---- offsets of the tile's queries and the union of shifts ----
    int tidf = tid;
    asm volatile("" : "+v"(tidf));
    if (tidf < 4) sm.uni[tidf] = (tidf & 1) ? INT_MIN : INT_MAX;
    if (first) {
      fetch_flow(dt, fh_next, fw_next);
      first = false;
    }
    __syncthreads();
    {
      const int jh = tidf / TQ, jw = tidf % TQ;
      const bool inside = tidf < QN && y0 + jh < g.H && x0 + jw < g.W;
      const float fh = fh_next, fw = fw_next;
      // integer shifts of a query's window: floor(disp) .. floor(disp) + 1
      // of its first .. last cell; non-finite or absurd offsets count as 0
      // here (their candidates fail the exact validity test below)
      const float fh_u = fabsf(fh) < kFarDisp ? fh : 0.f, fw_u = fabsf(fw) < kFarDisp ? fw : 0.f;
      const int lo_h = (int)floorf(cand_disp(fh_u, g.s1, 0, r));
      const int hi_h = (int)floorf(cand_disp(fh_u, g.s1, ws - 1, r)) + 1;
      const int lo_w = (int)floorf(cand_disp(fw_u, g.s1, 0, r));
      const int hi_w = (int)floorf(cand_disp(fw_u, g.s1, ws - 1, r)) + 1;
      if (tidf < QN) {
        sm.qlo_h[tidf] = lo_h;
        sm.qlo_w[tidf] = lo_w;
        sm.qf_h[tidf] = fh;
        sm.qf_w[tidf] = fw;
      }
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
    {  // next searched frame's offsets, in flight during this frame
      int sn = si + 1;
      while (sn <= 2 * g.wt && (t + sn - g.wt < 0 || t + sn - g.wt >= g.T)) ++sn;
      if (sn <= 2 * g.wt) fetch_flow(sn - g.wt, fh_next, fw_next);
    }
    __syncthreads();
    // Only shifts a valid cell can read matter: clip the union to the taps
    // of centres inside the frame (rows [-h_last, H - y0], likewise columns).
    const int h_last = min(y0 + TQ - 1, g.nH - 1);
    const int w_last = min(x0 + TQ - 1, g.nW - 1);
    const int u0 = max(__builtin_amdgcn_readfirstlane(sm.uni[0]), -h_last);
    const int u1 = min(__builtin_amdgcn_readfirstlane(sm.uni[1]), g.H - y0);
    const int u2 = max(__builtin_amdgcn_readfirstlane(sm.uni[2]), -w_last);
    const int u3 = min(__builtin_amdgcn_readfirstlane(sm.uni[3]), g.W - x0);
    const int UH = u1 - u0 + 1, UW = u3 - u2 + 1;
    const bool none = UH <= 0 || UW <= 0;  // every cell of the frame is invalid

    if (none || UW <= UWMAX) {
      if (!none) {
        if (UW <= MfLayout<2>::SP)
          mf_frame<2>(sm, q_rs, qoff, k_rs, g, Y0, X0, u0, u2, UH, UW, tid, wave);
        else
          mf_frame<3>(sm, q_rs, qoff, k_rs, g, Y0, X0, u0, u2, UH, UW, tid, wave);
      }
      __syncthreads();
      // ---- 4-tap combination and exact validity (one thread per window row) ----
      for (int e = tid; e < QN * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int mh = y0 + j / TQ, mw = x0 + j % TQ;
        if (mh >= g.nH || mw >= g.nW) continue;
        float* srow = scores + ((rowb + mh) * g.nW + mw) * pitch + cbase + dh * ws;
        const float fw = sm.qf_w[j];
        const int lw = sm.qlo_w[j];
        const float disp_h = cand_disp(sm.qf_h[j], g.s1, dh, r);
        const bool okh = !none && centre_ok(mh, disp_h, g.H);
        const float fl_h = floorf(disp_h), ah = disp_h - fl_h;
        const float* r0p = &sm.bw[j * WIN + (okh ? (int)fl_h - sm.qlo_h[j] : 0) * WP];
        const float* r1p = r0p + WP;
        for (int dw = 0; dw < ws; ++dw) {
          const float disp_w = cand_disp(fw, g.s1, dw, r);
          const bool ok = okh && centre_ok(mw, disp_w, g.W);
          const float fl_w = floorf(disp_w), aw = disp_w - fl_w;
          const int col = ok ? (int)fl_w - lw : 0;
          const float top = (1.f - aw) * r0p[col] + aw * r0p[col + 1];
          const float bot = (1.f - aw) * r1p[col] + aw * r1p[col + 1];
          const float dv = (1.f - ah) * top + ah * bot;
          srow[dw] = ok && dv == dv ? dv : -INFINITY;  // NaN scores as invalid
        }
      }
    } else {
      // union too wide for the key-column blocks: score this frame directly
      // (inner products for both distances: the top-k pass forms L2)
      Geo gp = g;
      gp.dist = SNLS_DIST_PROD;
      for (int e = tid; e < QN * ws; e += NTHREADS) {
        const int j = e / ws, dh = e % ws;
        const int mh = y0 + j / TQ, mw = x0 + j % TQ;
        if (mh >= g.nH || mw >= g.nW) continue;
        const float fh = sm.qf_h[j], fw = sm.qf_w[j];
        const float disp_h = cand_disp(fh, g.s1, dh, r);
        const bool okh = centre_ok(mh, disp_h, g.H);
        for (int dw = 0; dw < ws; ++dw) {
          const float disp_w = cand_disp(fw, g.s1, dw, r);
          float d = -INFINITY;
          if (okh && centre_ok(mw, disp_w, g.W)) d = score_candidate(q, k, gp, b, hd, t, mh, mw, t2, disp_h, disp_w);
          scores[((rowb + mh) * g.nW + mw) * pitch + cbase + dh * ws + dw] = d;
        }
      }
    }
    __syncthreads();
  }
}

bool mfma_scores_supported(const Geo& g) {
  return g.ps == tmf::PS && g.s0 == 1 && g.Ch == tmf::CH && g.ws <= tmf::WSM && g.s1 > 0.f && g.s1 <= 1.0f &&
         g.W >= 4 && (long long)g.Ch * g.HW * 4 < (1LL << 31) && (long long)g.C * g.HW * 4 < (1LL << 31);
}

snls_status launch_mfma_scores(const float* q, const float* k, const float* flows, const Geo& g, float* scores,
                               int pitch, hipStream_t s) {
  const int tiles_x = (g.nW + tmf::TQ - 1) / tmf::TQ;
  const int tiles_y = (g.nH + tmf::TQ - 1) / tmf::TQ;
  const long long nwg = (long long)tiles_x * tiles_y * g.B * g.HD * g.T;
  if (nwg == 0) return SNLS_OK;
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(search_mfma_scores_kernel, dim3((unsigned)nwg), dim3(tmf::NTHREADS), 0, s, q, k, flows, g,
                     tiles_x, scores, pitch);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

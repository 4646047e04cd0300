// search_l2.hip -- norm terms of the squared L2 distance for the tiled
// search (Sec. 3.2 patch similarity, L2 form).
//
// For a candidate at displacement disp of query (b, t, h, w) the squared L2
// distance over the query's in-frame patch pixels p and the head's channels is
//     d = sum_p |q(h+p)|^2 - 2 sum_p <q(h+p), k~(h+p+disp)> + sum_p |k~(h+p+disp)|^2 .
// The middle term is the inner-product score the tiled kernel computes; this
// file computes the two norm terms:
//   Qn(query)       = sum over in-frame patch pixels of |q|^2;
//   G(query, cell)  = sum over in-frame patch pixels p of |k~(h+p+disp_cell)|^2.
// With key stride S_K = 1 every cell of a query's window in one frame has the
// same bilinear fraction a = F - floor(F), so |k~|^2 is evaluated once per
// position of the (ws + P - 1)^2 region the window's patches cover, and G is
// a box sum of those values over the patch rows and columns that lie inside
// the frame.  (Per-cell fractions of fl32(F + d - r) can differ from a by
// rounding in the last bit; the effect on G is far below the fp32 score
// tolerance, and the positions reported come from the exact per-cell values.)
//
// |k~|^2 of a bilinear read with taps v_e and weights w_e expands into
//     sum_e w_e^2 |v_e|^2 + 2 sum_{e<e'} w_e w_e' <v_e, v_e'>,
// and the channel sums |v|^2 and <v, v'> of neighbouring key pixels do not
// depend on the query.  A first kernel computes, per key pixel (y, x) of
// every frame and head, five pair planes over the head's channels:
//   N = |k(y,x)|^2, R = <k(y,x), k(y,x+1)>, D = <k(y,x), k(y+1,x)>,
//   X = <k(y,x), k(y+1,x+1)>, A = <k(y,x+1), k(y+1,x)>
// (pixels outside the frame read 0), so each position costs ten products of
// plane values with the query's weights instead of four taps per channel.
// Every term reads only planes of the position's own four taps, so a
// non-finite key value reaches exactly the positions whose taps read it.
// A sixth plane holds |q(y,x)|^2 of the query video, so Qn is a sum of
// P^2 plane values per query.
//
// At a key stride S_K != 1 the cells of a window have fractions of their
// own, so G is formed per cell (l2_norms_cells_kernel; also for windows
// larger than the grids of l2_norms_kernel): with n = floor(disp)
// and the cell's weights, the ten terms above become ten box sums of the
// planes over the query's in-frame patch pixels, each at the offset of its
// term ((0|1, 0|1) for N, (0|1, 0) for R, (0, 0|1) for D, (0, 0) for X and
// A), each four reads of the plane's summed-area table (fp64, exact).
#include "snls_internal.h"

namespace snls {

namespace l2n {
constexpr int TY = 4, TX = 8;        // query tile
constexpr int NQ = TY * TX;          // queries per workgroup
constexpr int TPQ = 8;               // threads per query
constexpr int NT = NQ * TPQ;         // 256
constexpr int EG = 16;               // per-query grid of positions (ws + P - 1 <= 15, one spare)
constexpr int PPT = EG * EG / TPQ;   // positions per thread
constexpr int CC = 8;                // channels per staging chunk
constexpr int RH = 32, RW = 40;      // union region of the tile (rows, columns), +1 tap included
constexpr int RP = RW + 1;           // region row pitch (odd)
constexpr int WSMAX = 9;             // window side
constexpr int GRIDS = NQ * EG * EG;  // per-query |k~|^2 grids
constexpr int VSUM = NQ * WSMAX * EG;  // per-query column sums
constexpr int REGF = CC * RH * RP > GRIDS + VSUM ? CC * RH * RP : GRIDS + VSUM;
}  // namespace l2n

constexpr int NKP = 5;     // key planes N, R, D, X, A
constexpr int NPLANE = 6;  // ... and the query pixel norm |q|^2

// Pair planes of one (b, t, head): one thread per pixel.  Layout
// planes[((b*T + t)*HD + hd)*6 + m][H][W], m = N, R, D, X, A of k, |q|^2.
__global__ void __launch_bounds__(256) l2_pair_planes_kernel(const float* __restrict__ q,
                                                             const float* __restrict__ k, Geo g,
                                                             float* __restrict__ planes) {
  const long long slab = blockIdx.y;  // (b*T + t)*HD + hd
  const long long pix = (long long)blockIdx.x * 256 + threadIdx.x;
  if (pix >= g.HW) return;
  const int hd = (int)(slab % g.HD);
  const long long bt = slab / g.HD;
  const int y = (int)(pix / g.W), x = (int)(pix % g.W);
  const bool rin = x + 1 < g.W, din = y + 1 < g.H;
  const float* kb = k + (bt * g.C + (long long)hd * g.Ch) * g.HW + pix;
  const float* qb = q + (bt * g.C + (long long)hd * g.Ch) * g.HW + pix;
  float n = 0.f, r = 0.f, d = 0.f, xx = 0.f, a = 0.f, qq = 0.f;
  for (int c = 0; c < g.Ch; ++c, kb += g.HW, qb += g.HW) {
    const float qv = qb[0];
    qq = fmaf(qv, qv, qq);
    const float v00 = kb[0];
    const float v01 = rin ? kb[1] : 0.f;
    const float v10 = din ? kb[g.W] : 0.f;
    const float v11 = rin && din ? kb[g.W + 1] : 0.f;
    n = fmaf(v00, v00, n);
    r = fmaf(v00, v01, r);
    d = fmaf(v00, v10, d);
    xx = fmaf(v00, v11, xx);
    a = fmaf(v01, v10, a);
  }
  float* out = planes + slab * NPLANE * g.HW + pix;
  out[0] = n;
  out[g.HW] = r;
  out[2 * g.HW] = d;
  out[3 * g.HW] = xx;
  out[4 * g.HW] = a;
  out[5 * g.HW] = qq;
}

// One workgroup = a TY x TX tile of queries of one (b, head, t) and one
// frame step dt (grid z = dt + wt).
__global__ void __launch_bounds__(l2n::NT, 3) l2_norms_kernel(const float* __restrict__ q,
                                                          const float* __restrict__ planes,
                                                          const float* __restrict__ flows, Geo g, int tiles_x,
                                                          float* __restrict__ G, int pitch,
                                                          float* __restrict__ Qn) {
  using namespace l2n;
  __shared__ float reg[REGF];  // pair-plane region; then the per-query |k~|^2 grids and column sums
  __shared__ int ubox[4];              // union: min row, max row, min col, max col (region origins)
  __shared__ int qoy[NQ], qox[NQ];     // query's grid origin inside the region
  __shared__ int qay[NQ], qax[NQ];     // and in the frame (per-query blocks)
  __shared__ float qpart[NT];

  const int tid = threadIdx.x, jq = tid / TPQ, sub = tid % TPQ;
  const int dt = (int)blockIdx.z - g.wt;
  const int img = (int)blockIdx.y;  // (b, hd, t)
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  const int t2 = t + dt;
  if (t2 < 0 || t2 >= g.T) return;  // whole workgroup
  const int ty = (int)blockIdx.x / tiles_x, tx = (int)blockIdx.x % tiles_x;
  const int mh = ty * TY + jq / TX, mw = tx * TX + jq % TX;  // query grid position
  const bool inside = mh < g.nH && mw < g.nW;
  const int h = mh * g.s0, w = mw * g.s0;
  const int E = g.ws + g.ps - 1;  // grid side used (<= 15)

  // offset of the query's window and the integer origin of its grid
  float fh = 0.f, fw = 0.f;
  if (dt != 0 && inside) {
    const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
    const long long pix = (long long)h * g.W + w;
    fh = flows[base * g.HW + pix];
    fw = flows[(base + 1) * g.HW + pix];
  }
  // non-finite or absurd offsets: their candidates are invalid (the inner
  // product pass scores them so); any G value does
  const float fh_u = fabsf(fh) < kFarDisp ? fh : 0.f, fw_u = fabsf(fw) < kFarDisp ? fw : 0.f;
  const float flh = floorf(fh_u), flw = floorf(fw_u);
  const int oy = h + g.lo + (int)flh - g.r, ox = w + g.lo + (int)flw - g.r;  // key coords of grid (0, 0)
  if (tid < 4) ubox[tid] = (tid & 1) ? INT_MIN : INT_MAX;
  __syncthreads();
  if (sub == 0 && inside) {
    atomicMin(&ubox[0], oy);
    atomicMax(&ubox[1], oy);
    atomicMin(&ubox[2], ox);
    atomicMax(&ubox[3], ox);
  }
  __syncthreads();
  const int ry0 = ubox[0], rx0 = ubox[2];
  const int rh = ubox[1] - ry0 + E + 1, rw = ubox[3] - rx0 + E + 1;  // region extent (taps included)
  const bool staged = ubox[1] >= ubox[0] && rh <= RH && rw <= RW;  // else per-query blocks
  if (sub == 0) {
    qoy[jq] = oy - ry0;
    qox[jq] = ox - rx0;
    qay[jq] = oy;
    qax[jq] = ox;
  }
  const float ah = fh_u - flh, aw = fw_u - flw;

  const float* kb = planes + (((long long)b * g.T + t2) * g.HD + hd) * NPLANE * g.HW;
  float acc[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) acc[i] = 0.f;

  // value of pair plane m at (y, x): 0 outside the frame
  auto kval = [&](int m, int y, int x) -> float {
    return (y >= 0 && y < g.H && x >= 0 && x < g.W) ? kb[(long long)m * g.HW + (long long)y * g.W + x] : 0.f;
  };
  // the query's bilinear weights and the ten coefficients of the expansion
  const float w00 = (1.f - ah) * (1.f - aw), w01 = (1.f - ah) * aw, w10 = ah * (1.f - aw), w11 = ah * aw;
  // contribution of plane m at grid position b[0] = (y, x) (pitch: row stride)
  auto plane_term = [&](int m, const float* bp, int pitch) -> float {
    switch (m) {
      case 0:
        return w00 * w00 * bp[0] + w01 * w01 * bp[1] + w10 * w10 * bp[pitch] + w11 * w11 * bp[pitch + 1];
      case 1:
        return 2.f * w00 * w01 * bp[0] + 2.f * w10 * w11 * bp[pitch];
      case 2:
        return 2.f * w00 * w10 * bp[0] + 2.f * w01 * w11 * bp[1];
      case 3:
        return 2.f * w00 * w11 * bp[0];
      default:
        return 2.f * w01 * w10 * bp[0];
    }
  };
  // Thread sub owns grid columns sub and sub + TPQ (acc[2*zy + half] is row
  // zy of column sub + TPQ*half).
  static_assert(EG == 2 * TPQ && PPT == 2 * EG, "two grid columns per thread");
  // The tile's region of the five planes is staged at once when it fits;
  // otherwise each query's own EG x EG block, one plane at a time.
  static_assert(NKP <= CC, "the key planes fit in one chunk");
  const int xx = tid & 63;  // region staging: lane = column, waves = rows
  const int cpc = staged ? NKP : 1;
  const int bpitch = staged ? RP : EG, cstr = staged ? RH * RP : 0;
  const int qbase = staged ? qoy[jq] * RP + qox[jq] : jq * EG * EG;
  static_assert(NQ * EG * EG <= CC * RH * RP, "per-query blocks fit in the region buffer");
  for (int m0 = 0; m0 < NKP; m0 += cpc) {
    __syncthreads();  // previous chunk fully read
    if (staged) {
      // the whole chunk's loads in flight before the LDS stores
      float st[NKP][RH / (NT / 64)];
#pragma unroll
      for (int m = 0; m < NKP; ++m)
#pragma unroll
        for (int i = 0; i < RH / (NT / 64); ++i) {
          const int yy = (tid >> 6) + (NT / 64) * i;
          st[m][i] = (xx < rw && yy < rh) ? kval(m, ry0 + yy, rx0 + xx) : 0.f;
        }
#pragma unroll
      for (int m = 0; m < NKP; ++m)
#pragma unroll
        for (int i = 0; i < RH / (NT / 64); ++i) {
          const int yy = (tid >> 6) + (NT / 64) * i;
          if (xx < rw && yy < rh) reg[(m * RH + yy) * RP + xx] = st[m][i];
        }
    } else {
      for (int e = tid; e < NQ * EG * EG; e += NT) {
        const int jj = e / (EG * EG), rem = e % (EG * EG);
        reg[e] = kval(m0, qay[jj] + rem / EG, qax[jj] + rem % EG);
      }
    }
    __syncthreads();
    if (inside) {
      if (staged) {
#pragma unroll
        for (int m = 0; m < NKP; ++m) {
          const float* base = &reg[m * cstr + qbase];
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int zx = sub + TPQ * half;
            if (zx < E) {
#pragma unroll
              for (int zy = 0; zy < EG - 1; ++zy)
                if (zy < E) acc[2 * zy + half] += plane_term(m, base + zy * bpitch + zx, bpitch);
            }
          }
        }
      } else {
        const float* base = &reg[qbase];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int zx = sub + TPQ * half;
          if (zx < E) {
#pragma unroll
            for (int zy = 0; zy < EG - 1; ++zy)
              if (zy < E) acc[2 * zy + half] += plane_term(m0, base + zy * bpitch + zx, bpitch);
          }
        }
      }
    }
  }
  // the query's grid of |k~|^2 into LDS (over the region buffer)
  __syncthreads();
  float* gq = &reg[jq * EG * EG];
#pragma unroll
  for (int i = 0; i < PPT; ++i) gq[(i >> 1) * EG + sub + TPQ * (i & 1)] = acc[i];  // zero outside the frame
  __syncthreads();
  // patch rows and columns whose query pixel is inside the frame
  const int ip0 = max(0, -h - g.lo), ip1 = min(g.ps - 1, g.H - 1 - h - g.lo);
  const int jp0 = max(0, -w - g.lo), jp1 = min(g.ps - 1, g.W - 1 - w - g.lo);
  // column sums over the valid patch rows, for window row dh and grid column x
  float* vs = &reg[GRIDS + jq * WSMAX * EG];
  if (inside) {
    for (int e = sub; e < g.ws * E; e += TPQ) {
      const int dh = e / E, x = e % E;
      float sacc = 0.f;
      for (int ip = ip0; ip <= ip1; ++ip) sacc += gq[(ip + dh) * EG + x];
      vs[dh * EG + x] = sacc;
    }
  }
  __syncthreads();
  if (!inside) return;  // no barrier follows
  const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
  float* grow = G + row * pitch + (dt + g.wt) * g.ws * g.ws;
  for (int e = sub; e < g.ws * g.ws; e += TPQ) {
    const int dh = e / g.ws, dw = e % g.ws;
    float sacc = 0.f;
    for (int jp = jp0; jp <= jp1; ++jp) sacc += vs[dh * EG + jp + dw];
    grow[e] = sacc;
  }
  if (dt == 0) {
    // |q|^2 over the in-frame patch pixels (once per query: the query
    // frame's workgroup), from the query pixel-norm plane
    const float* qpl = planes + ((((long long)b * g.T + t) * g.HD + hd) * NPLANE + NKP) * g.HW;
    float sq = 0.f;
    const int pw_n = jp1 - jp0 + 1, npix = (ip1 - ip0 + 1) * pw_n;
    for (int e = sub; e < npix; e += TPQ) {
      const int y = h + g.lo + ip0 + e / pw_n, x = w + g.lo + jp0 + e % pw_n;
      sq += qpl[(long long)y * g.W + x];
    }
    qpart[tid] = sq;
    // the query's TPQ threads are lanes of one wave: order its LDS accesses
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (sub == 0) {
      float tot = 0.f;
      for (int i = 0; i < TPQ; ++i) tot += qpart[tid + i];
      Qn[row] = tot;
    }
  }
}

// Summed-area tables of the five key pair planes, in fp64 (exact box sums
// at any offset): S[y][x] = sum of the plane over rows < y, columns < x,
// (H + 1) x (W + 1) per (b, t, head, plane).  First the prefix along each
// row (one thread per row), then down each column (one thread per column).
__global__ void __launch_bounds__(256) l2_sat_rows_kernel(const float* __restrict__ planes, Geo g,
                                                          double* __restrict__ sat) {
  const int y = blockIdx.x * 256 + threadIdx.x;
  if (y >= g.H) return;
  const long long sp = blockIdx.y;  // slab * NKP + plane
  const long long slab = sp / NKP, m = sp - slab * NKP;
  const float* src = planes + (slab * NPLANE + m) * g.HW + (long long)y * g.W;
  double* dst = sat + (sp * (g.H + 1) + y + 1) * (long long)(g.W + 1);
  double acc = 0.0;
  dst[0] = 0.0;
  for (int x = 0; x < g.W; ++x) {
    acc += (double)src[x];
    dst[x + 1] = acc;
  }
}

__global__ void __launch_bounds__(256) l2_sat_cols_kernel(Geo g, double* __restrict__ sat) {
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x > g.W) return;
  const long long sp = blockIdx.y;
  double* col = sat + sp * (g.H + 1) * (long long)(g.W + 1) + x;
  const long long W1 = g.W + 1;
  double acc = 0.0;
  col[0] = 0.0;
  for (int y = 1; y <= g.H; ++y) {
    acc += col[y * W1];
    col[y * W1] = acc;
  }
}

// Sum of one plane over rows r0..r1, columns c0..c1 (inclusive), pixels
// outside the frame counting 0: four reads of its summed-area table.
SNLS_DEV double sat_rect(const double* __restrict__ S, const Geo& g, int r0, int r1, int c0, int c1) {
  r0 = max(r0, 0);
  r1 = min(r1, g.H - 1);
  c0 = max(c0, 0);
  c1 = min(c1, g.W - 1);
  if (r0 > r1 || c0 > c1) return 0.0;
  const long long W1 = g.W + 1;
  return (S[(r1 + 1) * W1 + c1 + 1] - S[r0 * W1 + c1 + 1]) - (S[(r1 + 1) * W1 + c0] - S[r0 * W1 + c0]);
}

// G of every cell, cell by cell (a key stride S_K != 1 gives the cells of a
// window fractions of their own; windows above 9 exceed the per-query grids
// of l2_norms_kernel): one thread per (query, cell) of one frame step (grid
// y = dt + wt), consecutive threads the cells of a query; Qn by the first
// cell's thread of the query frame.  Each of the ten terms is a box sum of
// one pair plane over the query's in-frame patch pixels at the term's tap
// offset: a rectangle of the plane's summed-area table.
__global__ void __launch_bounds__(256) l2_norms_cells_kernel(const float* __restrict__ planes,
                                                             const double* __restrict__ sat,
                                                             const float* __restrict__ flows, Geo g,
                                                             float* __restrict__ G, int pitch,
                                                             float* __restrict__ Qn) {
  const int ncf = g.ws * g.ws;  // cells per frame step
  const long long e = (long long)blockIdx.x * 256 + threadIdx.x;
  if (e >= g.rows * ncf) return;
  const long long row = e / ncf;
  const int cell = (int)(e - row * ncf);
  const int dt = (int)blockIdx.y - g.wt;
  const int mw = (int)(row % g.nW);
  long long rr = row / g.nW;
  const int mh = (int)(rr % g.nH);
  rr /= g.nH;
  const int t = (int)(rr % g.T);
  rr /= g.T;
  const int hd = (int)(rr % g.HD);
  const int b = (int)(rr / g.HD);
  const int t2 = t + dt;
  const int h = mh * g.s0, w = mw * g.s0;
  // patch rows and columns whose query pixel is inside the frame
  const int ip0 = max(0, -h - g.lo), ip1 = min(g.ps - 1, g.H - 1 - h - g.lo);
  const int jp0 = max(0, -w - g.lo), jp1 = min(g.ps - 1, g.W - 1 - w - g.lo);
  if (dt == 0 && cell == 0) {
    const float* qpl = planes + ((((long long)b * g.T + t) * g.HD + hd) * NPLANE + NKP) * g.HW;
    float sq = 0.f;
    for (int ip = ip0; ip <= ip1; ++ip)
      for (int jp = jp0; jp <= jp1; ++jp) sq += qpl[(long long)(h + g.lo + ip) * g.W + w + g.lo + jp];
    Qn[row] = sq;
  }
  if (t2 < 0 || t2 >= g.T) return;  // candidates of frames outside the clip rank as invalid
  float fh = 0.f, fw = 0.f;
  if (dt != 0) {
    const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
    const long long pix = (long long)h * g.W + w;
    fh = flows[base * g.HW + pix];
    fw = flows[(base + 1) * g.HW + pix];
  }
  float gsum = 0.f;
  // non-finite or absurd offsets: their candidates are invalid (the inner
  // product pass scores them so); any G value does
  if (fabsf(fh) < kFarDisp && fabsf(fw) < kFarDisp) {
    const int dh = cell / g.ws, dw = cell - (cell / g.ws) * g.ws;
    const float disp_h = cand_disp(fh, g.s1, dh, g.r), disp_w = cand_disp(fw, g.s1, dw, g.r);
    const float fly = floorf(disp_h), flx = floorf(disp_w);
    const float ay = disp_h - fly, ax = disp_w - flx;
    const int y0 = h + g.lo + (int)fly, x0 = w + g.lo + (int)flx;  // tap (0, 0) of patch pixel (0, 0)
    const long long pst = (long long)(g.H + 1) * (g.W + 1);
    const double* S = sat + (((long long)b * g.T + t2) * g.HD + hd) * NKP * pst;
    const double* SN = S, *SR = S + pst, *SD = S + 2 * pst, *SX = S + 3 * pst, *SA = S + 4 * pst;
    // patch rows a in [ip0, ip1] read rows y0 + a at row offset 0 and
    // y0 + a + 1 at offset 1 (likewise columns)
    const int ra0 = y0 + ip0, ra1 = y0 + ip1, ca0 = x0 + jp0, ca1 = x0 + jp1;
    const double n00 = sat_rect(SN, g, ra0, ra1, ca0, ca1), n01 = sat_rect(SN, g, ra0, ra1, ca0 + 1, ca1 + 1);
    const double n10 = sat_rect(SN, g, ra0 + 1, ra1 + 1, ca0, ca1);
    const double n11 = sat_rect(SN, g, ra0 + 1, ra1 + 1, ca0 + 1, ca1 + 1);
    const double r0 = sat_rect(SR, g, ra0, ra1, ca0, ca1), r1 = sat_rect(SR, g, ra0 + 1, ra1 + 1, ca0, ca1);
    const double d0 = sat_rect(SD, g, ra0, ra1, ca0, ca1), d1 = sat_rect(SD, g, ra0, ra1, ca0 + 1, ca1 + 1);
    const double xs = sat_rect(SX, g, ra0, ra1, ca0, ca1), as = sat_rect(SA, g, ra0, ra1, ca0, ca1);
    const double w00 = (1.0 - ay) * (1.0 - ax), w01 = (1.0 - ay) * ax, w10 = ay * (1.0 - ax), w11 = ay * ax;
    gsum = (float)(w00 * w00 * n00 + w01 * w01 * n01 + w10 * w10 * n10 + w11 * w11 * n11 + 2.0 * w00 * w01 * r0 +
                   2.0 * w10 * w11 * r1 + 2.0 * w00 * w10 * d0 + 2.0 * w01 * w11 * d1 + 2.0 * w00 * w11 * xs +
                   2.0 * w01 * w10 * as);
  }
  G[row * pitch + (dt + g.wt) * ncf + cell] = gsum;
}

static bool l2_cells(const Geo& g) { return g.s1 != 1.0f || g.ws > l2n::WSMAX; }
static size_t l2_plane_only_bytes(const Geo& g) {
  return ((size_t)NPLANE * g.B * g.T * g.HD * (size_t)g.HW * sizeof(float) + 255) & ~(size_t)255;
}
// pair planes, then (cell by cell only) their summed-area tables in fp64
size_t l2_planes_bytes(const Geo& g) {
  size_t b = l2_plane_only_bytes(g);
  if (l2_cells(g)) b += ((size_t)NKP * g.B * g.T * g.HD * (size_t)(g.H + 1) * (g.W + 1) * sizeof(double) + 255) & ~(size_t)255;
  return b;
}

snls_status launch_l2_norms(const float* q, const float* k, const float* flows, const Geo& g, float* G, int pitch,
                            float* Qn, float* planes, hipStream_t s) {
  const int tiles_x = (g.nW + l2n::TX - 1) / l2n::TX, tiles_y = (g.nH + l2n::TY - 1) / l2n::TY;
  const long long ntile = (long long)tiles_x * tiles_y;
  if (ntile == 0 || g.rows == 0) return SNLS_OK;
  if (ntile > 0x7fffffffLL || (long long)g.B * g.HD * g.T > 65535 || 2 * g.wt + 1 > 65535) return SNLS_ERR_UNSUPPORTED;
  const dim3 pgrid((unsigned)((g.HW + 255) / 256), (unsigned)(g.B * g.T * g.HD));
  hipLaunchKernelGGL(l2_pair_planes_kernel, pgrid, dim3(256), 0, s, q, k, g, planes);
  if (l2_cells(g)) {
    // per-cell fractions, or windows past the grids below: G cell by cell
    // from the planes' summed-area tables
    const long long nth = g.rows * (long long)(g.ws * g.ws);
    const long long nblk = (nth + 255) / 256;
    const long long nsp = (long long)g.B * g.T * g.HD * NKP;
    if (nblk > 0x7fffffffLL || nsp > 65535) return SNLS_ERR_UNSUPPORTED;
    double* sat = reinterpret_cast<double*>(reinterpret_cast<char*>(planes) + l2_plane_only_bytes(g));
    hipLaunchKernelGGL(l2_sat_rows_kernel, dim3((unsigned)((g.H + 255) / 256), (unsigned)nsp), dim3(256), 0, s, planes,
                       g, sat);
    hipLaunchKernelGGL(l2_sat_cols_kernel, dim3((unsigned)((g.W + 1 + 255) / 256), (unsigned)nsp), dim3(256), 0, s, g,
                       sat);
    dim3 cgrid((unsigned)nblk, (unsigned)(2 * g.wt + 1));
    hipLaunchKernelGGL(l2_norms_cells_kernel, cgrid, dim3(256), 0, s, planes, sat, flows, g, G, pitch, Qn);
    return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
  }
  dim3 grid((unsigned)ntile, (unsigned)(g.B * g.HD * g.T), (unsigned)(2 * g.wt + 1));
  hipLaunchKernelGGL(l2_norms_kernel, grid, dim3(l2n::NT), 0, s, q, planes, flows, g, tiles_x, G, pitch, Qn);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

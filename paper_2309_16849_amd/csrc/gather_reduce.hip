// gather_reduce.hip -- the code example's aggregation path (App. B): the
// gather with the caller's weights that keeps the k neighbours apart,
//     S[b,hd,l,t,f,y,x] = 1/cnt(y,x) * sum over the query patches covering
//                         (y,x) of w_l * v~_l(f, (y,x) + disp_l)
// (Sec. 3.2 "Aggregation" restricted to the l-th neighbours), and the
// reduction over the neighbours that follows it, a convolution with a
// (Cout, C, k, 1, 1) kernel at stride (k, 1, 1):
//     out[b,t,o,y,x] = sum over hd, f, l of proj[o, hd*F' + f, l] * S[b,hd,l,t,f,y,x].
//
// The reduction is a dense contraction per pixel (k * C inputs, Cout
// outputs), done on the matrix cores: per 8 x 8 pixel tile and per (head,
// neighbour rank), a (64 pixels x F') by (F' x Cout) product with
// v_mfma_f32_16x16x4f32, fp32 in and out; each of the 4 waves owns 16 pixels
// and all Cout columns.  The fused entry point gathers S for the tile into
// LDS and multiplies it straight away, so the k-fold stacked tensor never
// goes to memory.
//
// Gather: per (head, rank), the tile's covering queries' records (weight,
// frame, integer offset, fractions) are staged in LDS; thread (pixel, channel
// quarter) walks the queries covering its pixel and reads the four taps of
// each from a channels-last copy of v (4 consecutive channels per 16-byte
// load).  A neighbour whose weight is 0, whose frame is not an integer in
// [0, T) or whose offset is not finite (magnitude kFarDisp or more) adds
// nothing.
#include "snls_internal.h"

namespace snls {

namespace gr {
constexpr int TS = 8;             // 8 x 8 pixel tile
constexpr int NP = TS * TS;       // pixels per tile
constexpr int NT = 256;           // threads: 64 pixels x 4 channel quarters
constexpr int FMAX = 64;          // channels per head
constexpr int CPT = FMAX / 4;     // channels per thread (4 groups of 4)
constexpr int RMAX = 256;         // covering queries of a tile
constexpr int OMAX = 128;         // output channels (8 blocks of 16)
constexpr int SP = NP + 4;        // LDS pitch of a channel row of S (pixels)
}  // namespace gr

// Covering-query range of the tile along one axis: grid positions m with
// m*S in [y0 - lo - P + 1, y0 + TS - 1 - lo], clipped to [0, n).
SNLS_DEV void cover_range(int y0, int S, int n, int lo, int P, int* m0, int* m1) {
  const int a = y0 - lo - P + 1, bnd = y0 + gr::TS - 1 - lo;
  *m0 = a <= 0 ? 0 : (a + S - 1) / S;
  *m1 = bnd < 0 ? -1 : min(bnd / S, n - 1);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GrRecord {
  float w, ay, ax;
  int tf, ny, nx;
};

struct GrSmem {
  GrRecord rec[gr::RMAX];
  alignas(16) float S[gr::FMAX][gr::SP];           // gathered channels x pixels
  alignas(16) float Pm[gr::OMAX][gr::FMAX + 1];    // kernel slice [o][f] of one (head, rank)
};

// Gather of S_{hd,l} for the tile: thread (p = tid % 64, quarter = tid / 64)
// accumulates channels 4*(quarter + 4*i) .. +3 of head hd, i < 4, for pixel p.
SNLS_DEV void gr_gather(GrSmem& sm, const float* __restrict__ vcl, const float* __restrict__ weights,
                        const float* __restrict__ inds, const Geo& g, int b, int t, int hd, int l, int y0, int x0,
                        float (&acc)[gr::CPT], int* cnt_out) {
  using namespace gr;
  const int tid = threadIdx.x;
  int mh0, mh1, mw0, mw1;
  cover_range(y0, g.s0, g.nH, g.lo, g.ps, &mh0, &mh1);
  cover_range(x0, g.s0, g.nW, g.lo, g.ps, &mw0, &mw1);
  const int nmh = max(mh1 - mh0 + 1, 0), nmw = max(mw1 - mw0 + 1, 0);
  __syncthreads();  // the previous records are no longer read
  for (int e = tid; e < nmh * nmw; e += NT) {
    const int mh = mh0 + e / nmw, mw = mw0 + e % nmw;
    const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
    const float w = weights[row * g.k + l];
    const float* ind = inds + (row * g.k + l) * 3;
    const float tf = ind[0], dh = ind[1], dw = ind[2];
    GrRecord r;
    const bool ok = w != 0.f && tf >= 0.f && tf < (float)g.T && tf == floorf(tf) && fabsf(dh) < kFarDisp &&
                    fabsf(dw) < kFarDisp;
    r.w = ok ? w : 0.f;
    r.tf = ok ? (int)tf : 0;
    int ny = 0, nx = 0;
    float ay = 0.f, ax = 0.f;
    if (ok) {
      split_disp(dh, &ny, &ay);
      split_disp(dw, &nx, &ax);
    }
    r.ny = ny;
    r.nx = nx;
    r.ay = ay;
    r.ax = ax;
    sm.rec[e] = r;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < CPT; ++i) acc[i] = 0.f;
  const int p = tid % NP, quarter = tid / NP;
  const int y = y0 + p / TS, x = x0 + p % TS;
  *cnt_out = 0;
  if (y >= g.H || x >= g.W) return;
  // covering queries of the pixel
  int a0, a1, c0, c1;
  {
    const int a = y - g.lo - g.ps + 1, bb = y - g.lo;
    a0 = max(a <= 0 ? 0 : (a + g.s0 - 1) / g.s0, mh0);
    a1 = min(bb / g.s0, mh1);
    const int c = x - g.lo - g.ps + 1, cc = x - g.lo;
    c0 = max(c <= 0 ? 0 : (c + g.s0 - 1) / g.s0, mw0);
    c1 = min(cc / g.s0, mw1);
  }
  *cnt_out = max(a1 - a0 + 1, 0) * max(c1 - c0 + 1, 0);
  const int Fh = g.Ch;
  const long long fstride = g.HW * g.C;  // floats per frame of the channels-last copy
  const float* vb = vcl + (long long)b * g.T * fstride + (long long)hd * Fh;
  for (int mh = a0; mh <= a1; ++mh) {
    for (int mw = c0; mw <= c1; ++mw) {
      const GrRecord r = sm.rec[(mh - mh0) * nmw + (mw - mw0)];
      if (r.w == 0.f) continue;
      const int Y = y + r.ny, X = x + r.nx;
      const bool y0in = Y >= 0 && Y < g.H, y1in = Y + 1 >= 0 && Y + 1 < g.H;
      const bool x0in = X >= 0 && X < g.W, x1in = X + 1 >= 0 && X + 1 < g.W;
      const float w00 = r.w * (1.f - r.ay) * (1.f - r.ax), w01 = r.w * (1.f - r.ay) * r.ax;
      const float w10 = r.w * r.ay * (1.f - r.ax), w11 = r.w * r.ay * r.ax;
      const float* f0 = vb + (long long)r.tf * fstride;
#pragma unroll
      for (int i = 0; i < CPT / 4; ++i) {
        const int cg = quarter + 4 * i;  // channel group of 4
        if (4 * cg >= Fh) break;
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        auto tap = [&](bool in, int YY, int XX, float wt) {
          if (in && wt != 0.f) {
            const float4 v4 = *reinterpret_cast<const float4*>(f0 + ((long long)YY * g.W + XX) * g.C + 4 * cg);
            s.x = fmaf(wt, v4.x, s.x);
            s.y = fmaf(wt, v4.y, s.y);
            s.z = fmaf(wt, v4.z, s.z);
            s.w = fmaf(wt, v4.w, s.w);
          }
        };
        tap(y0in && x0in, Y, X, w00);
        tap(y0in && x1in, Y, X + 1, w01);
        tap(y1in && x0in, Y + 1, X, w10);
        tap(y1in && x1in, Y + 1, X + 1, w11);
        acc[4 * i + 0] += s.x;
        acc[4 * i + 1] += s.y;
        acc[4 * i + 2] += s.z;
        acc[4 * i + 3] += s.w;
      }
    }
  }
}

// ---- standalone gather: S to the stacked tensor (B, HD, k, T, F', H, W) ----

__global__ void __launch_bounds__(gr::NT) gather_stacked_tile_kernel(const float* __restrict__ vcl,
                                                                     const float* __restrict__ weights,
                                                                     const float* __restrict__ inds, Geo g,
                                                                     int tiles_x, int tiles_y,
                                                                     float* __restrict__ stacked) {
  using namespace gr;
  __shared__ GrSmem sm;
  const int tile = (int)(blockIdx.x % (unsigned)(tiles_x * tiles_y));
  const int bt = (int)(blockIdx.x / (unsigned)(tiles_x * tiles_y));
  const int b = bt / g.T, t = bt % g.T;
  const int y0 = (tile / tiles_x) * TS, x0 = (tile % tiles_x) * TS;
  const int tid = threadIdx.x, p = tid % NP, quarter = tid / NP;
  const int y = y0 + p / TS, x = x0 + p % TS;
  for (int hd = 0; hd < g.HD; ++hd)
    for (int l = 0; l < g.k; ++l) {
      float acc[CPT];
      int cnt;
      gr_gather(sm, vcl, weights, inds, g, b, t, hd, l, y0, x0, acc, &cnt);
      if (y < g.H && x < g.W) {
        const float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
        float* ob = stacked + ((((long long)b * g.HD + hd) * g.k + l) * g.T + t) * g.Ch * g.HW + (long long)y * g.W + x;
#pragma unroll
        for (int i = 0; i < CPT / 4; ++i) {
          const int cg = quarter + 4 * i;
          if (4 * cg >= g.Ch) break;
#pragma unroll
          for (int e = 0; e < 4; ++e) ob[(long long)(4 * cg + e) * g.HW] = cnt > 0 ? acc[4 * i + e] * inv : 0.f;
        }
      }
    }
}

// ---- reduction over the neighbours on the matrix cores ----
//
// For the tile's 64 pixels, out[p][o] += sum_f S[f][p] * Pm[o][f] for one
// (head, rank): wave w takes pixels 16w .. 16w+15 (A rows) and every block of
// 16 output channels (B columns); v_mfma_f32_16x16x4f32 takes A[i][kk] from
// lane i + 16 kk, B[kk][j] from lane j + 16 kk and leaves D[4 gq + r][j] in
// register r of lane j + 16 gq.
SNLS_DEV void gr_mfma(const GrSmem& sm, int Fh, int nob, f32x4 (&accv)[gr::OMAX / 16]) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int i = lane & 15, kk = lane >> 4;
  for (int f0 = 0; f0 < Fh; f0 += 4) {
    const float a = sm.S[f0 + kk][16 * wv + i];
#pragma unroll
    for (int ob = 0; ob < gr::OMAX / 16; ++ob) {
      if (ob < nob) {
        const float bv = sm.Pm[16 * ob + i][f0 + kk];
        accv[ob] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv, accv[ob], 0, 0, 0);
      }
    }
  }
}

// Kernel slice of (head hd, rank l): Pm[o][f] = proj[o, hd*F' + f, l] for the
// nob blocks of 16 output channels (0 past Cout).
SNLS_DEV void gr_stage_proj(GrSmem& sm, const float* __restrict__ proj, const Geo& g, int cout, int nob, int hd,
                            int l) {
  for (int e = threadIdx.x; e < 16 * nob * g.Ch; e += gr::NT) {
    const int o = e / g.Ch, f = e % g.Ch;
    sm.Pm[o][f] = o < cout ? proj[((long long)o * g.C + (long long)hd * g.Ch + f) * g.k + l] : 0.f;
  }
}

// out (B, T, Cout, H, W) from the accumulators of the tile.
SNLS_DEV void gr_store(const f32x4 (&accv)[gr::OMAX / 16], int nob, const Geo& g, int cout, int b, int t, int y0,
                       int x0, int tw, float* __restrict__ out) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int j = lane & 15, gq = lane >> 4;
#pragma unroll
  for (int ob = 0; ob < gr::OMAX / 16; ++ob) {
    if (ob >= nob) break;
    const int o = 16 * ob + j;
    const float vals[4] = {accv[ob][0], accv[ob][1], accv[ob][2], accv[ob][3]};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = 16 * wv + 4 * gq + r;
      const int y = y0 + p / tw, x = x0 + p % tw;
      if (o < cout && y < g.H && x < g.W)
        out[(((long long)b * g.T + t) * cout + o) * g.HW + (long long)y * g.W + x] = vals[r];
    }
  }
}

// Fused gather + reduction: the stacked tensor stays on chip.
__global__ void __launch_bounds__(gr::NT) gather_reduce_kernel(const float* __restrict__ vcl,
                                                               const float* __restrict__ weights,
                                                               const float* __restrict__ inds,
                                                               const float* __restrict__ proj, Geo g, int cout,
                                                               int tiles_x, int tiles_y, float* __restrict__ out) {
  using namespace gr;
  __shared__ GrSmem sm;
  const int tile = (int)(blockIdx.x % (unsigned)(tiles_x * tiles_y));
  const int bt = (int)(blockIdx.x / (unsigned)(tiles_x * tiles_y));
  const int b = bt / g.T, t = bt % g.T;
  const int y0 = (tile / tiles_x) * TS, x0 = (tile % tiles_x) * TS;
  const int tid = threadIdx.x, p = tid % NP, quarter = tid / NP;
  const int nob = (cout + 15) / 16;
  f32x4 accv[OMAX / 16];
#pragma unroll
  for (int ob = 0; ob < OMAX / 16; ++ob) accv[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int hd = 0; hd < g.HD; ++hd)
    for (int l = 0; l < g.k; ++l) {
      float acc[CPT];
      int cnt;
      gr_gather(sm, vcl, weights, inds, g, b, t, hd, l, y0, x0, acc, &cnt);  // (barriers inside)
      const float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
#pragma unroll
      for (int i = 0; i < CPT / 4; ++i) {
        const int cg = quarter + 4 * i;
        if (4 * cg >= g.Ch) break;
#pragma unroll
        for (int e = 0; e < 4; ++e) sm.S[4 * cg + e][p] = acc[4 * i + e] * inv;
      }
      gr_stage_proj(sm, proj, g, cout, nob, hd, l);
      __syncthreads();
      gr_mfma(sm, g.Ch, nob, accv);
      __syncthreads();  // S and Pm are rewritten for the next (head, rank)
    }
  gr_store(accv, nob, g, cout, b, t, y0, x0, TS, out);
}

// Reduction of a stacked tensor from memory: a tile is 64 consecutive
// pixels of one row, so the stack's channel rows are read coalesced.
__global__ void __launch_bounds__(gr::NT) stacked_reduce_kernel(const float* __restrict__ stacked,
                                                                const float* __restrict__ proj, Geo g, int cout,
                                                                int tiles_x, int tiles_y, float* __restrict__ out) {
  using namespace gr;
  __shared__ GrSmem sm;
  const int tile = (int)(blockIdx.x % (unsigned)(tiles_x * tiles_y));
  const int bt = (int)(blockIdx.x / (unsigned)(tiles_x * tiles_y));
  const int b = bt / g.T, t = bt % g.T;
  const int y0 = tile / tiles_x, x0 = (tile % tiles_x) * NP;
  const int nob = (cout + 15) / 16;
  f32x4 accv[OMAX / 16];
#pragma unroll
  for (int ob = 0; ob < OMAX / 16; ++ob) accv[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int hd = 0; hd < g.HD; ++hd)
    for (int l = 0; l < g.k; ++l) {
      const float* sb = stacked + ((((long long)b * g.HD + hd) * g.k + l) * g.T + t) * g.Ch * g.HW + (long long)y0 * g.W;
      for (int e = threadIdx.x; e < g.Ch * NP; e += NT) {
        const int f = e / NP, p = e % NP;
        const int x = x0 + p;
        sm.S[f][p] = x < g.W ? sb[(long long)f * g.HW + x] : 0.f;
      }
      gr_stage_proj(sm, proj, g, cout, nob, hd, l);
      __syncthreads();
      gr_mfma(sm, g.Ch, nob, accv);
      __syncthreads();
    }
  gr_store(accv, nob, g, cout, b, t, y0, x0, NP, out);
}

// The tiled kernels: channels of a head a multiple of 4 and at most 64, at
// most 256 covering queries per 8 x 8 tile, 32-bit frame offsets.
bool gather_tile_supported(const Geo& g) {
  const int nq = ((gr::TS + g.ps - 2) / g.s0 + 1);
  return g.Ch % 4 == 0 && g.Ch <= gr::FMAX && g.C % 4 == 0 && nq * nq <= gr::RMAX && g.k >= 1;
}

bool reduce_supported(const Geo& g, int cout) {
  return g.Ch % 4 == 0 && g.Ch <= gr::FMAX && cout >= 1 && cout <= gr::OMAX && g.k >= 1;
}

size_t gather_ws_bytes(const Geo& g) {
  return gather_tile_supported(g) ? (size_t)g.B * g.T * g.C * g.HW * sizeof(float) : 0;
}

static long long gr_tiles(const Geo& g, int* tx, int* ty) {
  *tx = (g.W + gr::TS - 1) / gr::TS;
  *ty = (g.H + gr::TS - 1) / gr::TS;
  return (long long)*tx * *ty * g.B * g.T;
}

snls_status launch_gather_stacked(const float* v, const float* weights, const float* inds, const Geo& g,
                                  float* stacked, void* ws, hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  if (!gather_tile_supported(g)) return launch_gather_stacked_plain(v, weights, inds, g, stacked, s);
  float* vcl = static_cast<float*>(ws);
  snls_status st = launch_to_channels_last(v, g, vcl, s);
  if (st != SNLS_OK) return st;
  int tx, ty;
  const long long nwg = gr_tiles(g, &tx, &ty);
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(gather_stacked_tile_kernel, dim3((unsigned)nwg), dim3(gr::NT), 0, s, vcl, weights, inds, g, tx,
                     ty, stacked);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_stacked_reduce(const float* stacked, const float* proj, const Geo& g, int cout, float* out,
                                  hipStream_t s) {
  const int tx = (g.W + gr::NP - 1) / gr::NP, ty = g.H;  // row strips of 64 pixels
  const long long nwg = (long long)tx * ty * g.B * g.T;
  if (nwg == 0) return SNLS_OK;
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  hipLaunchKernelGGL(stacked_reduce_kernel, dim3((unsigned)nwg), dim3(gr::NT), 0, s, stacked, proj, g, cout, tx, ty,
                     out);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_gather_reduce(const float* v, const float* weights, const float* inds, const float* proj,
                                 const Geo& g, int cout, float* out, void* ws, hipStream_t s) {
  int tx, ty;
  const long long nwg = gr_tiles(g, &tx, &ty);
  if (nwg == 0) return SNLS_OK;
  if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  float* vcl = static_cast<float*>(ws);
  snls_status st = launch_to_channels_last(v, g, vcl, s);
  if (st != SNLS_OK) return st;
  hipLaunchKernelGGL(gather_reduce_kernel, dim3((unsigned)nwg), dim3(gr::NT), 0, s, vcl, weights, inds, proj, g, cout,
                     tx, ty, out);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

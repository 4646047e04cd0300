// search_p1.hip -- scores of the shifted search for single-pixel patches
// (P = 1), any query stride, key stride 1, inner product (Sec. 3.2).
//
// With P = 1 a candidate's score is the bilinear combination of four pixel
// correlations c(y, x) = <q(query), K(y, x)>.  For one query and one window
// row d_h, every cell of the row reads its taps from key rows floor(disp_h)
// and floor(disp_h) + 1, and from the ws + 2 columns starting at
// floor(disp_w of cell 0) (the cells' floors are nondecreasing and, for key
// stride 1, each lies within one of its ideal column).  So a thread per
// (query, window row) accumulates the 2 x (ws + 2) correlations over the
// head's channels from an LDS copy of the key region the tile's windows span,
// then forms the row's scores with each cell's exact displacement, and writes
// them to the workspace row of the query (candidate id order) for the
// streaming top-k kernel.
#include "snls_internal.h"

namespace snls {

namespace p1 {
constexpr int TQ = 8;                  // 8 x 8 queries per workgroup (query-grid units)
constexpr int NQ = TQ * TQ;
constexpr int WSM = 15;                // largest window side
constexpr int NR = 16;                 // thread slots per query (window rows)
constexpr int NT = NQ * NR;            // 1024
constexpr int NC = WSM + 2;            // correlation columns per window row
constexpr int CC = 4;                  // channels per staging chunk (double-buffered)
constexpr int RH = 48, RW = 48;        // key region of the tile (taps included)
constexpr int RP = RW + 1;             // row pitch (odd)
constexpr int CHUNK = CC * RH * RP;
constexpr int QR = WSM + 2;            // per-query block (when the tile's region is too wide): rows ..
constexpr int QB = QR * NC;            // .. x NC columns, one channel at a time
static_assert(NQ * QB <= 2 * CHUNK, "per-query blocks fit in the two staging buffers");
}  // namespace p1

__global__ void __launch_bounds__(p1::NT) search_p1_scores_kernel(const float* __restrict__ q,
                                                                  const float* __restrict__ k,
                                                                  const float* __restrict__ flows, Geo g,
                                                                  int tiles_x, float* __restrict__ scores,
                                                                  int pitch) {
  using namespace p1;
  __shared__ float reg[2][CHUNK];
  __shared__ float qs[2][CC][NQ];
  __shared__ int ubox[4];
  __shared__ int y0q[NQ], x0q[NQ];  // first key row and column of each query's block

  const int tid = threadIdx.x, j = tid / NR, dh = tid % NR;
  const int dt = (int)blockIdx.z - g.wt;
  const int img = (int)blockIdx.y;  // (b, hd, t)
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  const int t2 = t + dt;
  if (t2 < 0 || t2 >= g.T) return;  // whole workgroup: frame outside the clip
  const int ty = (int)blockIdx.x / tiles_x, tx = (int)blockIdx.x % tiles_x;
  const int mh = ty * TQ + j / TQ, mw = tx * TQ + j % TQ;  // query-grid position
  const bool inside = mh < g.nH && mw < g.nW;
  const bool task = inside && dh < g.ws;
  const int h = mh * g.s0, w = mw * g.s0;

  float fh = 0.f, fw = 0.f;
  if (dt != 0 && inside) {
    const long long base = (((long long)b * g.T + t) * g.nslot + flow_slot(dt, g.wt)) * 2;
    const long long pix = (long long)h * g.W + w;
    fh = flows[base * g.HW + pix];
    fw = flows[(base + 1) * g.HW + pix];
  }
  // this task's key rows and the row's first column; offsets that are not
  // finite or absurdly large are placed at 0 for the region (their cells
  // fail the exact validity test)
  const float disp_h = cand_disp(fh, g.s1, dh, g.r);
  const float disp_w0 = cand_disp(fw, g.s1, 0, g.r);
  const bool sane = fabsf(fh) < 1.0e6f && fabsf(fw) < 1.0e6f;
  const int y0 = sane ? h + (int)floorf(disp_h) : h;
  const int x0 = sane ? w + (int)floorf(disp_w0) : w;
  if (tid < 4) ubox[tid] = (tid & 1) ? INT_MIN : INT_MAX;
  if (dh == 0) {
    y0q[j] = y0;
    x0q[j] = x0;
  }
  __syncthreads();
  if (task) {
    atomicMin(&ubox[0], y0);
    atomicMax(&ubox[1], y0);
    atomicMin(&ubox[2], x0);
    atomicMax(&ubox[3], x0);
  }
  __syncthreads();
  const int ry0 = ubox[0], rx0 = ubox[2];
  const int rh = ubox[1] - ry0 + 2, rw = ubox[3] - rx0 + NC;
  // The tile's key region is staged CC channels at a time when it fits;
  // otherwise (windows far apart) each query's own block of rows and
  // columns is staged, one channel at a time.
  const bool staged = ubox[1] >= ubox[0] && rh <= RH && rw <= RW;

  const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;
  auto kval = [&](int c, int y, int x) -> float {
    return (y >= 0 && y < g.H && x >= 0 && x < g.W) ? kb[(long long)c * g.HW + (long long)y * g.W + x] : 0.f;
  };
  const int cpc = staged ? CC : 1;        // channels per chunk
  const int nreg = rh * rw;
  auto stage = [&](int buf, int c0) {
    if (staged) {
      for (int e = tid; e < CC * nreg; e += NT) {
        const int c = e / nreg, rem = e - c * nreg;
        const int yy = rem / rw, xx = rem - yy * rw;
        reg[buf][(c * RH + yy) * RP + xx] = c0 + c < g.Ch ? kval(c0 + c, ry0 + yy, rx0 + xx) : 0.f;
      }
    } else {
      for (int e = tid; e < NQ * QB; e += NT) {  // both buffers: no double buffering
        const int jj = e / QB, rem = e - jj * QB;
        const int yy = rem / NC, xx = rem - yy * NC;
        (&reg[0][0])[e] = kval(c0, y0q[jj] + yy, x0q[jj] + xx);
      }
    }
    if (tid < cpc * NQ) {
      const int c = tid / NQ, jj = tid % NQ;
      const int qh = (ty * TQ + jj / TQ) * g.s0, qw = (tx * TQ + jj % TQ) * g.s0;
      qs[buf][c][jj] = (c0 + c < g.Ch && qh < g.H && qw < g.W)
                           ? qb[(long long)(c0 + c) * g.HW + (long long)qh * g.W + qw] : 0.f;
    }
  };
  // this task's two rows in the staging buffer
  const int toff = staged ? (y0 - ry0) * RP + (x0 - rx0) : j * QB + (y0 - y0q[j]) * NC;
  const int rp = staged ? RP : NC;             // row pitch
  const int cstride = staged ? RH * RP : 0;    // channel stride

  float c0r[NC], c1r[NC];  // correlations of key rows y0 and y0 + 1, columns x0 ..
#pragma unroll
  for (int x = 0; x < NC; ++x) c0r[x] = c1r[x] = 0.f;
  if (staged) stage(0, 0);
  int buf = 0;
  for (int c0 = 0; c0 < g.Ch; c0 += cpc, buf ^= staged ? 1 : 0) {
    if (staged) {
      __syncthreads();  // chunk c0 is staged in buf; buf^1 is free
      if (c0 + cpc < g.Ch) stage(buf ^ 1, c0 + cpc);
    } else {
      __syncthreads();  // the previous channel is no longer read
      stage(0, c0);
      __syncthreads();
    }
    if (task) {
      const float* base = staged ? reg[buf] : &reg[0][0];
      for (int c = 0; c < cpc && c0 + c < g.Ch; ++c) {
        const float qv = qs[buf][c][j];
        const float* r0 = base + c * cstride + toff;
#pragma unroll
        for (int x = 0; x < NC; ++x) {
          c0r[x] = fmaf(qv, r0[x], c0r[x]);
          c1r[x] = fmaf(qv, r0[rp + x], c1r[x]);
        }
      }
    }
  }
  if (!task) return;  // no barrier follows
  // the row's scores: taps from each cell's own displacement
  const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
  float* srow = scores + row * pitch + ((dt + g.wt) * g.ws + dh) * g.ws;
  const bool okh = centre_ok(h, disp_h, g.H) && sane;
  const float ah = disp_h - floorf(disp_h);
  const int fl0 = (int)floorf(disp_w0);
#pragma unroll
  for (int dw = 0; dw < WSM; ++dw) {
    if (dw < g.ws) {
      const float disp_w = cand_disp(fw, g.s1, dw, g.r);
      const bool ok = okh && centre_ok(w, disp_w, g.W);
      const float flw = floorf(disp_w);
      const float aw = disp_w - flw;
      // column of the cell's first tap: dw - 1, dw or dw + 1 (rounding of disp)
      const int dc = ok ? (int)flw - fl0 - dw : 0;
      const float a0 = dc < 0 ? c0r[dw > 0 ? dw - 1 : 0] : (dc > 0 ? c0r[dw + 1] : c0r[dw]);
      const float a1 = dc < 0 ? c0r[dw] : (dc > 0 ? c0r[dw + 2] : c0r[dw + 1]);
      const float b0 = dc < 0 ? c1r[dw > 0 ? dw - 1 : 0] : (dc > 0 ? c1r[dw + 1] : c1r[dw]);
      const float b1 = dc < 0 ? c1r[dw] : (dc > 0 ? c1r[dw + 2] : c1r[dw + 1]);
      const float top = (1.f - aw) * a0 + aw * a1;
      const float bot = (1.f - aw) * b0 + aw * b1;
      const float dv = (1.f - ah) * top + ah * bot;
      srow[dw] = ok && dv == dv ? dv : -INFINITY;  // NaN scores as invalid
    }
  }
}

// P = 1, key stride 1, inner product, ws <= 15 (any query stride).
bool p1_supported(const Geo& g) {
  return g.ps == 1 && g.s1 == 1.0f && g.dist == SNLS_DIST_PROD && g.ws <= p1::WSM && g.k >= 1 &&
         (long long)g.Ch * g.HW * 4 < (1LL << 31);
}

snls_status launch_search_p1_scores(const float* q, const float* k, const float* flows, const Geo& g, float* scores,
                                    int pitch, hipStream_t s) {
  const int tiles_x = (g.nW + p1::TQ - 1) / p1::TQ, tiles_y = (g.nH + p1::TQ - 1) / p1::TQ;
  const long long ntile = (long long)tiles_x * tiles_y;
  if (ntile == 0 || g.rows == 0) return SNLS_OK;
  if (ntile > 0x7fffffffLL || (long long)g.B * g.HD * g.T > 65535 || 2 * g.wt + 1 > 65535) return SNLS_ERR_UNSUPPORTED;
  dim3 grid((unsigned)ntile, (unsigned)(g.B * g.HD * g.T), (unsigned)(2 * g.wt + 1));
  hipLaunchKernelGGL(search_p1_scores_kernel, grid, dim3(p1::NT), 0, s, q, k, flows, g, tiles_x, scores, pitch);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

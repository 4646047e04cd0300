// search_p1.hip -- scores of the shifted search for single-pixel patches
// (P = 1), any query stride, key stride 1, inner product (Sec. 3.2).
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
// directly.  The scores are gathered per tile in LDS and written to the
// workspace rows of the queries (candidate id order, consecutive threads on
// consecutive addresses) for the streaming top-k kernel.
#include "snls_internal.h"

namespace snls {

namespace p1 {
constexpr int TQ = 8;                  // 8 x 8 queries per workgroup (query-grid units)
constexpr int NQ = TQ * TQ;
constexpr int WSM = 15;                // largest window side
constexpr int NR = 16;                 // thread slots per query (key rows): one 16-lane DPP row
constexpr int NT = NQ * NR;            // 1024
constexpr int NC = WSM + 2;            // correlation columns per key row
constexpr int CC = 4;                  // channels per staging chunk (double-buffered)
constexpr int RH = 48, RW = 48;        // key region of the tile
constexpr int RP = RW + 1;             // row pitch (odd)
constexpr int NRI = (RH + NT / 64 - 1) / (NT / 64);  // region rows per thread (lane = column)
constexpr int CHUNK = CC * RH * RP;
constexpr int QR = WSM + 2;            // per-query block (when the tile's region is too wide): rows ..
constexpr int QB = QR * NC;            // .. x NC columns, one channel at a time
static_assert(NQ * QB <= 2 * CHUNK, "per-query blocks fit in the two staging buffers");
static_assert(RW <= 64, "a region row is staged by one wave");
static_assert(NQ * WSM * WSM <= 2 * CHUNK, "the tile's scores of one frame fit in the staging buffers");
}  // namespace p1

// Value of lane i + 1 of the same 16-lane row (lane 15 reads 0).
SNLS_DEV float next_lane(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x101, 0xf, 0xf, true));
}
SNLS_DEV int next_lane(int v) { return __builtin_amdgcn_update_dpp(0, v, 0x101, 0xf, 0xf, true); }

__global__ void __launch_bounds__(p1::NT, 8) search_p1_scores_kernel(const float* __restrict__ q,
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
  const bool rowtask = inside && dh <= g.ws;  // thread accumulates a key row
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
  const int drow = min(dh, g.ws - 1);
  const float disp_h = cand_disp(fh, g.s1, drow, g.r);
  const float disp_w0 = cand_disp(fw, g.s1, 0, g.r);
  const bool sane = fabsf(fh) < kFarDisp && fabsf(fw) < kFarDisp;
  const int below = dh == g.ws ? 1 : 0;  // the row under the last window row
  const int y0 = (sane ? h + (int)floorf(disp_h) : h) + below;
  const int x0 = sane ? w + (int)floorf(disp_w0) : w;
  if (tid < 4) ubox[tid] = (tid & 1) ? INT_MIN : INT_MAX;
  if (dh == 0) {
    y0q[j] = y0;
    x0q[j] = x0;
  }
  __syncthreads();
  {
    // union bounds: wave reductions, then one LDS atomic per wave
    int a0 = rowtask ? y0 : INT_MAX, a1 = rowtask ? y0 : INT_MIN;
    int a2 = rowtask ? x0 : INT_MAX, a3 = rowtask ? x0 : INT_MIN;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      a0 = min(a0, __shfl_xor(a0, off));
      a1 = max(a1, __shfl_xor(a1, off));
      a2 = min(a2, __shfl_xor(a2, off));
      a3 = max(a3, __shfl_xor(a3, off));
    }
    if ((tid & 63) == 0 && a0 <= a1) {
      atomicMin(&ubox[0], a0);
      atomicMax(&ubox[1], a1);
      atomicMin(&ubox[2], a2);
      atomicMax(&ubox[3], a3);
    }
  }
  __syncthreads();
  const int ry0 = ubox[0], rx0 = ubox[2];
  const int rh = ubox[1] - ry0 + 1, rw = ubox[3] - rx0 + NC;
  // The tile's key region is staged CC channels at a time when it fits;
  // otherwise (windows far apart) each query's own block of rows and
  // columns is staged, one channel at a time.
  const bool staged = ubox[1] >= ubox[0] && rh <= RH && rw <= RW;

  const float* kb = k + (((long long)b * g.T + t2) * g.C + (long long)hd * g.Ch) * g.HW;
  const float* qb = q + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW;
  auto kval = [&](int c, int y, int x) -> float {
    return (y >= 0 && y < g.H && x >= 0 && x < g.W) ? kb[(long long)c * g.HW + (long long)y * g.W + x] : 0.f;
  };
  const int cpc = staged ? CC : 1;  // channels per chunk
  // Region staging through registers: lane = column, the 16 waves take the
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
#pragma unroll
  for (int i = 0; i < NRI; ++i) {
    const int yy = (tid >> 6) + (NT / 64) * i;
    const int y = ry0 + yy, x = rx0 + xx;
    roff[i] = (staged && xx < rw && yy < rh && y >= 0 && y < g.H && x >= 0 && x < g.W) ? (unsigned)((y * g.W + x) * 4)
                                                                                        : OOB;
  }
  // this thread's q staging item (tid < CC * NQ): channel tid / NQ of query
  // tid % NQ, as a byte offset in channel 0 (OOB: outside the frame)
  const __amdgpu_buffer_rsrc_t q_rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)qb, (short)0, (int)(g.Ch * g.HW * 4), 0x00020000);
  unsigned qoff = OOB;
  if (tid < CC * NQ) {
    const int c = tid / NQ, jj = tid % NQ;
    const int qh = (ty * TQ + jj / TQ) * g.s0, qw = (tx * TQ + jj % TQ) * g.s0;
    if (qh < g.H && qw < g.W) qoff = (unsigned)(((long long)c * g.HW + (long long)qh * g.W + qw) * 4);
  }
  float stg[CC][NRI];
  float qstg = 0.f;
  auto load_chunk = [&](int c0) {
#pragma unroll
    for (int c = 0; c < CC; ++c) {
      const unsigned coff = (unsigned)(c0 + c) * (unsigned)g.HW * 4u;
      const bool cin = c0 + c < g.Ch;
#pragma unroll
      for (int i = 0; i < NRI; ++i) {
        const unsigned off = (roff[i] != OOB && cin) ? roff[i] + coff : OOB;
        stg[c][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(k_rs, off, 0, 0));
      }
    }
    if (tid < CC * NQ) {
      const bool cin = c0 + tid / NQ < g.Ch;
      const unsigned off = (qoff != OOB && cin) ? qoff + (unsigned)c0 * (unsigned)g.HW * 4u : OOB;
      qstg = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(q_rs, off, 0, 0));
    }
  };
  auto store_chunk = [&](int buf) {
    // rows past the region and columns up to the pitch receive zeros that are never read
    if (xx < RP) {
#pragma unroll
      for (int c = 0; c < CC; ++c)
#pragma unroll
        for (int i = 0; i < NRI; ++i) reg[buf][(c * RH + (tid >> 6) + (NT / 64) * i) * RP + xx] = stg[c][i];
    }
    if (tid < CC * NQ) qs[buf][tid / NQ][tid % NQ] = qstg;
  };
  // Per-query blocks (windows far apart): one channel at a time.
  auto stage_blocks = [&](int c0) {
    for (int e = tid; e < NQ * QB; e += NT) {  // both buffers: no double buffering
      const int jj = e / QB, rem = e - jj * QB;
      const int yy = rem / NC, x = rem - yy * NC;
      (&reg[0][0])[e] = kval(c0, y0q[jj] + yy, x0q[jj] + x);
    }
    if (tid < NQ) {
      const int qh = (ty * TQ + tid / TQ) * g.s0, qw = (tx * TQ + tid % TQ) * g.s0;
      qs[0][0][tid] = (qh < g.H && qw < g.W) ? qb[(long long)c0 * g.HW + (long long)qh * g.W + qw] : 0.f;
    }
  };
  // this thread's row in the staging buffer
  const int toff = staged ? (y0 - ry0) * RP + (x0 - rx0) : j * QB + (y0 - y0q[j]) * NC;

  float cr[NC];  // correlations of key row y0, columns x0 ..
#pragma unroll
  for (int x = 0; x < NC; ++x) cr[x] = 0.f;
  if (staged) {
    load_chunk(0);
    store_chunk(0);
  }
  int buf = 0;
  for (int c0 = 0; c0 < g.Ch; c0 += cpc, buf ^= staged ? 1 : 0) {
    const bool more = staged && c0 + cpc < g.Ch;
    if (staged) {
      __syncthreads();  // chunk c0 is staged in buf; buf^1 is free
      if (more) load_chunk(c0 + cpc);  // in flight during this chunk's products
    } else {
      __syncthreads();  // the previous channel is no longer read
      stage_blocks(c0);
      __syncthreads();
    }
    if (rowtask) {
      if (staged) {
#pragma unroll
        for (int c = 0; c < CC; ++c) {
          if (c0 + c < g.Ch) {
            const float qv = qs[buf][c][j];
            const float* r0 = reg[buf] + c * (RH * RP) + toff;
#pragma unroll
            for (int x = 0; x < NC; ++x) cr[x] = fmaf(qv, r0[x], cr[x]);
          }
        }
      } else {
        const float qv = qs[0][0][j];
        const float* r0 = &reg[0][0] + toff;
#pragma unroll
        for (int x = 0; x < NC; ++x) cr[x] = fmaf(qv, r0[x], cr[x]);
      }
    }
    if (more) store_chunk(buf ^ 1);
  }
  // the key row below from the next lane (every lane takes part)
  float cn[NC];
#pragma unroll
  for (int x = 0; x < NC; ++x) cn[x] = next_lane(cr[x]);
  const int ynext = next_lane(y0);
  // The scores of the tile's queries for this frame go through LDS (the
  // staging buffers are free once every thread is past the channel loop):
  // query j's ws^2 scores at sbuf[j * ws^2 ..], then copied to the workspace
  // rows with consecutive threads on consecutive addresses.
  const int nc2 = g.ws * g.ws;
  float* sbuf = &reg[0][0];
  __syncthreads();
  if (inside && dh < g.ws) {
    float* dst = sbuf + j * nc2 + dh * g.ws;
    const bool okh = centre_ok(h, disp_h, g.H) && sane;
    if (okh && ynext != y0 + 1) {
      // rounding moved the next window row by two key rows: score directly
      for (int dw = 0; dw < g.ws; ++dw) {
        const float disp_w = cand_disp(fw, g.s1, dw, g.r);
        float d = -INFINITY;
        if (centre_ok(w, disp_w, g.W)) d = score_candidate(q, k, g, b, hd, t, h, w, t2, disp_h, disp_w);
        dst[dw] = d;
      }
    } else {
      // taps from each cell's own displacement
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
          const float a0 = dc < 0 ? cr[dw > 0 ? dw - 1 : 0] : (dc > 0 ? cr[dw + 1] : cr[dw]);
          const float a1 = dc < 0 ? cr[dw] : (dc > 0 ? cr[dw + 2] : cr[dw + 1]);
          const float b0 = dc < 0 ? cn[dw > 0 ? dw - 1 : 0] : (dc > 0 ? cn[dw + 1] : cn[dw]);
          const float b1 = dc < 0 ? cn[dw] : (dc > 0 ? cn[dw + 2] : cn[dw + 1]);
          const float top = (1.f - aw) * a0 + aw * a1;
          const float bot = (1.f - aw) * b0 + aw * b1;
          const float dv = (1.f - ah) * top + ah * bot;
          dst[dw] = ok && dv == dv ? dv : -INFINITY;  // NaN scores as invalid
        }
      }
    }
  }
  __syncthreads();
  // copy out: one wave per query row of the tile at a time
  const int lane = tid & 63;
  for (int jj = tid >> 6; jj < NQ; jj += NT / 64) {
    const int qh = ty * TQ + jj / TQ, qw = tx * TQ + jj % TQ;
    if (qh >= g.nH || qw >= g.nW) continue;
    const long long qrow = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + qh) * g.nW + qw;
    float* srow = scores + qrow * pitch + (dt + g.wt) * nc2;
    for (int e = lane; e < nc2; e += 64) srow[e] = sbuf[jj * nc2 + e];
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

// aggregate.hip -- weighted patch aggregation (Sec. 3.2 "Aggregation").
//
// out(y) = 1/cnt(y) * sum over query patches covering y, over the query's k
// neighbours l, of w_l * v~(frame_l, y + disp_l), with w = softmax over the
// row and v~ the bilinear read.  Written output-stationary (a gather, no
// float atomics on the output): for one output pixel, every (covering
// query, neighbour, bilinear tap) contribution lands on an integer source
// position of one frame.  Neighbouring queries select overlapping regions,
// so the ~4*k*P^2 contributions fall on far fewer distinct positions.  They
// are merged first -- weights summed per (frame, position) in a small LDS
// box, in 2^-24 fixed point with integer atomics so the sum does not depend
// on the order -- and only then is each distinct position's channel vector
// read once (channels-last copy of V, one coalesced 256-byte row per
// position for 64 channels) and accumulated.
//
// Kernels: softmax weights per (row, neighbour); transpose of V to
// (B,T,H,W,C); the tiled gather (query stride 1); the merged gather; the
// per-query gather of single-pixel patches (any query stride); plus the
// plain per-tap gather used when a configuration exceeds the other kernels'
// limits.
#include "snls_internal.h"

namespace snls {

namespace agg {
constexpr int TY = 8, TX = 8;          // output tile of one workgroup
constexpr int WAVES = 4;               // each wave processes 16 of the 64 pixels
constexpr int NSLOT = 7;               // frames per window: 2*wt + 1 <= 7
constexpr int BB = 16;                 // bin box side (positions base-7 .. base+8)
constexpr int BINS = NSLOT * BB * BB;  // per wave
constexpr int LMAX = BB * BB;          // non-zero list capacity per wave (one frame)
constexpr float QSCALE = 16777216.f;   // fixed point 2^24
}  // namespace agg

// Softmax weights of each row (0 for non-finite scores, for neighbours whose
// frame is not an integer in [0,T) or whose position is not finite).
// G lanes per row (G: the power of two >= k, at most 64): lane i of a row
// reads neighbours i, i + G, ... (consecutive lanes, consecutive addresses)
// and the row's maximum and normaliser are reduced across its G lanes.
template <int G>
__global__ void __launch_bounds__(256) softmax_weights_kernel(const float* __restrict__ dists,
                                                              const float* __restrict__ inds, Geo g, float scale,
                                                              float* __restrict__ wts) {
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = gid / G;
  const int sub = (int)(gid % G);
  const bool live = row < g.rows;  // every lane takes part in the shuffles
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  const float* d = dists + row * g.k;
  const float* ind = inds + row * g.k * 3;
  float m = -INFINITY;
  if (live)
    for (int l = sub; l < g.k; l += G)
      if (isfinite(d[l])) m = fmaxf(m, sscale * d[l]);
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  float z = 0.f;
  if (live)
    for (int l = sub; l < g.k; l += G)
      if (isfinite(d[l])) z += expf(sscale * d[l] - m);
#pragma unroll
  for (int off = G / 2; off > 0; off >>= 1) z += __shfl_xor(z, off);
  if (!live) return;
  const float inv = z > 0.f ? 1.f / z : 0.f;
  for (int l = sub; l < g.k; l += G) {
    const float tf = ind[3 * l], dh = ind[3 * l + 1], dw = ind[3 * l + 2];
    const bool ok = isfinite(d[l]) && tf >= 0.f && tf < (float)g.T && tf == floorf(tf) && fabsf(dh) < kFarDisp &&
                    fabsf(dw) < kFarDisp;
    wts[row * g.k + l] = ok ? expf(sscale * d[l] - m) * inv : 0.f;
  }
}

// (B,T,C,H,W) -> (B,T,H,W,C) through 64 x 64 LDS tiles.
__global__ void __launch_bounds__(256) to_channels_last_kernel(const float* __restrict__ v, Geo g,
                                                               float* __restrict__ vcl) {
  __shared__ float tileb[64][65];
  const long long bt = blockIdx.z;
  const int c0 = blockIdx.y * 64;
  const long long p0 = (long long)blockIdx.x * 64;
  const float* src = v + bt * g.C * g.HW;
  float* dst = vcl + bt * g.C * g.HW;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i;
    const long long p = p0 + tx;
    tileb[i][tx] = (c < g.C && p < g.HW) ? src[(long long)c * g.HW + p] : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const long long p = p0 + i;
    const int c = c0 + tx;
    if (c < g.C && p < g.HW) dst[p * g.C + c] = tileb[tx][i];
  }
}

// The same transpose with 16-byte accesses on both sides, for C and the
// head's channels multiples of 4 (HEAD: head-major order, each head's
// channels of a pixel contiguous): a thread loads 4 consecutive pixels of
// one channel (raw buffer loads at any 4-byte offset; pixels past the frame
// read 0) and stores 4 consecutive channels of one pixel.
template <bool HEAD>
__global__ void __launch_bounds__(256) to_channels_last4_kernel(const float* __restrict__ v, Geo g,
                                                                float* __restrict__ vcl) {
  __shared__ float tileb[64][65];  // [channel][pixel]
  const long long bt = blockIdx.z;
  const int c0 = blockIdx.y * 64;
  const long long p0 = (long long)blockIdx.x * 64;
  const float* src = v + bt * g.C * g.HW;
  float* dst = vcl + bt * g.C * g.HW;
  const int q4 = threadIdx.x & 15, r16 = threadIdx.x >> 4;
  // one channel plane per buffer: offsets past the frame read 0
  for (int i = r16; i < 64; i += 16) {
    const int c = c0 + i;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    const long long p = p0 + 4 * q4;
    if (c < g.C && p + 3 < g.HW) {
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc((void*)(src + (long long)c * g.HW), (short)0, (int)(g.HW * 4), 0x00020000);
      typedef float f32x4 __attribute__((ext_vector_type(4)));
      const f32x4 y = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (unsigned)(p * 4), 0, 0));
      x = make_float4(y.x, y.y, y.z, y.w);
    } else if (c < g.C) {  // the frame's last pixels: one at a time
      const float* sp = src + (long long)c * g.HW;
      x.x = p < g.HW ? sp[p] : 0.f;
      x.y = p + 1 < g.HW ? sp[p + 1] : 0.f;
      x.z = p + 2 < g.HW ? sp[p + 2] : 0.f;
    }
    tileb[i][4 * q4] = x.x;
    tileb[i][4 * q4 + 1] = x.y;
    tileb[i][4 * q4 + 2] = x.z;
    tileb[i][4 * q4 + 3] = x.w;
  }
  __syncthreads();
  for (int j = r16; j < 64; j += 16) {
    const long long p = p0 + j;
    const int c = c0 + 4 * q4;
    if (c < g.C && p < g.HW) {
      const float4 x = make_float4(tileb[4 * q4][j], tileb[4 * q4 + 1][j], tileb[4 * q4 + 2][j], tileb[4 * q4 + 3][j]);
      const long long o = HEAD ? ((long long)(c / g.Ch) * g.HW + p) * g.Ch + c % g.Ch : p * g.C + c;
      *reinterpret_cast<float4*>(dst + o) = x;
    }
  }
}

// Merged gather.  One workgroup = 8 x 8 output pixels of one (b, t, head);
// one wave per pixel at a time, lane = channel (CPL channels per lane).
template <int CPL>
__global__ void __launch_bounds__(256) aggregate_merged_kernel(const float* __restrict__ vcl,
                                                               const float* __restrict__ wts,
                                                               const float* __restrict__ inds, Geo g, int tiles_x,
                                                               int tiles_y, float* __restrict__ out) {
  using namespace agg;
  __shared__ int bins[WAVES][BINS];
  __shared__ int lst_off[WAVES][LMAX];
  __shared__ float lst_w[WAVES][LMAX];
  __shared__ float otile[64 * CPL][TY * TX + 1];

  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long long tiles_img = (long long)tiles_x * tiles_y;
  const long long wg = blockIdx.x;
  const int img = (int)(wg / tiles_img);
  const int trem = (int)(wg % tiles_img);
  const int ty = trem / tiles_x, tx = trem % tiles_x;
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  const int y0 = ty * TY, x0 = tx * TX;
  const int nslot = 2 * g.wt + 1;
  const int npairs = g.ps * g.ps * g.k;

  for (int i = lane; i < BINS; i += 64) bins[wv][i] = 0;

  for (int pi = wv; pi < TY * TX; pi += WAVES) {
    const int y = y0 + pi / TX, x = x0 + pi % TX;
    float acc[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) acc[c] = 0.f;
    if (y < g.H && x < g.W) {
      unsigned have = 0;  // slots with a base position (wave-uniform)
      int base_h[NSLOT], base_w[NSLOT];  // bin box origin per slot (wave-uniform)
#pragma unroll
      for (int s = 0; s < NSLOT; ++s) base_h[s] = base_w[s] = 0;
      for (int e0 = 0; e0 < npairs; e0 += 64) {
        const int e = e0 + lane;
        // this lane's contribution: (query patch offset p, neighbour l)
        bool has = false;
        int slot = -1, t2 = 0, nh = 0, nw = 0;
        float wl = 0.f, ah = 0.f, aw = 0.f;
        if (e < npairs) {
          const int pidx = e / g.k, l = e % g.k;
          const int ph = g.lo + pidx / g.ps, pw = g.lo + pidx % g.ps;
          const int h = y - ph, w = x - pw;
          if (h >= 0 && w >= 0 && h % g.s0 == 0 && w % g.s0 == 0 && h / g.s0 < g.nH && w / g.s0 < g.nW) {
            const long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + h / g.s0) * g.nW + w / g.s0;
            wl = wts[row * g.k + l];
            if (wl != 0.f) {
              const float* ind = inds + (row * g.k + l) * 3;
              t2 = (int)ind[0];  // an integer in [0,T): checked by the weight pass
              slot = t2 - t + g.wt;
              if (slot < 0 || slot >= nslot) slot = -1;  // outside the window: direct path
              const float fh = floorf(ind[1]), fw = floorf(ind[2]);
              nh = (int)fh;
              nw = (int)fw;
              ah = ind[1] - fh;
              aw = ind[2] - fw;
              has = true;
            }
          }
        }
        // bases of slots seen for the first time: the first such lane's position
#pragma unroll
        for (int s = 0; s < NSLOT; ++s) {
          if (s >= nslot || (have & (1u << s))) continue;
          const unsigned long long m = __ballot(has && slot == s);
          if (m) {
            const int src = __ffsll((long long)m) - 1;
            base_h[s] = __shfl(nh, src) - (BB / 2 - 1);
            base_w[s] = __shfl(nw, src) - (BB / 2 - 1);
            have |= 1u << s;
          }
        }
        bool over = has && slot < 0;
        if (has && slot >= 0) {
          int bh = 0, bw = 0;
#pragma unroll
          for (int s = 0; s < NSLOT; ++s)
            if (slot == s) {
              bh = base_h[s];
              bw = base_w[s];
            }
          const int rh = nh - bh, rw = nw - bw;
          if (rh >= 0 && rh + 1 < BB && rw >= 0 && rw + 1 < BB) {
            int* bb = &bins[wv][slot * BB * BB + rh * BB + rw];
            const float t00 = wl * (1.f - ah) * (1.f - aw), t01 = wl * (1.f - ah) * aw;
            const float t10 = wl * ah * (1.f - aw), t11 = wl * ah * aw;
            atomicAdd(bb, __float2int_rn(t00 * QSCALE));
            atomicAdd(bb + 1, __float2int_rn(t01 * QSCALE));
            atomicAdd(bb + BB, __float2int_rn(t10 * QSCALE));
            atomicAdd(bb + BB + 1, __float2int_rn(t11 * QSCALE));
          } else {
            over = true;
          }
        }
        // contributions outside the box: the whole wave reads their taps directly
        unsigned long long om = __ballot(over);
        while (om) {
          const int src = __ffsll((long long)om) - 1;
          om &= om - 1;
          const int t2_ = __shfl(t2, src), nh_ = __shfl(nh, src), nw_ = __shfl(nw, src);
          const float wl_ = __shfl(wl, src), ah_ = __shfl(ah, src), aw_ = __shfl(aw, src);
          const float* vb = vcl + ((long long)b * g.T + t2_) * g.HW * g.C + (long long)hd * g.Ch;
#pragma unroll
          for (int eh = 0; eh < 2; ++eh)
#pragma unroll
            for (int ew = 0; ew < 2; ++ew) {
              const int Y = y + nh_ + eh, X = x + nw_ + ew;
              const float tw = wl_ * (eh ? ah_ : 1.f - ah_) * (ew ? aw_ : 1.f - aw_);
              if (Y >= 0 && Y < g.H && X >= 0 && X < g.W && tw != 0.f) {
                const float* vp = vb + ((long long)Y * g.W + X) * g.C;
#pragma unroll
                for (int c = 0; c < CPL; ++c)
                  if (lane + 64 * c < g.Ch) acc[c] = fmaf(tw, vp[lane + 64 * c], acc[c]);
              }
            }
        }
      }
      __builtin_amdgcn_wave_barrier();
      // per frame: non-zero bins -> list (bin order: deterministic), bins
      // cleared on the way, then one channel-vector read per listed position
      wave_lds_sync();
      const float* vb = vcl + (long long)b * g.T * g.HW * g.C + (long long)hd * g.Ch;
#pragma unroll
      for (int s = 0; s < NSLOT; ++s) {
        if (s >= nslot || !(have & (1u << s))) continue;
        const int bh = base_h[s], bw = base_w[s];
        const int fbase = (t + s - g.wt) * (int)g.HW;
        int nlist = 0;
        for (int i0 = 0; i0 < BB * BB; i0 += 64) {
          const int i = i0 + lane;
          const int qv = bins[wv][s * BB * BB + i];
          const int Y = y + bh + i / BB, X = x + bw + i % BB;
          const bool nz = qv != 0 && Y >= 0 && Y < g.H && X >= 0 && X < g.W;
          if (qv != 0) bins[wv][s * BB * BB + i] = 0;
          const unsigned long long m = __ballot(nz);
          const int pos = nlist + __popcll(m & ((1ull << lane) - 1ull));
          if (nz) {
            lst_off[wv][pos] = (fbase + Y * g.W + X) * g.C;
            lst_w[wv][pos] = (float)qv * (1.f / QSCALE);
          }
          nlist += __popcll(m);
        }
        wave_lds_sync();
        int i = 0;
        for (; i + 4 <= nlist; i += 4) {
          const int o0 = lst_off[wv][i], o1 = lst_off[wv][i + 1], o2 = lst_off[wv][i + 2], o3 = lst_off[wv][i + 3];
          const float w0 = lst_w[wv][i], w1 = lst_w[wv][i + 1], w2 = lst_w[wv][i + 2], w3 = lst_w[wv][i + 3];
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            const int cc = lane + 64 * c;
            if (cc < g.Ch) {
              const float a0 = vb[o0 + cc], a1 = vb[o1 + cc], a2 = vb[o2 + cc], a3 = vb[o3 + cc];
              acc[c] = fmaf(w0, a0, acc[c]);
              acc[c] = fmaf(w1, a1, acc[c]);
              acc[c] = fmaf(w2, a2, acc[c]);
              acc[c] = fmaf(w3, a3, acc[c]);
            }
          }
        }
        for (; i < nlist; ++i) {
          const int o0 = lst_off[wv][i];
          const float w0 = lst_w[wv][i];
#pragma unroll
          for (int c = 0; c < CPL; ++c) {
            const int cc = lane + 64 * c;
            if (cc < g.Ch) acc[c] = fmaf(w0, vb[o0 + cc], acc[c]);
          }
        }
        wave_lds_sync();
      }
      const int cnt = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps) * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps);
      const float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
#pragma unroll
      for (int c = 0; c < CPL; ++c) acc[c] = cnt > 0 ? acc[c] * inv : 0.f;
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) otile[lane + 64 * c][pi] = acc[c];
  }
  __syncthreads();
  // write the tile: rows of TX pixels per (channel, tile row)
  for (int e = threadIdx.x; e < g.Ch * TY * TX; e += 256) {
    const int c = e / (TY * TX), pi = e % (TY * TX);
    const int y = y0 + pi / TX, x = x0 + pi % TX;
    if (y < g.H && x < g.W)
      out[(((long long)b * g.T + t) * g.C + (long long)hd * g.Ch + c) * g.HW + (long long)y * g.W + x] = otile[c][pi];
  }
}

// Tiled gather for the query stride S_Q = 1 (every pixel is a query).
//
// With S_Q = 1 the contribution of neighbour l of query i to the output
// pixel y = i + p lands at y + disp_l, i.e. at the offset disp_l from y,
// whatever the patch offset p.  So the (slot, offset) bin of a (query,
// neighbour, tap) triple is the same for every pixel the query covers, and
// it is computed once per tile instead of once per covered pixel:
//  * phase 1 (all threads): for the tile's covering queries, softmax over
//    the row, then per neighbour the fixed-point tap weights and the bin of
//    its first tap in an 8 x 8 box of offsets per frame slot, centred on the
//    mean offset of the tile's neighbours in that slot (a neighbour whose
//    taps leave the box, or whose frame is outside the window, is marked
//    for the direct path);
//  * phase 2 (one wave per output row, pixel after pixel): the wave's bins
//    hold the records of the pixel's P x P covering queries (integer
//    atomics: the sums do not depend on the order); moving one pixel along
//    the row removes one query column and adds one, so after the row's first
//    pixel only 2*P*k records change per pixel; each non-empty bin is one
//    position whose channel vector is read once from the channels-last copy
//    of V (lane = channel), in bin order.
namespace aggt {
constexpr int TY = 8, TX = 8;        // output tile; wave w owns tile row w
constexpr int WAVES = TY;
constexpr int NT = WAVES * 64;       // threads per workgroup
constexpr int NSLOT = 7;             // frames per window: 2*wt + 1 <= 7
constexpr int BOX = 8;               // offsets per axis and slot
constexpr int SB = BOX * BOX;        // bins per slot (one per lane)
constexpr int MAXREC = 2048;         // (covering query, neighbour) records per tile
constexpr int MAXQ = 256;            // covering queries per tile
constexpr float QSCALE = 16777216.f; // fixed point 2^24
static_assert(MAXREC <= WAVES * 64 * (TX + 1), "the covering queries' scores fit in the output buffer");
}  // namespace aggt

// floor(a / s) for s > 0 and any sign of a
SNLS_DEV int floor_div(int a, int s) { return a >= 0 ? a / s : -((-a + s - 1) / s); }

// SQ: the query stride when known at compile time (1), else 0 (g.s0).
// GW: bin positions gathered per pass (their channel-vector loads in flight
// together): 4 for patches up to 5 x 5, 2 for larger ones (measured faster
// each way on the 256 x 256 P = 3 and 480 x 854 P = 7 workloads).
template <int SQ, int GW>
__global__ void __launch_bounds__(aggt::NT) aggregate_tile_kernel(const float* __restrict__ vcl,
                                                                  const float* __restrict__ dists,
                                                                  const float* __restrict__ inds, Geo g,
                                                                  float scale, int tiles_x, int tiles_y,
                                                                  float* __restrict__ out) {
  using namespace aggt;
  __shared__ int4 rtap[MAXREC];     // fixed-point tap weights (0,0) (0,1) (1,0) (1,1)
  __shared__ int rcode[MAXREC];     // bin of tap (0,0); -1 nothing; -2 direct path
  __shared__ float qm[MAXQ], qinv[MAXQ];  // softmax max and 1/sum per covering query
  __shared__ int sstat[3 * NSLOT];  // per slot: sum of row offsets, of column offsets, count
  __shared__ int sbase[2 * NSLOT];  // per slot: box origin (row, column offset)
  __shared__ int ndirect;           // records of the tile outside the bin boxes
  __shared__ int bins[WAVES][NSLOT * SB];
  __shared__ float obuf[WAVES][64][TX + 1];

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  // XCD-aware order: each XCD takes a contiguous run of tiles (neighbouring
  // tiles read overlapping V regions, which then stay in that XCD's L2).
  const long long nwg = (long long)gridDim.x;
  const long long xcd = blockIdx.x % 8, xq = nwg / 8, xrem = nwg % 8;
  const long long wg = xcd * xq + (xcd < xrem ? xcd : xrem) + blockIdx.x / 8;
  const long long tiles_img = (long long)tiles_x * tiles_y;
  const int img = (int)(wg / tiles_img);
  const int trem = (int)(wg % tiles_img);
  const int ty = trem / tiles_x, tx = trem % tiles_x;
  const int t = img % g.T, hd = (img / g.T) % g.HD, b = img / (g.T * g.HD);
  const int y0 = ty * TY, x0 = tx * TX;
  const int P = g.ps, K = g.k, nslot = 2 * g.wt + 1, s0 = SQ ? SQ : g.s0;
  // covering queries of the tile: query-grid rows hq0 .. hq0+QY-1 and
  // columns wq0 .. wq0+QX-1 (query m covers pixels m*s0 + lo .. + P-1)
  const int QY = (TY + P - 2) / s0 + 1, QX = (TX + P - 2) / s0 + 1, NQ = QY * QX, NR = NQ * K;
  const int hq0 = floor_div(y0 - g.lo - P + 1 + s0 - 1, s0), wq0 = floor_div(x0 - g.lo - P + 1 + s0 - 1, s0);
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  const long long rowb = (((long long)b * g.HD + hd) * g.T + t) * g.nH;

  for (int i = tid; i < WAVES * NSLOT * SB; i += NT) (&bins[0][0])[i] = 0;
  if (tid < 3 * NSLOT) sstat[tid] = 0;
  if (tid == 0) ndirect = 0;

  // ---- phase 1a: scores of the covering queries (coalesced, into the
  // output buffer, which phase 2 alone uses), softmax statistics ----
  float* const dq = &obuf[0][0][0];
  for (int e = tid; e < NR; e += NT) {
    const int j = e / K, l = e - (e / K) * K;
    const int h = hq0 + j / QX, w = wq0 + j % QX;  // query grid position
    dq[e] = (h >= 0 && h < g.nH && w >= 0 && w < g.nW) ? dists[((rowb + h) * g.nW + w) * K + l] : -INFINITY;
  }
  __syncthreads();
  for (int j = tid; j < NQ; j += NT) {
    const float* d = dq + j * K;
    float m = -INFINITY, z = 0.f;
    for (int l = 0; l < K; ++l)
      if (isfinite(d[l])) m = fmaxf(m, sscale * d[l]);
    for (int l = 0; l < K; ++l)
      if (isfinite(d[l])) z += expf(sscale * d[l] - m);
    qm[j] = m;
    qinv[j] = z > 0.f ? 1.f / z : 0.f;
  }
  __syncthreads();

  // A neighbour's weight (0: contributes nothing) and its position; the
  // same tests as the softmax of the other aggregation kernels.
  // (score from LDS in phase 1, from global memory in phase 2)
  auto neighbour = [&](int e, float& wl, int& t2, int& nh, int& nw, float& ah, float& aw, bool lds) {
    const int j = e / K, l = e - (e / K) * K;
    const int h = hq0 + j / QX, w = wq0 + j % QX;
    wl = 0.f;
    if (qinv[j] == 0.f) return;  // query outside the frame, or no finite score
    const long long row = (rowb + h) * g.nW + w;
    const float d = lds ? dq[e] : dists[row * K + l];
    const float* ind = inds + (row * K + l) * 3;
    const float tf = ind[0], dh = ind[1], dw = ind[2];
    const bool ok = isfinite(d) && tf >= 0.f && tf < (float)g.T && tf == floorf(tf) && fabsf(dh) < kFarDisp &&
                    fabsf(dw) < kFarDisp;
    if (!ok) return;
    wl = expf(sscale * d - qm[j]) * qinv[j];
    t2 = (int)tf;
    const float fh = floorf(dh), fw = floorf(dw);
    nh = (int)fh;
    nw = (int)fw;
    ah = dh - fh;
    aw = dw - fw;
  };

  // ---- phase 1b: mean offset per frame slot (centres the bin boxes) ----
  // per-thread sums per slot, then wave sums and one LDS atomic per wave
  {
    int ssh[NSLOT], ssw[NSLOT], ssc[NSLOT];
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) ssh[s] = ssw[s] = ssc[s] = 0;
    for (int e = tid; e < NR; e += NT) {
      float wl, ah, aw;
      int t2, nh, nw;
      neighbour(e, wl, t2, nh, nw, ah, aw, true);
      const int slot = t2 - t + g.wt;
      // kept for phase 1c: weight, fractions, offsets (16 bits each: an
      // offset beyond them is far outside every bin box), frame slot
      const int ph = min(max(nh, -32768), 32767), pw = min(max(nw, -32768), 32767);
      rtap[e] = make_int4(__float_as_int(wl), __float_as_int(ah), __float_as_int(aw), (ph & 0xffff) | (pw << 16));
      rcode[e] = wl != 0.f ? slot : INT_MIN;
      if (wl != 0.f && slot >= 0 && slot < nslot) {
        const int ch = min(max(nh, -4096), 4096), cw = min(max(nw, -4096), 4096);
#pragma unroll
        for (int s = 0; s < NSLOT; ++s)
          if (slot == s) {
            ssh[s] += ch;
            ssw[s] += cw;
            ssc[s] += 1;
          }
      }
    }
#pragma unroll
    for (int s = 0; s < NSLOT; ++s) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        ssh[s] += __shfl_xor(ssh[s], off);
        ssw[s] += __shfl_xor(ssw[s], off);
        ssc[s] += __shfl_xor(ssc[s], off);
      }
      if (lane == 0 && ssc[s] != 0) {
        atomicAdd(&sstat[s], ssh[s]);
        atomicAdd(&sstat[NSLOT + s], ssw[s]);
        atomicAdd(&sstat[2 * NSLOT + s], ssc[s]);
      }
    }
  }
  __syncthreads();
  if (tid < NSLOT) {
    const int c = sstat[2 * NSLOT + tid];
    sbase[tid] = c ? (int)floorf((float)sstat[tid] / (float)c + 0.5f) - (BOX / 2 - 1) : 0;
    sbase[NSLOT + tid] = c ? (int)floorf((float)sstat[NSLOT + tid] / (float)c + 0.5f) - (BOX / 2 - 1) : 0;
  }
  __syncthreads();

  // ---- phase 1c: records ----
  for (int e = tid; e < NR; e += NT) {
    const int4 st = rtap[e];
    const int slot = rcode[e];
    int code = -1;
    int4 tp = make_int4(0, 0, 0, 0);
    if (slot != INT_MIN) {
      const float wl = __int_as_float(st.x), ah = __int_as_float(st.y), aw = __int_as_float(st.z);
      const int nh = (st.w << 16) >> 16, nw = st.w >> 16;
      const int rh = slot >= 0 && slot < nslot ? nh - sbase[slot] : -1;
      const int rw = slot >= 0 && slot < nslot ? nw - sbase[NSLOT + slot] : -1;
      code = (rh >= 0 && rh < BOX - 1 && rw >= 0 && rw < BOX - 1) ? slot * SB + rh * BOX + rw : -2;
      tp.x = __float2int_rn(wl * (1.f - ah) * (1.f - aw) * QSCALE);
      tp.y = __float2int_rn(wl * (1.f - ah) * aw * QSCALE);
      tp.z = __float2int_rn(wl * ah * (1.f - aw) * QSCALE);
      tp.w = __float2int_rn(wl * ah * aw * QSCALE);
    }
    rcode[e] = code;
    rtap[e] = tp;
    const unsigned long long bd = __ballot(code == -2);
    if (lane == 0 && bd) atomicAdd(&ndirect, __popcll(bd));
  }
  __syncthreads();

  // ---- phase 2: output row wv, pixel after pixel ----
  // The bins of pixel x hold the fixed-point tap weights of the records of
  // its covering queries: query rows ra .. rb of the wave's output row and
  // query columns ca(x) .. cb(x).  Moving along the row, columns leave and
  // enter one at a time, and integer sums do not depend on the order, so the
  // bins slide: only the records of changed columns are added or removed.
  const int y = y0 + wv;
  const float inv_k = 1.f / (float)K;
  const float* vb = vcl + (long long)b * g.T * g.HW * g.C + (long long)hd * g.Ch;
  const int cov_y = cover_count_1d(y, s0, g.nH, g.lo, P);
  const int ra = floor_div(y - g.lo - P + 1 + s0 - 1, s0) - hq0, rb = floor_div(y - g.lo, s0) - hq0;
  const int nrow = rb - ra + 1;  // covering query rows (0 < nrow <= QY)
  const int RK = nrow * K;       // records of one query column
  const float inv_rk = 1.f / (float)max(RK, 1);
  unsigned slots = 0;  // slots with entries in the tile (wave-uniform)
  for (int s = 0; s < nslot; ++s)
    if (sstat[2 * NSLOT + s] != 0) slots |= 1u << s;
  const bool any_direct = ndirect != 0;
  int* const wbins = bins[wv];
  // add (sign +1) or remove (-1) the records of query columns c0 .. c0+nc-1
  auto slide = [&](int c0, int nc, int sign) {
    for (int e0 = 0; e0 < nc * RK; e0 += 64) {
      const int e = e0 + lane;
      const int cc = (int)(((float)e + 0.5f) * inv_rk);
      const int rem = e - cc * RK;
      const int qy = (int)(((float)rem + 0.5f) * inv_k);
      const int l = rem - qy * K;
      const int ri = ((ra + qy) * QX + c0 + cc) * K + l;
      const int code = e < nc * RK ? rcode[ri] : -1;
      if (code >= 0) {
        const int4 tp = rtap[ri];
        if (tp.x) atomicAdd(&wbins[code], sign * tp.x);
        if (tp.y) atomicAdd(&wbins[code + 1], sign * tp.y);
        if (tp.z) atomicAdd(&wbins[code + BOX], sign * tp.z);
        if (tp.w) atomicAdd(&wbins[code + BOX + 1], sign * tp.w);
      }
    }
  };
  int pa = 0, pb = -1;  // query columns in the bins
  for (int px = 0; px < TX; ++px) {
    const int x = x0 + px;
    if (y >= g.H || x >= g.W) break;  // wave-uniform
    float acc = 0.f;
    const int ca = floor_div(x - g.lo - P + 1 + s0 - 1, s0) - wq0, cb = floor_div(x - g.lo, s0) - wq0;
    if constexpr (SQ == 1) {  // columns px .. px+P-1: all P at the first pixel, then one in, one out
      if (px == 0) {
        slide(0, P, 1);
      } else {
        slide(px + P - 1, 1, 1);
        slide(px - 1, 1, -1);
      }
    } else {
      const int add0 = max(pb + 1, ca);
      if (cb >= add0) slide(add0, cb - add0 + 1, 1);
      const int del1 = min(ca - 1, pb);
      if (del1 >= pa) slide(pa, del1 - pa + 1, -1);
      pa = ca;
      pb = cb;
    }
    if (any_direct) {
      // neighbours outside the bin boxes: the whole wave reads their taps directly
      const int ncov = (cb - ca + 1) * RK;
      for (int e0 = 0; e0 < ncov; e0 += 64) {
        const int e = e0 + lane;
        const int cc = (int)(((float)e + 0.5f) * inv_rk);
        const int rem = e - cc * RK;
        const int qy = (int)(((float)rem + 0.5f) * inv_k);
        const int l = rem - qy * K;
        const int ri = ((ra + qy) * QX + ca + cc) * K + l;
        const int code = e < ncov ? rcode[ri] : -1;
        unsigned long long om = __ballot(code == -2);
        while (om) {
          const int src = __ffsll((long long)om) - 1;
          om &= om - 1;
          const int e_ = __builtin_amdgcn_readlane(ri, src);
          float wl, ah, aw;
          int t2, nh, nw;
          neighbour(e_, wl, t2, nh, nw, ah, aw, false);
          const float* vf = vb + (long long)t2 * g.HW * g.C;
#pragma unroll
          for (int eh = 0; eh < 2; ++eh)
#pragma unroll
            for (int ew = 0; ew < 2; ++ew) {
              const int Y = y + nh + eh, X = x + nw + ew;
              const float tw = wl * (eh ? ah : 1.f - ah) * (ew ? aw : 1.f - aw);
              if (Y >= 0 && Y < g.H && X >= 0 && X < g.W && tw != 0.f && lane < g.Ch)
                acc = fmaf(tw, vf[((long long)Y * g.W + X) * g.C + lane], acc);
            }
        }
      }
    }
    wave_lds_sync();
    // non-empty bins in bin order: one channel-vector read per position
    for (int s = 0; s < nslot; ++s) {
      if (!(slots & (1u << s))) continue;
      const int v = wbins[s * SB + lane];
      const int Y = y + sbase[s] + (lane >> 3), X = x + sbase[NSLOT + s] + (lane & 7);
      const bool nz = v != 0 && Y >= 0 && Y < g.H && X >= 0 && X < g.W;
      const int off = ((t + s - g.wt) * (int)g.HW + Y * g.W + X) * g.C;
      const float wgt = (float)v * (1.f / QSCALE);
      unsigned long long m = __ballot(nz);
      // up to GW positions per pass (in bin order), their loads in flight
      // together; the pass's count n is wave-uniform, and a padded slot
      // re-reads the first position and adds nothing
      while (m) {
        int sl[GW];
        int n = 0;
#pragma unroll
        for (int i = 0; i < GW; ++i) {
          sl[i] = m ? __ffsll((long long)m) - 1 : sl[0];
          if (m) {
            m &= m - 1;
            ++n;
          }
        }
        float wv[GW];
        int ov[GW];
#pragma unroll
        for (int i = 0; i < GW; ++i) {
          wv[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wgt), sl[i]));
          ov[i] = __builtin_amdgcn_readlane(off, sl[i]);
        }
        if (lane < g.Ch) {
          float a[GW];
#pragma unroll
          for (int i = 0; i < GW; ++i) a[i] = vb[ov[i] + lane];
#pragma unroll
          for (int i = 0; i < GW; ++i)
            if (i < n) acc = fmaf(wv[i], a[i], acc);
        }
      }
    }
    wave_lds_sync();
    const int cnt = cov_y * cover_count_1d(x, s0, g.nW, g.lo, P);
    obuf[wv][lane][px] = cnt > 0 ? acc * (1.f / (float)cnt) : 0.f;
  }
  // write the row: TX consecutive pixels per channel
  if (y < g.H) {
    const int nx = min(TX, g.W - x0);
    float* ob = out + (((long long)b * g.T + t) * g.C + (long long)hd * g.Ch) * g.HW + (long long)y * g.W + x0;
    for (int e = lane; e < g.Ch * TX; e += 64) {
      const int c = e / TX, px = e % TX;
      if (px < nx) ob[(long long)c * g.HW + px] = obuf[wv][c][px];
    }
  }
}

// (B,T,C,H,W) -> (B,T,HD,H,W,C_h): channels last within each head, so that
// one head's channels of a pixel are contiguous (64 B for 16 channels).
__global__ void __launch_bounds__(256) to_head_channels_last_kernel(const float* __restrict__ v, Geo g,
                                                                    float* __restrict__ vhl) {
  __shared__ float tileb[64][65];
  const long long bt = blockIdx.z;
  const int c0 = blockIdx.y * 64;
  const long long p0 = (long long)blockIdx.x * 64;
  const float* src = v + bt * g.C * g.HW;
  float* dst = vhl + bt * g.C * g.HW;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i;
    const long long p = p0 + tx;
    tileb[i][tx] = (c < g.C && p < g.HW) ? src[(long long)c * g.HW + p] : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const long long p = p0 + i;
    const int c = c0 + tx;
    if (c < g.C && p < g.HW) dst[((long long)(c / g.Ch) * g.HW + p) * g.Ch + c % g.Ch] = tileb[tx][i];
  }
}

// Single-pixel patches (P = 1): a query covers only its own pixel (count 1),
// so the output at a query pixel is the weighted sum of the k bilinear reads
// of its neighbours and every other pixel is 0 (a query stride above 1
// leaves holes).  A workgroup takes an 8 x 8 tile of queries of one (b,
// head, t): one wave per query row reads its scores and positions (lane =
// neighbour, coalesced), forms the softmax weights with wave reductions and
// stores (weight, frame, offsets) per neighbour in LDS as one 16-byte
// record.  The tiles of one (b, head) run in the order (tile
// row, tile column, t), so that the workgroups in flight on an XCD cover a
// band of the frame in every query frame: their neighbours' taps then fall
// in a few MB of V that the XCD's L2 holds, instead of a whole frame per
// query frame.
// Then each thread takes (query, group of 4 channels) pairs -- consecutive
// lanes the channel groups of one query, then the next query -- and reads
// per neighbour four 16-byte pieces of the head-major channels-last V (the
// lanes of a query read one contiguous pixel record per tap).  Each pair
// also clears the other pixels of its S_Q x S_Q cell.
namespace aggp1 {
constexpr int TH = 8, TW = 8;  // query tile (query-grid units)
constexpr int NQ = TH * TW;    // query rows per workgroup
constexpr int KMAX = 60;  // neighbours per row (a wave's lanes; LDS below 64 KB)
// dynamic LDS: NQ rows of k (weight, frame, disp_h, disp_w) records
inline size_t lds_bytes(int k) { return (size_t)NQ * k * 4 * sizeof(float); }
}  // namespace aggp1

__global__ void __launch_bounds__(256) aggregate_p1_kernel(const float* __restrict__ vhl,
                                                           const float* __restrict__ dists,
                                                           const float* __restrict__ inds, Geo g, float scale,
                                                           float* __restrict__ out) {
  using namespace aggp1;
  extern __shared__ float4 nb_s[];  // [NQ][k]: weight (0: skipped), frame, disp_h, disp_w
  const int k = g.k;
  const int tid = threadIdx.x;
  // Consecutive workgroups land on different XCDs (8 per device): give each
  // XCD a contiguous run of tiles, whose neighbours' taps overlap in its L2.
  const long long nwg = (long long)gridDim.x;
  const long long xcd = blockIdx.x % 8, xq = nwg / 8, xrem = nwg % 8;
  const long long wg = xcd * xq + (xcd < xrem ? xcd : xrem) + blockIdx.x / 8;
  const int tqx = (g.nW + TW - 1) / TW, tqy = (g.nH + TH - 1) / TH;
  long long rr = wg;
  const int t = (int)(rr % g.T);
  rr /= g.T;
  const int tx = (int)(rr % tqx);
  rr /= tqx;
  const int ty = (int)(rr % tqy);
  rr /= tqy;
  const int hd = (int)(rr % g.HD);
  const int b = (int)(rr / g.HD);
  const long long rowimg = (((long long)b * g.HD + hd) * g.T + t) * g.nH;
  // query jq of the tile: grid position, whether it exists, its row
  auto qpos = [&](int jq, int& mh, int& mw) {
    mh = ty * TH + jq / TW;
    mw = tx * TW + jq % TW;
    return mh < g.nH && mw < g.nW;
  };
  // softmax weights: one wave per query row, lane = neighbour
  const int lane = tid & 63;
  const float sscale = (g.dist == SNLS_DIST_PROD ? 1.f : -1.f) * scale;
  for (int jq = tid >> 6; jq < NQ; jq += 4) {
    int mh, mw;
    if (!qpos(jq, mh, mw)) continue;  // the same for the whole wave
    const long long row = (rowimg + mh) * g.nW + mw;
    const bool on = lane < k;
    const float d = on ? dists[row * k + lane] : 0.f;
    float tf = 0.f, dh = 0.f, dw = 0.f;
    if (on) {
      tf = inds[(row * k + lane) * 3];
      dh = inds[(row * k + lane) * 3 + 1];
      dw = inds[(row * k + lane) * 3 + 2];
    }
    const bool fin = on && isfinite(d);
    const float x = sscale * d;
    float m = fin ? x : -INFINITY;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const float e = fin ? expf(x - m) : 0.f;
    float z = e;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o);
    const float inv = z > 0.f ? 1.f / z : 0.f;
    const bool ok = fin && tf >= 0.f && tf < (float)g.T && tf == floorf(tf) && fabsf(dh) < kFarDisp &&
                    fabsf(dw) < kFarDisp;
    if (on) nb_s[jq * k + lane] = make_float4(ok ? e * inv : 0.f, tf, dh, dw);
  }
  __syncthreads();
  const int ngrp = g.Ch / 4;
  for (int pr = tid; pr < NQ * ngrp; pr += 256) {
    const int jq = pr / ngrp, cg = pr - jq * ngrp;
    int mh, mw;
    if (!qpos(jq, mh, mw)) continue;
    const int h = mh * g.s0, w = mw * g.s0;
    const float4* nb = &nb_s[jq * k];
    // head plane of V (frame added per neighbour), this thread's 4 channels
    const float* vh = vhl + ((long long)b * g.T * g.HD + hd) * g.HW * g.Ch + 4 * cg;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    // branch-free body (a skipped neighbour reads nothing and adds 0), so
    // the reads of several neighbours are in flight together
#pragma unroll 2
    for (int l = 0; l < k; ++l) {
      const float4 rec = nb[l];
      const float wl = rec.x;
      const bool use = wl != 0.f;
      const float tf = use ? rec.y : 0.f;
      const float dh = use ? rec.z : 0.f, dw = use ? rec.w : 0.f;
      int ny, nx;
      float ay, ax;
      split_disp(dh, &ny, &ay);
      split_disp(dw, &nx, &ax);
      const int y0 = h + ny, x0 = w + nx;
      const float* vb = vh + (long long)(int)tf * g.HD * g.HW * g.Ch;
      const bool y0in = use && y0 >= 0 && y0 < g.H, y1in = use && y0 + 1 >= 0 && y0 + 1 < g.H;
      const bool x0in = x0 >= 0 && x0 < g.W, x1in = x0 + 1 >= 0 && x0 + 1 < g.W;
      const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
      const long long o = ((long long)y0 * g.W + x0) * g.Ch;
      // unconditional 16-byte reads (taps outside the frame read the head
      // plane's first record and are replaced by 0), so the compiler issues
      // four vector loads per neighbour instead of branching per component
      typedef float f32x4 __attribute__((ext_vector_type(4)));
      auto tap4 = [&](bool ok, long long off) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(ok ? vb + off : vh);
        return ok ? make_float4(v.x, v.y, v.z, v.w) : zero;
      };
      const float4 v00 = tap4(y0in && x0in, o);
      const float4 v01 = tap4(y0in && x1in, o + g.Ch);
      const float4 v10 = tap4(y1in && x0in, o + (long long)g.W * g.Ch);
      const float4 v11 = tap4(y1in && x1in, o + (long long)(g.W + 1) * g.Ch);
      auto tap = [&](float a00, float a01, float a10, float a11) {
        const float top = (1.f - ax) * a00 + ax * a01;
        const float bot = (1.f - ax) * a10 + ax * a11;
        return (1.f - ay) * top + ay * bot;
      };
      acc.x = fmaf(wl, tap(v00.x, v01.x, v10.x, v11.x), acc.x);
      acc.y = fmaf(wl, tap(v00.y, v01.y, v10.y, v11.y), acc.y);
      acc.z = fmaf(wl, tap(v00.z, v01.z, v10.z, v11.z), acc.z);
      acc.w = fmaf(wl, tap(v00.w, v01.w, v10.w, v11.w), acc.w);
    }
    float* ob = out + (((long long)b * g.T + t) * g.C + hd * g.Ch + 4 * cg) * g.HW;
    const float res[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* pl = ob + (long long)i * g.HW;
      for (int a = 0; a < g.s0 && h + a < g.H; ++a)
        for (int e = 0; e < g.s0 && w + e < g.W; ++e) pl[(long long)(h + a) * g.W + w + e] = (a | e) ? 0.f : res[i];
    }
  }
}

// Plain per-tap gather for configurations beyond the merged kernel's limits
// (more than 7 frames per window or more than 256 channels per head).
constexpr int kAggChunk = 16;

__global__ void __launch_bounds__(256) aggregate_gather_kernel(const float* __restrict__ v,
                                                               const float* __restrict__ wts,
                                                               const float* __restrict__ inds, Geo g,
                                                               float* __restrict__ out) {
  const int nchunk = (g.Ch + kAggChunk - 1) / kAggChunk;
  long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  long long total = (long long)g.B * g.T * g.HD * nchunk * g.HW;
  if (gid >= total) return;
  int x = (int)(gid % g.W);
  long long r = gid / g.W;
  int y = (int)(r % g.H);
  r /= g.H;
  int chunk = (int)(r % nchunk);
  r /= nchunk;
  int hd = (int)(r % g.HD);
  r /= g.HD;
  int t = (int)(r % g.T);
  int b = (int)(r / g.T);
  const int c0 = hd * g.Ch + chunk * kAggChunk;
  const int nc = min(kAggChunk, g.Ch - chunk * kAggChunk);
  float acc[kAggChunk];
#pragma unroll
  for (int c = 0; c < kAggChunk; ++c) acc[c] = 0.f;
  for (int ph = g.lo; ph < g.lo + g.ps; ++ph) {
    int h = y - ph;
    if (h < 0 || h % g.s0) continue;
    int mh = h / g.s0;
    if (mh >= g.nH) continue;
    for (int pw = g.lo; pw < g.lo + g.ps; ++pw) {
      int w = x - pw;
      if (w < 0 || w % g.s0) continue;
      int mw = w / g.s0;
      if (mw >= g.nW) continue;
      long long row = ((((long long)b * g.HD + hd) * g.T + t) * g.nH + mh) * g.nW + mw;
      for (int l = 0; l < g.k; ++l) {
        const float wl = wts[row * g.k + l];
        if (wl == 0.f) continue;
        const float* ind = inds + (row * g.k + l) * 3;
        float py = (float)y + ind[1], px = (float)x + ind[2];
        if (!(py > -1.f && py < (float)g.H && px > -1.f && px < (float)g.W)) continue;
        int ny, nx;
        float ay, ax;
        split_disp(ind[1], &ny, &ay);
        split_disp(ind[2], &nx, &ax);
        const float* vb = v + (((long long)b * g.T + (int)ind[0]) * g.C + c0) * g.HW;
#pragma unroll
        for (int c = 0; c < kAggChunk; ++c)
          if (c < nc) acc[c] = fmaf(wl, bilinear_plane(vb + c * g.HW, g.H, g.W, y + ny, x + nx, ay, ax), acc[c]);
      }
    }
  }
  int cnt = cover_count_1d(y, g.s0, g.nH, g.lo, g.ps) * cover_count_1d(x, g.s0, g.nW, g.lo, g.ps);
  float inv = cnt > 0 ? 1.f / (float)cnt : 0.f;
  float* ob = out + (((long long)b * g.T + t) * g.C + c0) * g.HW + (long long)y * g.W + x;
#pragma unroll
  for (int c = 0; c < kAggChunk; ++c)
    if (c < nc) ob[c * g.HW] = cnt > 0 ? acc[c] * inv : 0.f;
}

snls_status launch_to_channels_last(const float* x, const Geo& g, float* xcl, hipStream_t s) {
  dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
  if (g.C % 4 == 0 && (long long)g.HW * 4 < (1LL << 31))
    hipLaunchKernelGGL(to_channels_last4_kernel<false>, tgrid, dim3(256), 0, s, x, g, xcl);
  else
    hipLaunchKernelGGL(to_channels_last_kernel, tgrid, dim3(256), 0, s, x, g, xcl);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

snls_status launch_softmax_weights(const float* dists, const float* inds, const Geo& g, float scale, float* wts,
                                   hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  const int G = g.k <= 1 ? 1 : g.k <= 2 ? 2 : g.k <= 4 ? 4 : g.k <= 8 ? 8 : g.k <= 16 ? 16 : g.k <= 32 ? 32 : 64;
  const long long nthr = g.rows * G;
  if ((nthr + 255) / 256 > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
  const dim3 grid((unsigned)((nthr + 255) / 256));
  switch (G) {
#define SNLS_SOFTMAX_CASE(N)                                                                                   \
  case N:                                                                                                      \
    hipLaunchKernelGGL(softmax_weights_kernel<N>, grid, dim3(256), 0, s, dists, inds, g, scale, wts);          \
    break;
    SNLS_SOFTMAX_CASE(1)
    SNLS_SOFTMAX_CASE(2)
    SNLS_SOFTMAX_CASE(4)
    SNLS_SOFTMAX_CASE(8)
    SNLS_SOFTMAX_CASE(16)
    SNLS_SOFTMAX_CASE(32)
    SNLS_SOFTMAX_CASE(64)
#undef SNLS_SOFTMAX_CASE
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

size_t aggregate_ws_bytes(const Geo& g) {
  size_t w = (size_t)g.rows * (size_t)g.k * sizeof(float);
  w = (w + 255) & ~(size_t)255;
  return w + (size_t)g.B * g.T * g.C * g.HW * sizeof(float);
}

snls_status launch_aggregate(const float* v, const float* dists, const float* inds, const Geo& g, float scale,
                             float* out, void* ws, hipStream_t s) {
  if (g.rows == 0) return SNLS_OK;
  float* wts = static_cast<float*>(ws);
  size_t woff = ((size_t)g.rows * g.k * sizeof(float) + 255) & ~(size_t)255;
  float* vcl = reinterpret_cast<float*>(static_cast<char*>(ws) + woff);
  const int nslot = 2 * g.wt + 1;
  if (g.ps == 1 && g.Ch % 4 == 0 && g.k <= aggp1::KMAX) {
    // single-pixel patches: per-query gather, holes cleared
    const long long nblk = (long long)g.B * g.HD * g.T * ((g.nH + aggp1::TH - 1) / aggp1::TH) *
                           ((g.nW + aggp1::TW - 1) / aggp1::TW);
    if (nblk > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
    dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
    if (g.C % 4 == 0 && (long long)g.HW * 4 < (1LL << 31))
      hipLaunchKernelGGL(to_channels_last4_kernel<true>, tgrid, dim3(256), 0, s, v, g, vcl);
    else
      hipLaunchKernelGGL(to_head_channels_last_kernel, tgrid, dim3(256), 0, s, v, g, vcl);
    hipLaunchKernelGGL(aggregate_p1_kernel, dim3((unsigned)nblk), dim3(256), aggp1::lds_bytes(g.k), s, vcl, dists,
                       inds, g, scale, out);
    return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
  }
  // merged kernel limits: frames per window, channels per head, 32-bit
  // offsets inside one batch entry, per-bin weight sums below 2^31 in 2^-24
  // fixed point (at most P^2 <= 121 covering patches)
  const long long nq_tile =
      (long long)((aggt::TY + g.ps - 2) / g.s0 + 1) * ((aggt::TX + g.ps - 2) / g.s0 + 1);  // covering queries
  if (nslot <= aggt::NSLOT && g.Ch <= 64 && (long long)g.T * g.HW * g.C < (1LL << 31) &&
      g.ps <= 11 && nq_tile <= aggt::MAXQ && nq_tile * g.k <= aggt::MAXREC) {
    dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
    if (g.C % 4 == 0 && (long long)g.HW * 4 < (1LL << 31))
      hipLaunchKernelGGL(to_channels_last4_kernel<false>, tgrid, dim3(256), 0, s, v, g, vcl);
    else
      hipLaunchKernelGGL(to_channels_last_kernel, tgrid, dim3(256), 0, s, v, g, vcl);
    const int tiles_x = (g.W + aggt::TX - 1) / aggt::TX, tiles_y = (g.H + aggt::TY - 1) / aggt::TY;
    const long long nwg = (long long)tiles_x * tiles_y * g.B * g.T * g.HD;
    if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
#define SNLS_AGGT(SQ, GW)                                                                                    \
  hipLaunchKernelGGL((aggregate_tile_kernel<SQ, GW>), dim3((unsigned)nwg), dim3(aggt::NT), 0, s, vcl, dists, inds, \
                     g, scale, tiles_x, tiles_y, out)
    if (g.s0 == 1) {
      if (g.ps <= 5) SNLS_AGGT(1, 4);
      else SNLS_AGGT(1, 2);
    } else {
      if (g.ps <= 5) SNLS_AGGT(0, 4);
      else SNLS_AGGT(0, 2);
    }
#undef SNLS_AGGT
    return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
  }
  {
    const snls_status st = launch_softmax_weights(dists, inds, g, scale, wts, s);
    if (st != SNLS_OK) return st;
  }
  if (nslot <= agg::NSLOT && g.Ch <= 256 && (long long)g.T * g.HW * g.C < (1LL << 31) && g.ps <= 11) {
    dim3 tgrid((unsigned)((g.HW + 63) / 64), (unsigned)((g.C + 63) / 64), (unsigned)(g.B * g.T));
    if (g.C % 4 == 0 && (long long)g.HW * 4 < (1LL << 31))
      hipLaunchKernelGGL(to_channels_last4_kernel<false>, tgrid, dim3(256), 0, s, v, g, vcl);
    else
      hipLaunchKernelGGL(to_channels_last_kernel, tgrid, dim3(256), 0, s, v, g, vcl);
    const int tiles_x = (g.W + agg::TX - 1) / agg::TX, tiles_y = (g.H + agg::TY - 1) / agg::TY;
    const long long nwg = (long long)tiles_x * tiles_y * g.B * g.T * g.HD;
    if (nwg > 0x7fffffffLL) return SNLS_ERR_UNSUPPORTED;
    const int cpl = (g.Ch + 63) / 64;
    if (cpl == 1)
      hipLaunchKernelGGL(aggregate_merged_kernel<1>, dim3((unsigned)nwg), dim3(256), 0, s, vcl, wts, inds, g,
                         tiles_x, tiles_y, out);
    else if (cpl == 2)
      hipLaunchKernelGGL(aggregate_merged_kernel<2>, dim3((unsigned)nwg), dim3(256), 0, s, vcl, wts, inds, g,
                         tiles_x, tiles_y, out);
    else
      hipLaunchKernelGGL(aggregate_merged_kernel<4>, dim3((unsigned)nwg), dim3(256), 0, s, vcl, wts, inds, g,
                         tiles_x, tiles_y, out);
  } else {
    const int nchunk = (g.Ch + kAggChunk - 1) / kAggChunk;
    long long total = (long long)g.B * g.T * g.HD * nchunk * g.HW;
    hipLaunchKernelGGL(aggregate_gather_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, v, wts, inds,
                       g, out);
  }
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

/*
 * snls_oracle.c -- oracle for the Shifted Non-Local Search path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow reference that the
 * HIP library is checked against.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it; the product path never
 * does.  It shares no source with the HIP library.
 *
 * Written from "Space-Time Attention with Shifted Non-Local Search"
 * (Gauen & Chan, ICLR 2024), Section 3.1 (non-local search, the patch sum
 * with query stride) and Section 3.2 (the shifted window, the output offsets,
 * top-L, the temporal window W_t, the key stride S_K, bilinear indexing and
 * the weighted patch aggregation).  Appendix "Pytorch Example" fixes the
 * tensor layouts (B,T,F,H,W), the head split (hd f) and the inds shape.
 *
 * Every sum is accumulated in double precision.  Candidate displacements are
 * formed, by default, with the fp32 convention of the library's outputs
 * (disp = fl32(delta + fl32(S_K * (d - r)))); with fp32_positions = 0 they
 * are exact doubles, which the finite-difference checks of the backward pass
 * need.
 *
 * Readings of the paper that the code takes (listed with reasons in the
 * design notes of the repository):
 *  - window offsets are S_K*(d - floor(Ws/2)), d = 0..Ws-1, patch offsets
 *    p = -floor(P/2) .. P-1-floor(P/2)  (Sec. 3.1 writes Ws/2 and P/2);
 *  - the query patch is Q[t, h+p_h, w+p_w] (Sec. 3.2 drops the +p on Q, a
 *    typo against the Sec. 3.1 sum);
 *  - searched frames are t-wt .. t+wt, the query frame included with zero
 *    offset; frames outside [0,T) are skipped (invalid);
 *  - flows hold one (dh, dw) offset per neighbour slot, read at the query
 *    centre; slot order dt = -wt..-1, +1..+wt;
 *  - bilinear sampling with pixel centres on integers, taps outside the frame
 *    read 0, query patch pixels outside the frame are skipped;
 *  - a candidate whose centre lies outside [0,H-1]x[0,W-1] is invalid and
 *    scores -inf (inner product) or +inf (squared L2); so does a candidate
 *    whose similarity is not a number (non-finite inputs), so that every
 *    score is ordered;
 *  - top-k is joint over all frames of the window, best first, ties to the
 *    smaller candidate id ((dt+wt)*Ws + dh)*Ws + dw;
 *  - aggregation weights are softmax(sign*scale*d) over the k entries
 *    (sign +1 for inner product, -1 for L2), entries with non-finite d get
 *    weight 0; every in-frame output pixel is divided by the number of query
 *    patches that cover it, pixels that no patch covers are 0.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int B, T, C, H, W, HD;
  int ws, wt, ps, stride0;
  double stride1;
  int k;
  int dist_type;       /* 0: inner product (larger is better), 1: squared L2 */
  int fp32_positions;  /* 1: fp32 displacement convention, 0: exact double */
} oracle_params;

/* ---- indexing of the tensors (layouts from the appendix example) ---- */

static int64_t vid_index(const oracle_params* p, int b, int t, int c, int y, int x) {
  return ((((int64_t)b * p->T + t) * p->C + c) * p->H + y) * (int64_t)p->W + x;
}

/* flows: (B, T, 2*wt, 2, H, W); component 0 = row offset, 1 = column offset */
static int64_t flow_index(const oracle_params* p, int b, int t, int slot, int comp, int y, int x) {
  return (((((int64_t)b * p->T + t) * (2 * p->wt) + slot) * 2 + comp) * p->H + y) * (int64_t)p->W + x;
}

/* neighbour slot of a frame step dt != 0: dt = -wt..-1 -> 0..wt-1, dt = 1..wt -> wt..2wt-1 */
static int flow_slot(const oracle_params* p, int dt) { return dt < 0 ? dt + p->wt : dt + p->wt - 1; }

static int grid_h(const oracle_params* p) { return (p->H - 1) / p->stride0 + 1; }
static int grid_w(const oracle_params* p) { return (p->W - 1) / p->stride0 + 1; }
static int n_cand(const oracle_params* p) { return (2 * p->wt + 1) * p->ws * p->ws; }
static int patch_lo(const oracle_params* p) { return -(p->ps / 2); }

/* Decompose a flattened query index over (b, hd, t, m_h, m_w). */
static void query_coords(const oracle_params* p, int64_t qi, int* b, int* hd, int* t, int* h, int* w) {
  int nH = grid_h(p), nW = grid_w(p);
  int mw = (int)(qi % nW); qi /= nW;
  int mh = (int)(qi % nH); qi /= nH;
  *t = (int)(qi % p->T); qi /= p->T;
  *hd = (int)(qi % p->HD); qi /= p->HD;
  *b = (int)qi;
  *h = mh * p->stride0;
  *w = mw * p->stride0;
}

/* Offset of the search window centre from the query for frame step dt
 * (Sec. 3.2: the predicted offset F_in at the query's own coordinate; the
 * query frame itself is searched with zero offset). */
static double shift_of(const double* flows, const oracle_params* p, int b, int t, int dt, int comp, int h, int w) {
  if (dt == 0) return 0.0;
  return flows[flow_index(p, b, t, flow_slot(p, dt), comp, h, w)];
}

/* Displacement of grid cell d from the query: shift + S_K*(d - floor(Ws/2))
 * (Sec. 3.2, key stride). */
static double displacement(const oracle_params* p, double shift, int d) {
  int r = p->ws / 2;
  if (p->fp32_positions) {
    float off = (float)p->stride1 * (float)(d - r);
    float disp = (float)shift + off;
    return (double)disp;
  }
  return shift + p->stride1 * (double)(d - r);
}

/* Bilinear read of channel c of frame (b,t) of X at real position (y, x)
 * (Sec. 3.2, "bilinear interpolation is used for efficient indexing").
 * Pixel centres sit on integer coordinates; taps outside the frame read 0. */
static double bilinear(const double* X, const oracle_params* p, int b, int t, int c, double y, double x) {
  if (!(y > -1.0 && y < (double)p->H && x > -1.0 && x < (double)p->W)) return 0.0;
  double y0 = floor(y), x0 = floor(x);
  double ay = y - y0, ax = x - x0;
  double s = 0.0;
  for (int ey = 0; ey < 2; ey++) {
    for (int ex = 0; ex < 2; ex++) {
      int yy = (int)y0 + ey, xx = (int)x0 + ex;
      if (yy < 0 || yy >= p->H || xx < 0 || xx >= p->W) continue;
      double wgt = (ey ? ay : 1.0 - ay) * (ex ? ax : 1.0 - ax);
      s += wgt * X[vid_index(p, b, t, c, yy, xx)];
    }
  }
  return s;
}

/* Partial derivatives of the bilinear read with respect to y and x, taken on
 * the cell with corner (floor(y), floor(x)). */
static void bilinear_grad(const double* X, const oracle_params* p, int b, int t, int c, double y, double x,
                          double* dy, double* dx) {
  *dy = 0.0; *dx = 0.0;
  if (!(y > -1.0 && y < (double)p->H && x > -1.0 && x < (double)p->W)) return;
  double y0 = floor(y), x0 = floor(x);
  double ay = y - y0, ax = x - x0;
  for (int ey = 0; ey < 2; ey++) {
    for (int ex = 0; ex < 2; ex++) {
      int yy = (int)y0 + ey, xx = (int)x0 + ex;
      if (yy < 0 || yy >= p->H || xx < 0 || xx >= p->W) continue;
      double val = X[vid_index(p, b, t, c, yy, xx)];
      *dy += (ey ? 1.0 : -1.0) * (ex ? ax : 1.0 - ax) * val;
      *dx += (ey ? ay : 1.0 - ay) * (ex ? 1.0 : -1.0) * val;
    }
  }
}

/* Adjoint of the bilinear read: add val * tap weight into each in-frame tap. */
static void bilinear_scatter(double* G, const oracle_params* p, int b, int t, int c, double y, double x, double val) {
  if (!(y > -1.0 && y < (double)p->H && x > -1.0 && x < (double)p->W)) return;
  double y0 = floor(y), x0 = floor(x);
  double ay = y - y0, ax = x - x0;
  for (int ey = 0; ey < 2; ey++) {
    for (int ex = 0; ex < 2; ex++) {
      int yy = (int)y0 + ey, xx = (int)x0 + ex;
      if (yy < 0 || yy >= p->H || xx < 0 || xx >= p->W) continue;
      double wgt = (ey ? ay : 1.0 - ay) * (ex ? ax : 1.0 - ax);
      G[vid_index(p, b, t, c, yy, xx)] += wgt * val;
    }
  }
}

/* Patch similarity of the query at (b, t, h, w) in head hd against frame tk at
 * displacement (dh, dw) (Sec. 3.1 / 3.2 similarity sum over the patch and the
 * head's channels).  Query patch pixels outside the frame are skipped. */
static double similarity(const double* q, const double* k, const oracle_params* p, int b, int hd, int t,
                         int h, int w, int tk, double disp_h, double disp_w) {
  int Ch = p->C / p->HD, lo = patch_lo(p);
  double d = 0.0;
  for (int ph = lo; ph < lo + p->ps; ph++) {
    for (int pw = lo; pw < lo + p->ps; pw++) {
      int yq = h + ph, xq = w + pw;
      if (yq < 0 || yq >= p->H || xq < 0 || xq >= p->W) continue;
      double yk = (double)yq + disp_h, xk = (double)xq + disp_w;
      for (int c = hd * Ch; c < (hd + 1) * Ch; c++) {
        double qv = q[vid_index(p, b, t, c, yq, xq)];
        double kv = bilinear(k, p, b, tk, c, yk, xk);
        if (p->dist_type == 0) d += qv * kv;
        else d += (qv - kv) * (qv - kv);
      }
    }
  }
  return d;
}

static int centre_in_frame(const oracle_params* p, int h, int w, double disp_h, double disp_w) {
  double yc = (double)h + disp_h, xc = (double)w + disp_w;
  return yc >= 0.0 && yc <= (double)(p->H - 1) && xc >= 0.0 && xc <= (double)(p->W - 1);
}

/* Full search for a list of queries: every candidate of the W_t x Ws x Ws
 * window in candidate-id order.  dists: nq x n_cand, inds: nq x n_cand x 3
 * holding (frame, disp_h, disp_w); invalid candidates score -inf / +inf. */
void oracle_search(const double* q, const double* k, const double* flows, const oracle_params* p,
                   const int64_t* qids, int64_t nq, double* dists, double* inds) {
  int nc = n_cand(p);
  double bad = p->dist_type == 0 ? -INFINITY : INFINITY;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t i = 0; i < nq; i++) {
    int b, hd, t, h, w;
    query_coords(p, qids[i], &b, &hd, &t, &h, &w);
    for (int dt = -p->wt; dt <= p->wt; dt++) {
      int tk = t + dt;
      double sh = shift_of(flows, p, b, t, dt, 0, h, w);
      double sw = shift_of(flows, p, b, t, dt, 1, h, w);
      for (int dh = 0; dh < p->ws; dh++) {
        for (int dw = 0; dw < p->ws; dw++) {
          int id = ((dt + p->wt) * p->ws + dh) * p->ws + dw;
          double disp_h = displacement(p, sh, dh), disp_w = displacement(p, sw, dw);
          int64_t o = i * nc + id;
          inds[3 * o + 0] = (double)tk;
          inds[3 * o + 1] = disp_h;
          inds[3 * o + 2] = disp_w;
          if (tk < 0 || tk >= p->T || !centre_in_frame(p, h, w, disp_h, disp_w)) {
            dists[o] = bad;
          } else {
            double d = similarity(q, k, p, b, hd, t, h, w, tk, disp_h, disp_w);
            dists[o] = isnan(d) ? bad : d;
          }
        }
      }
    }
  }
}

typedef struct { double d; int id; } scored;

static int better_ip(const void* a, const void* b) {
  const scored* x = (const scored*)a; const scored* y = (const scored*)b;
  if (x->d > y->d) return -1;
  if (x->d < y->d) return 1;
  return x->id - y->id;
}

static int better_l2(const void* a, const void* b) {
  const scored* x = (const scored*)a; const scored* y = (const scored*)b;
  if (x->d < y->d) return -1;
  if (x->d > y->d) return 1;
  return x->id - y->id;
}

/* top-L of each row (Sec. 3.2): the kk best columns, best first, ties to the
 * smaller column id.  out_d: rows x kk, out_id: rows x kk. */
void oracle_topk(const double* dists, int64_t rows, int ncols, int kk, int dist_type, double* out_d, int64_t* out_id) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; r++) {
    scored* s = (scored*)malloc(sizeof(scored) * (size_t)ncols);
    for (int j = 0; j < ncols; j++) { s[j].d = dists[r * ncols + j]; s[j].id = j; }
    qsort(s, (size_t)ncols, sizeof(scored), dist_type == 0 ? better_ip : better_l2);
    for (int j = 0; j < kk; j++) { out_d[r * kk + j] = s[j].d; out_id[r * kk + j] = s[j].id; }
    free(s);
  }
}

/* Softmax over one row of k distances (Sec. 3.2 aggregation, sigma(S_L)):
 * w_l = exp(s_l - max) / sum, s_l = sign * scale * d_l; non-finite d -> 0. */
static void softmax_row(const double* d, int kk, int dist_type, double scale, double* wout) {
  double sign = dist_type == 0 ? 1.0 : -1.0, m = -INFINITY, z = 0.0;
  for (int l = 0; l < kk; l++) if (isfinite(d[l]) && sign * scale * d[l] > m) m = sign * scale * d[l];
  for (int l = 0; l < kk; l++) {
    wout[l] = isfinite(d[l]) ? exp(sign * scale * d[l] - m) : 0.0;
    z += wout[l];
  }
  for (int l = 0; l < kk; l++) wout[l] = z > 0.0 ? wout[l] / z : 0.0;
}

/* Frame of a stored neighbour; -1 when it is not an integer inside [0,T). */
static int neighbour_frame(const oracle_params* p, double tf) {
  if (!(tf >= 0.0 && tf < (double)p->T) || tf != floor(tf)) return -1;
  return (int)tf;
}

/* Weighted patch aggregation (Sec. 3.2, "Aggregation"), literal scatter
 * form: the output starts at zero, each query adds its softmax-weighted
 * neighbour patches pixel by pixel, then every pixel is divided by the number
 * of query patches that covered it.  dists: (B,HD,T,nH,nW,k), inds: (...,k,3),
 * out: (B,T,C,H,W). */
void oracle_aggregate(const double* v, const double* dists, const double* inds, const oracle_params* p,
                      double scale, double* out) {
  int nH = grid_h(p), nW = grid_w(p), Ch = p->C / p->HD, lo = patch_lo(p), kk = p->k;
  int64_t nvid = (int64_t)p->B * p->T * p->C * p->H * p->W;
  double* cnt = (double*)calloc((size_t)p->B * p->T * p->H * p->W, sizeof(double));
  double* wts = (double*)malloc(sizeof(double) * (size_t)kk);
  memset(out, 0, sizeof(double) * (size_t)nvid);
  for (int b = 0; b < p->B; b++)
    for (int t = 0; t < p->T; t++)
      for (int mh = 0; mh < nH; mh++)
        for (int mw = 0; mw < nW; mw++) {
          int h = mh * p->stride0, w = mw * p->stride0;
          for (int ph = lo; ph < lo + p->ps; ph++)
            for (int pw = lo; pw < lo + p->ps; pw++) {
              int y = h + ph, x = w + pw;
              if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
              cnt[(((int64_t)b * p->T + t) * p->H + y) * p->W + x] += 1.0;
            }
          for (int hd = 0; hd < p->HD; hd++) {
            int64_t row = ((((int64_t)b * p->HD + hd) * p->T + t) * nH + mh) * nW + mw;
            softmax_row(dists + row * kk, kk, p->dist_type, scale, wts);
            for (int l = 0; l < kk; l++) {
              if (wts[l] == 0.0) continue;
              const double* ind = inds + 3 * (row * kk + l);
              int tk = neighbour_frame(p, ind[0]);
              if (tk < 0) continue;
              for (int ph = lo; ph < lo + p->ps; ph++)
                for (int pw = lo; pw < lo + p->ps; pw++) {
                  int y = h + ph, x = w + pw;
                  if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
                  for (int c = hd * Ch; c < (hd + 1) * Ch; c++)
                    out[vid_index(p, b, t, c, y, x)] +=
                        wts[l] * bilinear(v, p, b, tk, c, (double)y + ind[1], (double)x + ind[2]);
                }
            }
          }
        }
  for (int b = 0; b < p->B; b++)
    for (int t = 0; t < p->T; t++)
      for (int c = 0; c < p->C; c++)
        for (int y = 0; y < p->H; y++)
          for (int x = 0; x < p->W; x++) {
            double n = cnt[(((int64_t)b * p->T + t) * p->H + y) * p->W + x];
            int64_t o = vid_index(p, b, t, c, y, x);
            out[o] = n > 0.0 ? out[o] / n : 0.0;
          }
  free(wts);
  free(cnt);
}

/* The same aggregation evaluated at a list of output pixels, one at a time:
 * for pixel (b,t,y,x) visit every query patch that covers it.  pix: npix
 * flattened (b,t,y,x) indices; out: npix x C. */
void oracle_aggregate_at(const double* v, const double* dists, const double* inds, const oracle_params* p,
                         double scale, const int64_t* pix, int64_t npix, double* out) {
  int nH = grid_h(p), nW = grid_w(p), Ch = p->C / p->HD, lo = patch_lo(p), kk = p->k;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t i = 0; i < npix; i++) {
    double* wts = (double*)malloc(sizeof(double) * (size_t)kk);
    int64_t r = pix[i];
    int x = (int)(r % p->W); r /= p->W;
    int y = (int)(r % p->H); r /= p->H;
    int t = (int)(r % p->T); r /= p->T;
    int b = (int)r;
    double n = 0.0;
    double* acc = out + i * p->C;
    for (int c = 0; c < p->C; c++) acc[c] = 0.0;
    for (int ph = lo; ph < lo + p->ps; ph++)
      for (int pw = lo; pw < lo + p->ps; pw++) {
        int h = y - ph, w = x - pw;
        if (h < 0 || w < 0 || h % p->stride0 || w % p->stride0) continue;
        int mh = h / p->stride0, mw = w / p->stride0;
        if (mh >= nH || mw >= nW) continue;
        n += 1.0;
        for (int hd = 0; hd < p->HD; hd++) {
          int64_t row = ((((int64_t)b * p->HD + hd) * p->T + t) * nH + mh) * nW + mw;
          softmax_row(dists + row * kk, kk, p->dist_type, scale, wts);
          for (int l = 0; l < kk; l++) {
            if (wts[l] == 0.0) continue;
            const double* ind = inds + 3 * (row * kk + l);
            int tk = neighbour_frame(p, ind[0]);
            if (tk < 0) continue;
            for (int c = hd * Ch; c < (hd + 1) * Ch; c++)
              acc[c] += wts[l] * bilinear(v, p, b, tk, c, (double)y + ind[1], (double)x + ind[2]);
          }
        }
      }
    for (int c = 0; c < p->C; c++) acc[c] = n > 0.0 ? acc[c] / n : 0.0;
    free(wts);
  }
}

/* Search distances and displacements for a fixed choice of candidates:
 * sel holds, per query row and neighbour, (dt, d_h, d_w) with the window
 * cells d in 0..Ws-1.  Used to evaluate the forward map at a fixed top-k set
 * (the set itself is piecewise constant; Sec. 3.2 notes top-L is not
 * differentiable).  dists: rows x k, inds: rows x k x 3. */
void oracle_search_fixed(const double* q, const double* k, const double* flows, const oracle_params* p,
                         const int32_t* sel, double* dists, double* inds) {
  int64_t rows = (int64_t)p->B * p->HD * p->T * grid_h(p) * grid_w(p);
  double bad = p->dist_type == 0 ? -INFINITY : INFINITY;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < rows; i++) {
    int b, hd, t, h, w;
    query_coords(p, i, &b, &hd, &t, &h, &w);
    for (int l = 0; l < p->k; l++) {
      const int32_t* s = sel + 3 * (i * p->k + l);
      int dt = s[0], tk = t + dt;
      double disp_h = displacement(p, shift_of(flows, p, b, t, dt, 0, h, w), s[1]);
      double disp_w = displacement(p, shift_of(flows, p, b, t, dt, 1, h, w), s[2]);
      int64_t o = i * p->k + l;
      inds[3 * o + 0] = (double)tk;
      inds[3 * o + 1] = disp_h;
      inds[3 * o + 2] = disp_w;
      if (tk < 0 || tk >= p->T || !centre_in_frame(p, h, w, disp_h, disp_w)) dists[o] = bad;
      else dists[o] = similarity(q, k, p, b, hd, t, h, w, tk, disp_h, disp_w);
    }
  }
}

/* Backward pass (the differentiable search and aggregation of Sec. 1 and
 * Sec. 3.2), by the chain rule through aggregation, softmax, similarity and
 * the bilinear reads, for the selected candidates (the top-k set is held
 * constant).  grad_out: (B,T,C,H,W); grad_dists: (B,HD,T,nH,nW,k) or NULL.
 * Every gradient array is overwritten.  grad_flows: (B,T,2wt,2,H,W).
 *
 * The query rows are split over OpenMP threads; each thread adds its rows'
 * terms into gradient arrays of its own, which are summed in thread order at
 * the end (the per-row arithmetic is the same as in a single pass). */
static void backward_row(const double* q, const double* k, const double* v, const double* dists,
                         const double* inds, const double* grad_out, const double* grad_dists,
                         const oracle_params* p, double scale, const double* cnt, int64_t row, double* wts,
                         double* G, double* grad_q, double* grad_k, double* grad_v, double* grad_flows) {
  int Ch = p->C / p->HD, lo = patch_lo(p), kk = p->k;
  double sign = p->dist_type == 0 ? 1.0 : -1.0;
  int b, hd, t, h, w;
  query_coords(p, row, &b, &hd, &t, &h, &w);
  softmax_row(dists + row * kk, kk, p->dist_type, scale, wts);
  /* aggregation: out = sum_l w_l vtilde_l / cnt */
  for (int l = 0; l < kk; l++) {
    G[l] = 0.0;
    const double* ind = inds + 3 * (row * kk + l);
    int tk = neighbour_frame(p, ind[0]);
    if (tk < 0 || !isfinite(dists[row * kk + l])) continue;
    double ddisp_h = 0.0, ddisp_w = 0.0;
    for (int ph = lo; ph < lo + p->ps; ph++)
      for (int pw = lo; pw < lo + p->ps; pw++) {
        int y = h + ph, x = w + pw;
        if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
        double n = cnt[(((int64_t)b * p->T + t) * p->H + y) * p->W + x];
        double yv = (double)y + ind[1], xv = (double)x + ind[2];
        for (int c = hd * Ch; c < (hd + 1) * Ch; c++) {
          double g = grad_out[vid_index(p, b, t, c, y, x)] / n;
          G[l] += g * bilinear(v, p, b, tk, c, yv, xv);
          bilinear_scatter(grad_v, p, b, tk, c, yv, xv, wts[l] * g);
          double gy, gx;
          bilinear_grad(v, p, b, tk, c, yv, xv, &gy, &gx);
          ddisp_h += wts[l] * g * gy;
          ddisp_w += wts[l] * g * gx;
        }
      }
    if (tk != t) {
      int slot = flow_slot(p, tk - t);
      grad_flows[flow_index(p, b, t, slot, 0, h, w)] += ddisp_h;
      grad_flows[flow_index(p, b, t, slot, 1, h, w)] += ddisp_w;
    }
  }
  /* softmax backward, then the similarity of each selected candidate */
  double wg = 0.0;
  for (int l = 0; l < kk; l++) wg += wts[l] * G[l];
  for (int l = 0; l < kk; l++) {
    const double* ind = inds + 3 * (row * kk + l);
    int tk = neighbour_frame(p, ind[0]);
    if (tk < 0 || !isfinite(dists[row * kk + l])) continue;
    double dd = sign * scale * wts[l] * (G[l] - wg);
    if (grad_dists) dd += grad_dists[row * kk + l];
    if (dd == 0.0) continue;
    double ddisp_h = 0.0, ddisp_w = 0.0;
    for (int ph = lo; ph < lo + p->ps; ph++)
      for (int pw = lo; pw < lo + p->ps; pw++) {
        int y = h + ph, x = w + pw;
        if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
        double yk = (double)y + ind[1], xk = (double)x + ind[2];
        for (int c = hd * Ch; c < (hd + 1) * Ch; c++) {
          double qv = q[vid_index(p, b, t, c, y, x)];
          double kv = bilinear(k, p, b, tk, c, yk, xk);
          double dq, dkv;
          if (p->dist_type == 0) { dq = dd * kv; dkv = dd * qv; }
          else { dq = 2.0 * dd * (qv - kv); dkv = -2.0 * dd * (qv - kv); }
          grad_q[vid_index(p, b, t, c, y, x)] += dq;
          bilinear_scatter(grad_k, p, b, tk, c, yk, xk, dkv);
          double gy, gx;
          bilinear_grad(k, p, b, tk, c, yk, xk, &gy, &gx);
          ddisp_h += dkv * gy;
          ddisp_w += dkv * gx;
        }
      }
    if (tk != t) {
      int slot = flow_slot(p, tk - t);
      grad_flows[flow_index(p, b, t, slot, 0, h, w)] += ddisp_h;
      grad_flows[flow_index(p, b, t, slot, 1, h, w)] += ddisp_w;
    }
  }
}

void oracle_backward(const double* q, const double* k, const double* v, const double* flows,
                     const double* dists, const double* inds, const double* grad_out, const double* grad_dists,
                     const oracle_params* p, double scale, double* grad_q, double* grad_k, double* grad_v,
                     double* grad_flows) {
  int nH = grid_h(p), nW = grid_w(p), lo = patch_lo(p), kk = p->k;
  int64_t nvid = (int64_t)p->B * p->T * p->C * p->H * p->W;
  int64_t nflow = (int64_t)p->B * p->T * 2 * p->wt * 2 * p->H * p->W;
  int64_t rows = (int64_t)p->B * p->HD * p->T * nH * nW;
  (void)flows;
  memset(grad_q, 0, sizeof(double) * (size_t)nvid);
  memset(grad_k, 0, sizeof(double) * (size_t)nvid);
  memset(grad_v, 0, sizeof(double) * (size_t)nvid);
  memset(grad_flows, 0, sizeof(double) * (size_t)nflow);

  /* number of query patches covering each pixel */
  double* cnt = (double*)calloc((size_t)p->B * p->T * p->H * p->W, sizeof(double));
  for (int b = 0; b < p->B; b++)
    for (int t = 0; t < p->T; t++)
      for (int mh = 0; mh < nH; mh++)
        for (int mw = 0; mw < nW; mw++)
          for (int ph = lo; ph < lo + p->ps; ph++)
            for (int pw = lo; pw < lo + p->ps; pw++) {
              int y = mh * p->stride0 + ph, x = mw * p->stride0 + pw;
              if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
              cnt[(((int64_t)b * p->T + t) * p->H + y) * p->W + x] += 1.0;
            }

  /* private gradient arrays: at most about 8 GB of them in total */
  int64_t per_thread = (3 * nvid + nflow) * (int64_t)sizeof(double);
  int nthr = omp_get_max_threads();
  int64_t cap = per_thread > 0 ? (int64_t)8000000000LL / per_thread : nthr;
  if (cap < 1) cap = 1;
  if (nthr > cap) nthr = (int)cap;
  if ((int64_t)nthr > rows) nthr = rows > 0 ? (int)rows : 1;
  double** priv = (double**)calloc((size_t)nthr, sizeof(double*));
  int used = 1;
#pragma omp parallel num_threads(nthr)
  {
    int tid = omp_get_thread_num();
#pragma omp single
    used = omp_get_num_threads();
    /* thread 0 adds straight into the outputs */
    double* buf = tid == 0 ? NULL : (double*)calloc((size_t)(3 * nvid + nflow), sizeof(double));
    double* gq = tid == 0 ? grad_q : buf;
    double* gk = tid == 0 ? grad_k : buf + nvid;
    double* gv = tid == 0 ? grad_v : buf + 2 * nvid;
    double* gf = tid == 0 ? grad_flows : buf + 3 * nvid;
    priv[tid] = buf;
    double* wts = (double*)malloc(sizeof(double) * (size_t)(kk > 0 ? kk : 1));
    double* G = (double*)malloc(sizeof(double) * (size_t)(kk > 0 ? kk : 1));
#pragma omp for schedule(static)
    for (int64_t row = 0; row < rows; row++)
      backward_row(q, k, v, dists, inds, grad_out, grad_dists, p, scale, cnt, row, wts, G, gq, gk, gv, gf);
    free(G);
    free(wts);
  }
  for (int i = 1; i < used; i++) {
    const double* buf = priv[i];
    for (int64_t j = 0; j < nvid; j++) {
      grad_q[j] += buf[j];
      grad_k[j] += buf[nvid + j];
      grad_v[j] += buf[2 * nvid + j];
    }
    for (int64_t j = 0; j < nflow; j++) grad_flows[j] += buf[3 * nvid + j];
    free(priv[i]);
  }
  free(priv);
  free(cnt);
}

/* Bilinear reads of one H x W image at n positions (exported so the tests can
 * pin the sampling convention against an independent library routine). */
void oracle_bilinear_image(const double* img, int H, int W, const double* ys, const double* xs, int64_t n,
                           double* out) {
  oracle_params p;
  memset(&p, 0, sizeof(p));
  p.B = 1; p.T = 1; p.C = 1; p.H = H; p.W = W; p.HD = 1;
  for (int64_t i = 0; i < n; i++) out[i] = bilinear(img, &p, 0, 0, 0, ys[i], xs[i]);
}

/* ---- front-end of the paper's example interface (Appendix "Pytorch
 * Example"): the search there takes one forward flow (t -> t+1) and one
 * backward flow (t -> t-1) per frame while its window spans wt > 1 frames
 * each way.  How the one-step flows are combined is not described; the
 * reading taken here composes them along the motion path:
 *   F_{+1}(x) = f_t(x),  F_{+s}(x) = F_{+(s-1)}(x) + f_{t+s-1}(x + F_{+(s-1)}(x)),
 * and mirrored with the backward flows for negative steps.  A one-step flow
 * is read bilinearly at a fractional position clamped into the frame (the
 * field continues at its border).  Steps whose frame lies outside the clip
 * are left at 0 (such frames are never searched).
 * fflow, bflow: (B, T, 2, H, W); flows: (B, T, 2*wt, 2, H, W), slot order as
 * in the search (dt = -wt..-1, +1..+wt), component 0 = row offset. */
static double clamped_bilinear(const double* f, int H, int W, double y, double x) {
  double yc = y < 0.0 ? 0.0 : (y > H - 1 ? (double)(H - 1) : y);
  double xc = x < 0.0 ? 0.0 : (x > W - 1 ? (double)(W - 1) : x);
  int y0 = (int)floor(yc), x0 = (int)floor(xc);
  double ay = yc - y0, ax = xc - x0;
  int y1 = y0 + 1 < H ? y0 + 1 : H - 1, x1 = x0 + 1 < W ? x0 + 1 : W - 1;
  return (1.0 - ay) * ((1.0 - ax) * f[(int64_t)y0 * W + x0] + ax * f[(int64_t)y0 * W + x1]) +
         ay * ((1.0 - ax) * f[(int64_t)y1 * W + x0] + ax * f[(int64_t)y1 * W + x1]);
}

void oracle_chain_flows(const double* fflow, const double* bflow, int B, int T, int H, int W, int wt,
                        double* flows) {
  int64_t HW = (int64_t)H * W;
  memset(flows, 0, sizeof(double) * (size_t)B * T * 2 * wt * 2 * HW);
  for (int b = 0; b < B; b++)
    for (int t = 0; t < T; t++)
      for (int dir = -1; dir <= 1; dir += 2) {
        const double* one = dir > 0 ? fflow : bflow;
        for (int y = 0; y < H; y++)
          for (int x = 0; x < W; x++) {
            double fh = 0.0, fw = 0.0;
            for (int s = 1; s <= wt; s++) {
              int t1 = t + dir * (s - 1), t2 = t + dir * s;
              if (t2 < 0 || t2 >= T) break;
              const double* fh1 = one + (((int64_t)b * T + t1) * 2 + 0) * HW;
              const double* fw1 = one + (((int64_t)b * T + t1) * 2 + 1) * HW;
              double py = y + fh, px = x + fw;
              double dh = clamped_bilinear(fh1, H, W, py, px), dw = clamped_bilinear(fw1, H, W, py, px);
              fh += dh;
              fw += dw;
              int slot = dir < 0 ? -s + wt : s + wt - 1;
              flows[((((int64_t)b * T + t) * 2 * wt + slot) * 2 + 0) * HW + (int64_t)y * W + x] = fh;
              flows[((((int64_t)b * T + t) * 2 * wt + slot) * 2 + 1) * HW + (int64_t)y * W + x] = fw;
            }
          }
      }
}

/* The aggregation that keeps the k neighbours apart (Sec. 3.2 aggregation;
 * the example's NonLocalGather returns (B,HD,K,T,F',H,W) and reduces over K
 * afterwards): stacked[b,hd,l,t,c,y,x] = (1/count(y,x)) * sum over the query
 * patches covering (y,x) of w_l * v~_l, with the softmax weights, bilinear
 * reads and count of oracle_aggregate.  Summed over l it is that
 * aggregation. */
void oracle_aggregate_stacked(const double* v, const double* dists, const double* inds, const oracle_params* p,
                              double scale, double* stacked) {
  int nH = grid_h(p), nW = grid_w(p), Ch = p->C / p->HD, lo = patch_lo(p), kk = p->k;
  int64_t HW = (int64_t)p->H * p->W;
  int64_t nst = (int64_t)p->B * p->HD * kk * p->T * Ch * HW;
  double* cnt = (double*)calloc((size_t)p->B * p->T * HW, sizeof(double));
  double* wts = (double*)malloc(sizeof(double) * (size_t)kk);
  memset(stacked, 0, sizeof(double) * (size_t)nst);
  for (int b = 0; b < p->B; b++)
    for (int t = 0; t < p->T; t++)
      for (int mh = 0; mh < nH; mh++)
        for (int mw = 0; mw < nW; mw++) {
          int h = mh * p->stride0, w = mw * p->stride0;
          for (int ph = lo; ph < lo + p->ps; ph++)
            for (int pw = lo; pw < lo + p->ps; pw++) {
              int y = h + ph, x = w + pw;
              if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
              cnt[((int64_t)b * p->T + t) * HW + (int64_t)y * p->W + x] += 1.0;
            }
          for (int hd = 0; hd < p->HD; hd++) {
            int64_t row = ((((int64_t)b * p->HD + hd) * p->T + t) * nH + mh) * nW + mw;
            softmax_row(dists + row * kk, kk, p->dist_type, scale, wts);
            for (int l = 0; l < kk; l++) {
              if (wts[l] == 0.0) continue;
              const double* ind = inds + 3 * (row * kk + l);
              int tk = neighbour_frame(p, ind[0]);
              if (tk < 0) continue;
              for (int ph = lo; ph < lo + p->ps; ph++)
                for (int pw = lo; pw < lo + p->ps; pw++) {
                  int y = h + ph, x = w + pw;
                  if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
                  for (int c = 0; c < Ch; c++) {
                    int64_t o = (((((int64_t)b * p->HD + hd) * kk + l) * p->T + t) * Ch + c) * HW +
                                (int64_t)y * p->W + x;
                    stacked[o] += wts[l] * bilinear(v, p, b, tk, hd * Ch + c, (double)y + ind[1], (double)x + ind[2]);
                  }
                }
            }
          }
        }
  for (int64_t o = 0; o < nst; o++) {
    int64_t pix = o % HW;
    int64_t r = o / HW / Ch;
    int t = (int)(r % p->T);
    int b = (int)(r / p->T / kk / p->HD);
    double n = cnt[((int64_t)b * p->T + t) * HW + pix];
    stacked[o] = n > 0.0 ? stacked[o] / n : 0.0;
  }
  free(wts);
  free(cnt);
}

/* The stacked gather of the code example with the caller's weights (the
 * example passes softmax(-10 * dists) computed outside the gather):
 * stacked[b,hd,l,t,c,y,x] = (1/count(y,x)) * sum over the query patches
 * covering (y,x) of weights_l * v~_l, the bilinear read of the l-th
 * neighbour's frame at (y,x) + its displacement (head hd's channels).  A
 * neighbour whose weight is 0, whose frame is not an integer in [0,T) or
 * whose displacement is not finite contributes nothing.  weights:
 * (B,HD,T,nH,nW,k); stacked: (B,HD,k,T,C/HD,H,W). */
void oracle_gather_stacked(const double* v, const double* weights, const double* inds, const oracle_params* p,
                           double* stacked) {
  int nH = grid_h(p), nW = grid_w(p), Ch = p->C / p->HD, lo = patch_lo(p), kk = p->k;
  int64_t HW = (int64_t)p->H * p->W;
  int64_t nst = (int64_t)p->B * p->HD * kk * p->T * Ch * HW;
  double* cnt = (double*)calloc((size_t)p->B * p->T * HW, sizeof(double));
  memset(stacked, 0, sizeof(double) * (size_t)nst);
  for (int b = 0; b < p->B; b++)
    for (int t = 0; t < p->T; t++)
      for (int mh = 0; mh < nH; mh++)
        for (int mw = 0; mw < nW; mw++) {
          int h = mh * p->stride0, w = mw * p->stride0;
          for (int ph = lo; ph < lo + p->ps; ph++)
            for (int pw = lo; pw < lo + p->ps; pw++) {
              int y = h + ph, x = w + pw;
              if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
              cnt[((int64_t)b * p->T + t) * HW + (int64_t)y * p->W + x] += 1.0;
            }
          for (int hd = 0; hd < p->HD; hd++) {
            int64_t row = ((((int64_t)b * p->HD + hd) * p->T + t) * nH + mh) * nW + mw;
            for (int l = 0; l < kk; l++) {
              double wl = weights[row * kk + l];
              const double* ind = inds + 3 * (row * kk + l);
              int tk = neighbour_frame(p, ind[0]);
              if (wl == 0.0 || tk < 0 || !isfinite(ind[1]) || !isfinite(ind[2])) continue;
              for (int ph = lo; ph < lo + p->ps; ph++)
                for (int pw = lo; pw < lo + p->ps; pw++) {
                  int y = h + ph, x = w + pw;
                  if (y < 0 || y >= p->H || x < 0 || x >= p->W) continue;
                  for (int c = 0; c < Ch; c++) {
                    int64_t o = (((((int64_t)b * p->HD + hd) * kk + l) * p->T + t) * Ch + c) * HW +
                                (int64_t)y * p->W + x;
                    stacked[o] += wl * bilinear(v, p, b, tk, hd * Ch + c, (double)y + ind[1], (double)x + ind[2]);
                  }
                }
            }
          }
        }
  for (int64_t o = 0; o < nst; o++) {
    int64_t pix = o % HW;
    int64_t r = o / HW / Ch;
    int t = (int)(r % p->T);
    int b = (int)(r / p->T / kk / p->HD);
    double n = cnt[((int64_t)b * p->T + t) * HW + pix];
    stacked[o] = n > 0.0 ? stacked[o] / n : 0.0;
  }
  free(cnt);
}

/* The reduction over the k neighbours that follows the gather in the code
 * example: the stacked tensor is rearranged to ((b t), (hd f), k, h, w) and
 * convolved with a (Cout, C, k, 1, 1) kernel at stride (k, 1, 1), so
 * out[b,t,o,y,x] = sum over hd, f, l of proj[o, hd*C/HD + f, l] *
 * stacked[b,hd,l,t,f,y,x].  proj: (Cout, C, k) row-major; out:
 * (B,T,Cout,H,W). */
void oracle_stacked_reduce(const double* stacked, const double* proj, const oracle_params* p, int cout,
                           double* out) {
  int Ch = p->C / p->HD, kk = p->k;
  int64_t HW = (int64_t)p->H * p->W;
#pragma omp parallel for schedule(static)
  for (int64_t bt = 0; bt < (int64_t)p->B * p->T; bt++) {
    int b = (int)(bt / p->T), t = (int)(bt % p->T);
    for (int o = 0; o < cout; o++)
      for (int64_t pix = 0; pix < HW; pix++) {
        double s = 0.0;
        for (int hd = 0; hd < p->HD; hd++)
          for (int f = 0; f < Ch; f++)
            for (int l = 0; l < kk; l++)
              s += proj[((int64_t)o * p->C + hd * Ch + f) * kk + l] *
                   stacked[(((((int64_t)b * p->HD + hd) * kk + l) * p->T + t) * Ch + f) * HW + pix];
        out[(bt * cout + o) * HW + pix] = s;
      }
  }
}

/*
 * snls.h -- C ABI of the Shifted Non-Local Search library for AMD MI355X
 * (gfx950).
 *
 * The operations follow "Space-Time Attention with Shifted Non-Local Search"
 * (Gauen & Chan, ICLR 2024):
 *   snls_search     Sec. 3.2, the shifted search S, F_out and top-L
 *                   (S_L, F_out,L = Shifted-NLS(Q, K, F_in, L)), computed in
 *                   parallel over a temporal window W_t with key stride S_K
 *                   and bilinear reads;
 *   snls_topk       Sec. 3.2, the top-L operator on already computed scores;
 *   snls_aggregate  Sec. 3.2 "Aggregation", softmax-weighted sum of the
 *                   selected patches, normalised per pixel;
 *   snls_backward   Sec. 1 / 3.2, gradients of the differentiable search and
 *                   aggregation;
 *   snls_aggregate_stacked, snls_chain_flows  the code example's neighbour-
 *                   stacked gather and its forward/backward flow interface;
 *   snls_gather_stacked, snls_stacked_reduce, snls_gather_reduce  the
 *                   example's gather with caller weights and its reduction
 *                   over the k neighbours (App. B);
 *   snls_aggregate_static  snls_aggregate without a caller workspace, for
 *                   callers that cannot allocate.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Pointers named as device buffers must point to device memory of the
 *    current HIP device; all are fp32, dense, C-contiguous, 4-byte aligned.
 *    The caller owns every buffer; the library keeps no pointer and no state
 *    between calls (apart from the scratch array of snls_aggregate_static),
 *    so concurrent calls on different streams are safe when their output
 *    buffers do not overlap.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL is the
 *    default stream).  Buffers must stay alive until the stream has
 *    completed the work.
 *  - Videos are laid out (B, T, C, H, W) as in the paper's code example;
 *    head hd owns channels [hd*C/HD, (hd+1)*C/HD).
 *  - Flows are (B, T, 2*wt, 2, H, W): for query frame t, slot s holds the
 *    offset to frame t+dt with dt = -wt..-1 for s = 0..wt-1 and dt = 1..wt
 *    for s = wt..2wt-1; component 0 is the row (h) offset, 1 the column (w)
 *    offset, read at the query's own pixel (Sec. 3.2, F_in[t_i, h_i, w_i]).
 *  - Query grid: h = m_h*stride0, w = m_w*stride0 for m_h < nH = (H-1)/stride0+1,
 *    m_w < nW = (W-1)/stride0+1.
 *  - Candidate (dt, d_h, d_w), d in 0..ws-1, is the window cell at
 *    displacement disp = fl32(F + fl32(stride1*(d - ws/2))) from the query
 *    (F = 0 for dt = 0); its id is ((dt+wt)*ws + d_h)*ws + d_w.  It is
 *    invalid when frame t+dt is outside [0,T) or its centre (h+disp_h,
 *    w+disp_w) is outside [0,H-1]x[0,W-1]; invalid candidates score -inf
 *    (inner product) or +inf (squared L2).  A candidate whose similarity is
 *    NaN (only with non-finite inputs) scores as an invalid one, so no NaN
 *    score is ever returned or ranked.  With non-finite inputs the scores are
 *    otherwise unspecified, but every kept neighbour is a candidate of the
 *    query's own window.
 *  - Similarity of a valid candidate: sum over patch offsets
 *    p in {-(ps/2) .. ps-1-(ps/2)}^2 with the query pixel (h+p_h, w+p_w)
 *    inside the frame, and over the head's channels, of q*k~ (inner product,
 *    larger is better) or (q-k~)^2 (squared L2, smaller is better), where
 *    k~ is the bilinear read of frame t+dt at (h+p_h+disp_h, w+p_w+disp_w)
 *    with taps outside the frame reading 0.
 *  - inds entries are (frame t+dt, disp_h, disp_w) stored as fp32.
 *  - H and W must be below 1,000,000 (SNLS_ERR_UNSUPPORTED otherwise), so a
 *    displacement of magnitude 1e6 or more leaves every frame: a neighbour
 *    carrying one (aggregation, backward) contributes nothing, exactly as
 *    its out-of-frame bilinear reads would give.
 *  - On an argument error the call returns before touching any buffer or
 *    launching anything.
 */
#ifndef SNLS_H_
#define SNLS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SNLS_ABI_VERSION 4

typedef enum {
  SNLS_OK = 0,
  SNLS_ERR_INVALID_ARG = 1, /* a size, pointer or parameter is out of range */
  SNLS_ERR_UNSUPPORTED = 2, /* valid, but beyond this build's limits (e.g. k > 128) */
  SNLS_ERR_HIP = 3,         /* the HIP runtime reported an error (no device, launch failure) */
  SNLS_ERR_WORKSPACE = 4,   /* workspace missing or smaller than snls_workspace_size() */
  SNLS_ERR_SCRATCH = 5      /* the call needs more than SNLS_STATIC_SCRATCH_BYTES (snls_aggregate_static) */
} snls_status;

typedef enum {
  SNLS_DIST_PROD = 0, /* inner product, larger is better (the paper's similarity) */
  SNLS_DIST_L2 = 1    /* squared L2 distance, smaller is better */
} snls_dist_type;

/* Search parameters.  struct_size must be sizeof(snls_params).
 *   B, T, C, H, W  video shape; HD heads (C % HD == 0)
 *   ws             spatial window Ws >= 1 (Ws x Ws cells per frame)
 *   wt             temporal radius >= 0 (W_t = 2*wt+1 frames, query frame included)
 *   ps             patch size P >= 1
 *   stride0        query stride S_Q >= 1
 *   stride1        key stride S_K > 0 (spacing of the window cells)
 *   k              neighbours kept per query and head (0 = keep all, see snls_search)
 *   dist_type      an snls_dist_type value */
typedef struct {
  uint32_t struct_size;
  int32_t B, T, C, H, W, HD;
  int32_t ws, wt, ps, stride0;
  float stride1;
  int32_t k;
  int32_t dist_type;
} snls_params;

/* Largest k that snls_search (fused top-k) and snls_topk accept. */
#define SNLS_MAX_K 128

/* snls_search -- shifted non-local search (Sec. 3.2).
 *   q, k      device, (B, T, C, H, W) query and key videos
 *   flows     device, (B, T, 2*wt, 2, H, W) window offsets (see above);
 *             may be NULL only when wt == 0
 *   p         host, parameters; p->k selects the output form:
 *   p->k >= 1 top-k per query and head, best first, ties to the smaller
 *             candidate id:  dists (B, HD, T, nH, nW, k),
 *                            inds  (B, HD, T, nH, nW, k, 3)
 *   p->k == 0 every candidate in id order (invalid ones at -inf / +inf):
 *             dists (B, HD, T, nH, nW, (2wt+1)*ws*ws), inds (..., 3)
 *   workspace device scratch of at least snls_workspace_size(SNLS_OP_SEARCH, p)
 *             bytes, 256-byte aligned; may be NULL when that size is 0.  The
 *             tiled top-k path (ps <= 7 with ws <= 9, or ps = 7 with ws <=
 *             15; stride1 <= 1; any stride0) and the single-pixel path with
 *             k > 32 (ps = 1, stride1 = 1, ws <= 15, inner product) score
 *             every candidate into it (4 bytes per query row and candidate,
 *             rows padded to 32 candidates) before selecting; squared L2
 *             adds the key-norm term of every candidate, the query norm of
 *             every row, five key pair products per key pixel, frame and
 *             head, the squared norm of every query pixel per frame and head
 *             and, where the norm terms are formed cell by cell (stride1 < 1
 *             or ws > 9), fp64 summed-area tables of the five products.  The
 *             fused single-pixel path (k <= 32) needs none.  Its contents
 *             are not needed between calls
 * Errors: SNLS_ERR_INVALID_ARG for shapes/parameters out of range or NULL
 * buffers; SNLS_ERR_UNSUPPORTED for k > SNLS_MAX_K; SNLS_ERR_WORKSPACE for a
 * missing, short or misaligned workspace; SNLS_ERR_HIP on a launch failure. */
snls_status snls_search(const float* q, const float* k, const float* flows, const snls_params* p, float* dists,
                        float* inds, void* workspace, size_t workspace_bytes, void* stream);

/* snls_topk -- top-L of precomputed scores (Sec. 3.2).
 *   dists_all  device, rows x n_cand scores; column j is candidate id j
 *   inds_all   device, rows x n_cand x 3 positions carried with the scores
 *   k          1 <= k <= min(n_cand, SNLS_MAX_K)
 *   dist_type  order: SNLS_DIST_PROD descending, SNLS_DIST_L2 ascending;
 *              ties go to the smaller column
 *   dists      device out, rows x k;  inds  device out, rows x k x 3
 * Errors: SNLS_ERR_INVALID_ARG (rows < 0, n_cand < 1, k out of range, NULL
 * buffers), SNLS_ERR_UNSUPPORTED (k > SNLS_MAX_K), SNLS_ERR_HIP. */
snls_status snls_topk(const float* dists_all, const float* inds_all, int64_t rows, int32_t n_cand, int32_t k,
                      int32_t dist_type, float* dists, float* inds, void* stream);

/* snls_aggregate -- weighted patch aggregation (Sec. 3.2 "Aggregation").
 * For each query (b,t,h,w) and head, weights w_l = softmax_l(sign*scale*d_l)
 * over its k neighbours (sign +1 inner product, -1 L2; non-finite d_l get
 * weight 0); every in-frame patch pixel (h+p_h, w+p_w) receives
 * sum_l w_l * v~(frame_l, c, h+p_h+disp_h,l, w+p_w+disp_w,l) for the head's
 * channels; each output pixel is divided by the number of query patches
 * covering it, and pixels no patch covers are 0.  Neighbours whose frame
 * entry is not an integer in [0,T) or whose displacement is not finite
 * contribute nothing.
 *   v          device, (B, T, C, H, W) value video
 *   dists      device, (B, HD, T, nH, nW, k) with k = p->k >= 1
 *   inds       device, (B, HD, T, nH, nW, k, 3)
 *   scale      softmax temperature factor (finite)
 *   out        device out, (B, T, C, H, W), fully overwritten
 *   workspace  device scratch of at least snls_workspace_size(SNLS_OP_AGGREGATE,
 *              p) bytes, 256-byte aligned (softmax weights and a channels-last
 *              copy of v); its contents are not needed between calls
 * The result does not depend on scheduling: it is bit-identical between runs.
 * Errors: SNLS_ERR_INVALID_ARG, SNLS_ERR_UNSUPPORTED (k > SNLS_MAX_K),
 * SNLS_ERR_WORKSPACE, SNLS_ERR_HIP. */
snls_status snls_aggregate(const float* v, const float* dists, const float* inds, const snls_params* p,
                           float scale, float* out, void* workspace, size_t workspace_bytes, void* stream);

/* Size of the library's own device scratch array used by
 * snls_aggregate_static (64 MiB on every GPU the library runs on). */
#define SNLS_STATIC_SCRATCH_BYTES (64u << 20)

/* snls_aggregate_static -- snls_aggregate for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same computation and kernels, with
 * the workspace taken from a device array of SNLS_STATIC_SCRATCH_BYTES that
 * the library holds on each GPU until the process ends.  The call allocates
 * nothing (no hipMalloc / hipFree, no allocating library routine).
 *   v, dists, inds, p, scale, out  as in snls_aggregate (caller-owned)
 * The array is shared by every call on one GPU and keeps the last call's
 * contents; calls that overlap in time on one GPU (several streams or host
 * threads) race on it and must be serialised by the caller.
 * Errors: as snls_aggregate; SNLS_ERR_SCRATCH (nothing launched) when
 * snls_workspace_size(SNLS_OP_AGGREGATE, p) exceeds
 * SNLS_STATIC_SCRATCH_BYTES. */
snls_status snls_aggregate_static(const float* v, const float* dists, const float* inds, const snls_params* p,
                                  float scale, float* out, void* stream);

/* snls_backward -- gradients of search + aggregation (Sec. 1: the grid
 * search is differentiable; the top-k set is held fixed, Sec. 3.2).
 * Inputs as in snls_search / snls_aggregate; dists and inds are the forward
 * outputs (p->k >= 1).  grad_out (B,T,C,H,W) is dL/d out; grad_dists
 * (B,HD,T,nH,nW,k) is dL/d dists or NULL.  Outputs, fully overwritten:
 * grad_q, grad_k, grad_v (B,T,C,H,W) and grad_flows (B,T,2wt,2,H,W) (may be
 * NULL when wt == 0).  workspace: device scratch of at least
 * snls_workspace_size(SNLS_OP_BACKWARD, p) bytes, 256-byte aligned (the
 * per-neighbour aggregation terms, channels-last copies of q, k, v and
 * grad_out, and channels-last gradient accumulators: about 7 videos).
 * Gradients are accumulated with floating-point atomics, so the last bits
 * may differ between runs.
 * Errors: SNLS_ERR_INVALID_ARG, SNLS_ERR_UNSUPPORTED, SNLS_ERR_WORKSPACE,
 * SNLS_ERR_HIP. */
snls_status snls_backward(const float* q, const float* k, const float* v, const float* flows, const float* dists,
                          const float* inds, const float* grad_out, const float* grad_dists, const snls_params* p,
                          float scale, float* grad_q, float* grad_k, float* grad_v, float* grad_flows,
                          void* workspace, size_t workspace_bytes, void* stream);

/* snls_aggregate_stacked -- the aggregation with the k neighbours kept apart
 * (Sec. 3.2 "Aggregation" as the paper's code example uses it: its gather
 * returns (B, HD, K, T, F', H, W) and a convolution reduces over K
 * afterwards).  Slice l holds, for each output pixel, the sum over the query
 * patches covering it of w_l * v~(frame_l, ...) (the weights, reads and
 * validity rules of snls_aggregate), divided by the number of covering
 * patches; summed over l it is snls_aggregate's output.
 *   v, dists, inds, p, scale  as in snls_aggregate
 *   stacked    device out, (B, HD, k, T, C/HD, H, W), fully overwritten
 *   workspace  device scratch of at least
 *              snls_workspace_size(SNLS_OP_AGGREGATE_STACKED, p) bytes,
 *              256-byte aligned (softmax weights)
 * Errors: as snls_aggregate; SNLS_ERR_UNSUPPORTED for outputs beyond 2^40
 * elements. */
snls_status snls_aggregate_stacked(const float* v, const float* dists, const float* inds, const snls_params* p,
                                   float scale, float* stacked, void* workspace, size_t workspace_bytes,
                                   void* stream);

/* snls_chain_flows -- window offsets from one-step flows, the front-end of
 * the paper's code example, whose search takes a forward flow (t -> t+1) and
 * a backward flow (t -> t-1) per frame while its window spans wt frames each
 * way.  The offset to frame t+s (s = 1..wt) is composed along the motion
 * path: F_1(x) = fflow_t(x), F_s(x) = F_{s-1}(x) + fflow_{t+s-1}(x + F_{s-1}(x)),
 * with each one-step flow read bilinearly at the position clamped into the
 * frame; the backward direction mirrors it with bflow.  Offsets to frames
 * outside the clip are 0 (never searched).
 *   fflow, bflow  device, (B, T, 2, H, W); component 0 = row offset
 *   flows         device out, (B, T, 2*wt, 2, H, W) in the slot order of
 *                 snls_search, fully overwritten; nothing is touched when
 *                 wt == 0 (NULL pointers are then allowed)
 * Errors: SNLS_ERR_INVALID_ARG for sizes < 1, wt < 0 or NULL buffers;
 * SNLS_ERR_UNSUPPORTED for H*W > 2^30, wt > 63 or more than 2^40 output
 * pixels; SNLS_ERR_HIP on a launch failure. */
snls_status snls_chain_flows(const float* fflow, const float* bflow, int32_t B, int32_t T, int32_t H, int32_t W,
                             int32_t wt, float* flows, void* stream);

/* snls_gather_stacked -- the gather of the paper's code example, with the
 * caller's weights (the example passes softmax(-10 * dists) computed outside
 * the gather): stacked[b,hd,l,t,f,y,x] = (1/cnt(y,x)) * sum over the query
 * patches covering (y,x) of weights_l * v~(frame_l, f, (y,x) + disp_l),
 * the aggregation of Sec. 3.2 restricted to the l-th neighbours (cnt: the
 * number of query patches covering the pixel; pixels no patch covers are
 * 0).  A neighbour whose weight is 0, whose frame entry is not an integer in
 * [0,T) or whose displacement is not finite contributes nothing; weights are
 * otherwise used as given (finite values expected).
 *   v          device, (B, T, C, H, W)
 *   weights    device, (B, HD, T, nH, nW, k) with k = p->k >= 1
 *   inds       device, (B, HD, T, nH, nW, k, 3), as snls_search returns
 *   stacked    device out, (B, HD, k, T, C/HD, H, W), fully overwritten
 *   workspace  device scratch of at least
 *              snls_workspace_size(SNLS_OP_GATHER_STACKED, p) bytes, 256-byte
 *              aligned (a channels-last copy of v; 0 bytes when a head has
 *              more than 64 channels, a channel count not a multiple of 4, or
 *              an 8 x 8 pixel tile more than 256 covering queries)
 * Errors: SNLS_ERR_INVALID_ARG, SNLS_ERR_UNSUPPORTED (outputs beyond 2^40
 * elements), SNLS_ERR_WORKSPACE, SNLS_ERR_HIP. */
snls_status snls_gather_stacked(const float* v, const float* weights, const float* inds, const snls_params* p,
                                float* stacked, void* workspace, size_t workspace_bytes, void* stream);

/* snls_stacked_reduce -- the reduction over the k neighbours that follows
 * the gather in the code example: the stacked tensor rearranged to
 * ((b t), (hd f), k, h, w) and convolved with a (Cout, C, k, 1, 1) kernel at
 * stride (k, 1, 1):
 *   out[b,t,o,y,x] = sum over hd, f, l of proj[o, hd*C/HD + f, l] * stacked[b,hd,l,t,f,y,x]
 * computed in fp32 on the matrix cores.
 *   stacked  device, (B, HD, k, T, C/HD, H, W)
 *   proj     device, (Cout, C, k) (the conv3d kernel without its 1 x 1 tail)
 *   cout     output channels, 1 <= cout <= 128
 *   out      device out, (B, T, Cout, H, W), fully overwritten
 * Errors: SNLS_ERR_INVALID_ARG; SNLS_ERR_UNSUPPORTED when C/HD is not a
 * multiple of 4 or exceeds 64, or cout > 128; SNLS_ERR_HIP. */
snls_status snls_stacked_reduce(const float* stacked, const float* proj, const snls_params* p, int32_t cout,
                                float* out, void* stream);

/* snls_gather_reduce -- snls_stacked_reduce(snls_gather_stacked(...)) in one
 * pass: the stacked tensor (k times the size of v) is formed per 8 x 8 pixel
 * tile on chip and never written.  Arguments as in the two calls; workspace:
 * at least snls_workspace_size(SNLS_OP_GATHER_REDUCE, p) bytes, 256-byte
 * aligned (a channels-last copy of v).
 * Errors: SNLS_ERR_INVALID_ARG; SNLS_ERR_UNSUPPORTED beyond the limits of
 * snls_stacked_reduce or when an 8 x 8 tile has more than 256 covering
 * queries; SNLS_ERR_WORKSPACE; SNLS_ERR_HIP. */
snls_status snls_gather_reduce(const float* v, const float* weights, const float* inds, const float* proj,
                               const snls_params* p, int32_t cout, float* out, void* workspace,
                               size_t workspace_bytes, void* stream);

#define SNLS_OP_SEARCH 0
#define SNLS_OP_AGGREGATE 1
#define SNLS_OP_BACKWARD 2
#define SNLS_OP_AGGREGATE_STACKED 3
#define SNLS_OP_GATHER_STACKED 4
#define SNLS_OP_GATHER_REDUCE 5

/* Device workspace in bytes that operation op needs for parameters p
 * (0 when none is needed; (size_t)-1 for invalid arguments). */
size_t snls_workspace_size(int op, const snls_params* p);

/* Static, NUL-terminated description of a status code. */
const char* snls_status_string(snls_status s);

/* SNLS_ABI_VERSION of the built library. */
int snls_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SNLS_H_ */

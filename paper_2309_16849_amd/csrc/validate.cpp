// validate.cpp -- host-only argument checks of the C ABI.  Nothing here
// touches the GPU, so every error path can be exercised on a machine
// without one.
#include <limits.h>
#include <math.h>

#include "snls_internal.h"

namespace snls {

// Sizes stay below 2^31 per tensor dimension product where kernels index
// with 32-bit arithmetic inside a frame; whole tensors use 64-bit offsets.
static const long long kMaxPlane = 1LL << 30;

snls_status check_params(const snls_params* p, bool need_k, Geo* g) {
  if (!p) return SNLS_ERR_INVALID_ARG;
  if (p->struct_size != sizeof(snls_params)) return SNLS_ERR_INVALID_ARG;
  if (p->B < 1 || p->T < 1 || p->C < 1 || p->H < 1 || p->W < 1 || p->HD < 1) return SNLS_ERR_INVALID_ARG;
  if (p->C % p->HD != 0) return SNLS_ERR_INVALID_ARG;
  if (p->ws < 1 || p->wt < 0 || p->ps < 1 || p->stride0 < 1) return SNLS_ERR_INVALID_ARG;
  if (!(p->stride1 > 0.f) || !isfinite(p->stride1)) return SNLS_ERR_INVALID_ARG;
  if (p->dist_type != SNLS_DIST_PROD && p->dist_type != SNLS_DIST_L2) return SNLS_ERR_INVALID_ARG;
  if ((long long)p->H * p->W > kMaxPlane) return SNLS_ERR_UNSUPPORTED;
  // displacements of kFarDisp or more must leave every frame
  if (p->H >= (long long)kFarDisp || p->W >= (long long)kFarDisp) return SNLS_ERR_UNSUPPORTED;
  if (p->ws > 255 || p->ps > 255 || p->wt > 63) return SNLS_ERR_UNSUPPORTED;
  long long ncand = (long long)(2 * p->wt + 1) * p->ws * p->ws;
  if (ncand > INT_MAX / 4) return SNLS_ERR_UNSUPPORTED;
  if (p->k < 0 || p->k > ncand) return SNLS_ERR_INVALID_ARG;
  if (need_k && p->k < 1) return SNLS_ERR_INVALID_ARG;
  if (p->k > SNLS_MAX_K) return SNLS_ERR_UNSUPPORTED;
  if (g) {
    g->B = p->B; g->T = p->T; g->C = p->C; g->H = p->H; g->W = p->W; g->HD = p->HD;
    g->ws = p->ws; g->wt = p->wt; g->ps = p->ps; g->s0 = p->stride0; g->s1 = p->stride1;
    g->k = p->k; g->dist = p->dist_type;
    g->nH = (p->H - 1) / p->stride0 + 1;
    g->nW = (p->W - 1) / p->stride0 + 1;
    g->Ch = p->C / p->HD;
    g->r = p->ws / 2;
    g->lo = -(p->ps / 2);
    g->ncand = (int)ncand;
    g->nslot = 2 * p->wt;
    g->HW = (long long)p->H * p->W;
    g->rows = (long long)p->B * p->HD * p->T * g->nH * g->nW;
  }
  return SNLS_OK;
}

snls_status check_topk_args(int64_t rows, int32_t n_cand, int32_t k, int32_t dist_type) {
  if (rows < 0 || n_cand < 1 || k < 1 || k > n_cand) return SNLS_ERR_INVALID_ARG;
  if (dist_type != SNLS_DIST_PROD && dist_type != SNLS_DIST_L2) return SNLS_ERR_INVALID_ARG;
  if (k > SNLS_MAX_K) return SNLS_ERR_UNSUPPORTED;
  return SNLS_OK;
}

}  // namespace snls

// api.hip -- extern "C" entry points of libsnls.so (declared in
// include/snls.h).  Each call validates its arguments on the host, then
// launches the kernels on the caller's stream.  Nothing is allocated and no
// state is kept between calls.
#include <cmath>

#include "snls_internal.h"

using namespace snls;

namespace {

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Device present and usable (the first HIP call of a process may fail here
// on a machine without a GPU).
snls_status device_ready() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return SNLS_ERR_HIP;
  }
  return SNLS_OK;
}

// Only the scored top-k paths need scratch: the scores of every candidate.
size_t search_ws_bytes(const Geo& g) {
  if (g.k < 1) return 0;
  const SearchRoute r = search_route(g);
  return r == SearchRoute::Tile || r == SearchRoute::P1Scored ? tile_ws_bytes(g) : 0;
}

}  // namespace

extern "C" {

int snls_abi_version(void) { return SNLS_ABI_VERSION; }

const char* snls_status_string(snls_status s) {
  switch (s) {
    case SNLS_OK: return "ok";
    case SNLS_ERR_INVALID_ARG: return "invalid argument";
    case SNLS_ERR_UNSUPPORTED: return "unsupported parameters";
    case SNLS_ERR_HIP: return "HIP runtime error";
    case SNLS_ERR_WORKSPACE: return "workspace missing or too small";
    case SNLS_ERR_SCRATCH: return "problem larger than the library's static scratch array";
  }
  return "unknown status";
}

size_t snls_workspace_size(int op, const snls_params* p) {
  Geo g;
  if (op == SNLS_OP_SEARCH) return check_params(p, false, &g) == SNLS_OK ? search_ws_bytes(g) : (size_t)-1;
  if (op == SNLS_OP_AGGREGATE) return check_params(p, true, &g) == SNLS_OK ? aggregate_ws_bytes(g) : (size_t)-1;
  if (op == SNLS_OP_BACKWARD) return check_params(p, true, &g) == SNLS_OK ? backward_ws_bytes(g) : (size_t)-1;
  if (op == SNLS_OP_AGGREGATE_STACKED)
    return check_params(p, true, &g) == SNLS_OK ? aggregate_stacked_ws_bytes(g) : (size_t)-1;
  if (op == SNLS_OP_GATHER_STACKED) return check_params(p, true, &g) == SNLS_OK ? gather_ws_bytes(g) : (size_t)-1;
  if (op == SNLS_OP_GATHER_REDUCE)
    return check_params(p, true, &g) == SNLS_OK ? (size_t)g.B * g.T * g.C * g.HW * sizeof(float) : (size_t)-1;
  return (size_t)-1;
}

snls_status snls_gather_stacked(const float* v, const float* weights, const float* inds, const snls_params* p,
                                float* stacked, void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!v || !weights || !inds || !stacked) return SNLS_ERR_INVALID_ARG;
  if ((long long)g.B * g.HD * g.k * g.T * ((g.Ch + 15) / 16) * g.HW > 0xffffffffLL * 256) return SNLS_ERR_UNSUPPORTED;
  const size_t need = gather_ws_bytes(g);
  if (need > 0 && (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_gather_stacked(v, weights, inds, g, stacked, workspace, as_stream(stream));
}

snls_status snls_stacked_reduce(const float* stacked, const float* proj, const snls_params* p, int32_t cout,
                                float* out, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!stacked || !proj || !out || cout < 1) return SNLS_ERR_INVALID_ARG;
  if (!reduce_supported(g, cout)) return SNLS_ERR_UNSUPPORTED;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_stacked_reduce(stacked, proj, g, cout, out, as_stream(stream));
}

snls_status snls_gather_reduce(const float* v, const float* weights, const float* inds, const float* proj,
                               const snls_params* p, int32_t cout, float* out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!v || !weights || !inds || !proj || !out || cout < 1) return SNLS_ERR_INVALID_ARG;
  if (!reduce_supported(g, cout) || !gather_tile_supported(g)) return SNLS_ERR_UNSUPPORTED;
  const size_t need = (size_t)g.B * g.T * g.C * g.HW * sizeof(float);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_gather_reduce(v, weights, inds, proj, g, cout, out, workspace, as_stream(stream));
}

snls_status snls_search(const float* q, const float* k, const float* flows, const snls_params* p, float* dists,
                        float* inds, void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  snls_status st = check_params(p, false, &g);
  if (st != SNLS_OK) return st;
  if (!q || !k || !dists || !inds || (g.wt > 0 && !flows)) return SNLS_ERR_INVALID_ARG;
  const size_t need = search_ws_bytes(g);
  if (need > 0 && (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  if (g.k == 0) return launch_search_full(q, k, flows, g, dists, inds, as_stream(stream));
  return launch_search_topk(q, k, flows, g, dists, inds, workspace, as_stream(stream));
}

snls_status snls_topk(const float* dists_all, const float* inds_all, int64_t rows, int32_t n_cand, int32_t k,
                      int32_t dist_type, float* dists, float* inds, void* stream) {
  snls_status st = check_topk_args(rows, n_cand, k, dist_type);
  if (st != SNLS_OK) return st;
  if (!dists_all || !inds_all || !dists || !inds) return SNLS_ERR_INVALID_ARG;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_topk(dists_all, inds_all, rows, n_cand, k, dist_type, dists, inds, as_stream(stream));
}

snls_status snls_aggregate(const float* v, const float* dists, const float* inds, const snls_params* p,
                           float scale, float* out, void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!v || !dists || !inds || !out || !std::isfinite(scale)) return SNLS_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < aggregate_ws_bytes(g) || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_aggregate(v, dists, inds, g, scale, out, workspace, as_stream(stream));
}

snls_status snls_aggregate_stacked(const float* v, const float* dists, const float* inds, const snls_params* p,
                                   float scale, float* stacked, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!v || !dists || !inds || !stacked || !std::isfinite(scale)) return SNLS_ERR_INVALID_ARG;
  if ((long long)g.B * g.HD * g.k * g.T * ((g.Ch + 15) / 16) * g.HW > 0xffffffffLL * 256) return SNLS_ERR_UNSUPPORTED;
  if (!workspace || workspace_bytes < aggregate_stacked_ws_bytes(g) || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_aggregate_stacked(v, dists, inds, g, scale, stacked, workspace, as_stream(stream));
}

snls_status snls_chain_flows(const float* fflow, const float* bflow, int32_t B, int32_t T, int32_t H, int32_t W,
                             int32_t wt, float* flows, void* stream) {
  if (B < 1 || T < 1 || H < 1 || W < 1 || wt < 0) return SNLS_ERR_INVALID_ARG;
  if ((long long)H * W > (1LL << 30) || wt > 63) return SNLS_ERR_UNSUPPORTED;
  if ((long long)B * T * 2 * H * W > 0xffffffffLL * 256) return SNLS_ERR_UNSUPPORTED;
  if (wt > 0 && (!fflow || !bflow || !flows)) return SNLS_ERR_INVALID_ARG;
  snls_status st;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_chain_flows(fflow, bflow, B, T, H, W, wt, flows, as_stream(stream));
}

snls_status snls_backward(const float* q, const float* k, const float* v, const float* flows, const float* dists,
                          const float* inds, const float* grad_out, const float* grad_dists, const snls_params* p,
                          float scale, float* grad_q, float* grad_k, float* grad_v, float* grad_flows,
                          void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  (void)flows;  // positions come from inds; d disp / d flow = 1
  if (!q || !k || !v || !dists || !inds || !grad_out || !grad_q || !grad_k || !grad_v) return SNLS_ERR_INVALID_ARG;
  if (g.wt > 0 && !grad_flows) return SNLS_ERR_INVALID_ARG;
  if (!std::isfinite(scale)) return SNLS_ERR_INVALID_ARG;
  size_t need = backward_ws_bytes(g);
  if (need > 0 && (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)))
    return SNLS_ERR_WORKSPACE;
  if ((st = device_ready()) != SNLS_OK) return st;
  return launch_backward(q, k, v, dists, inds, grad_out, grad_dists, g, scale, grad_q, grad_k, grad_v, grad_flows,
                         static_cast<float*>(workspace), as_stream(stream));
}

}  // extern "C"

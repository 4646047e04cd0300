// static_scratch.hip -- snls_aggregate_static: the aggregation with its
// workspace (softmax weights and the channels-last copy of v) taken from a
// fixed device array of this library instead of a caller's buffer, for
// callers that cannot allocate device memory.
//
// The array is a file-scope __device__ symbol: every GPU the library runs on
// holds its own copy, at its own address, until the process ends.  Host code
// never uses the symbol's name as an address (on the host it only names the
// symbol); the device address is looked up once per device with
// hipGetSymbolAddress, on that device's first call, and kept.
#include <mutex>

#include "snls_internal.h"

namespace snls {
namespace {

static __device__ __align__(256) unsigned char scratch[SNLS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of scratch per device, once resolved

// Device address of this device's copy of the scratch array.
snls_status scratch_for_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return SNLS_ERR_HIP;
  }
  if (dev >= kMaxDevices) return SNLS_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return SNLS_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SNLS_OK;
}

}  // namespace
}  // namespace snls

using namespace snls;

extern "C" snls_status snls_aggregate_static(const float* v, const float* dists, const float* inds,
                                             const snls_params* p, float scale, float* out, void* stream) {
  Geo g;
  snls_status st = check_params(p, true, &g);
  if (st != SNLS_OK) return st;
  if (!v || !dists || !inds || !out || !(scale - scale == 0.f)) return SNLS_ERR_INVALID_ARG;
  if (aggregate_ws_bytes(g) > (size_t)SNLS_STATIC_SCRATCH_BYTES) return SNLS_ERR_SCRATCH;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return SNLS_ERR_HIP;
  }
  void* ws = nullptr;
  if ((st = scratch_for_current_device(&ws)) != SNLS_OK) return st;
  // Every kernel of the aggregation writes the part of the workspace it
  // reads before reading it (weights, then the transposed v), so nothing
  // left by an earlier call needs clearing.
  return launch_aggregate(v, dists, inds, g, scale, out, ws, reinterpret_cast<hipStream_t>(stream));
}

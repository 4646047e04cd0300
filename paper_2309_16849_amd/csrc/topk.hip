// topk.hip -- top-L of precomputed candidate scores (Sec. 3.2): per row,
// the k best columns, best first, ties to the smaller column.  One wave per
// row: each lane keeps a register list over a strided slice of the row, then
// the 64 lists are merged by repeated wave-wide arg-best selection.
#include "snls_internal.h"

namespace snls {

template <int KMAX>
__global__ void __launch_bounds__(256) topk_kernel(const float* __restrict__ dall, const float* __restrict__ iall,
                                                   long long rows, int ncand, int k, int dist,
                                                   float* __restrict__ dists, float* __restrict__ inds) {
  const int lane = threadIdx.x & 63;
  const long long row = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (row >= rows) return;  // whole wave leaves together
  const float* drow = dall + row * ncand;
  TopList<KMAX> lst;
  lst.init(k);
  for (int j = lane; j < ncand; j += 64) {
    float d = drow[j];
    float sc = to_score(d, dist);
    if (sc != sc) sc = -INFINITY;  // NaN ranks last
    lst.push(sc, j);
  }
  // Merge: k rounds of wave arg-best over the lanes' list heads.
  int head = KMAX - k;  // slot of the lane's best entry
  for (int i = 0; i < k; ++i) {
    float hs = -INFINITY;
    int hid = 0x7fffffff;
#pragma unroll
    for (int e = 0; e < KMAX; ++e) {
      if (e == head) {
        hs = lst.s[e];
        hid = lst.id[e];
      }
    }
    float bs = hs;
    int bid = hid;
    for (int off = 32; off > 0; off >>= 1) {
      float os = __shfl_xor(bs, off, 64);
      int oid = __shfl_xor(bid, off, 64);
      if (ranks_before(os, oid, bs, bid)) {
        bs = os;
        bid = oid;
      }
    }
    if (hid == bid && head < KMAX) ++head;
    if (lane == 0) {
      dists[row * k + i] = drow[bid];
      const float* src = iall + ((long long)row * ncand + bid) * 3;
      float* dst = inds + ((long long)row * k + i) * 3;
      dst[0] = src[0];
      dst[1] = src[1];
      dst[2] = src[2];
    }
  }
}

snls_status launch_topk(const float* dall, const float* iall, int64_t rows, int ncand, int k, int dist,
                        float* dists, float* inds, hipStream_t s) {
  if (rows == 0) return SNLS_OK;
  unsigned blocks = (unsigned)((rows + 3) / 4);
  if (k <= 16)
    hipLaunchKernelGGL(topk_kernel<16>, dim3(blocks), dim3(256), 0, s, dall, iall, (long long)rows, ncand, k, dist,
                       dists, inds);
  else if (k <= 32)
    hipLaunchKernelGGL(topk_kernel<32>, dim3(blocks), dim3(256), 0, s, dall, iall, (long long)rows, ncand, k, dist,
                       dists, inds);
  else if (k <= 64)
    hipLaunchKernelGGL(topk_kernel<64>, dim3(blocks), dim3(256), 0, s, dall, iall, (long long)rows, ncand, k, dist,
                       dists, inds);
  else
    hipLaunchKernelGGL(topk_kernel<128>, dim3(blocks), dim3(256), 0, s, dall, iall, (long long)rows, ncand, k, dist,
                       dists, inds);
  return hipGetLastError() == hipSuccess ? SNLS_OK : SNLS_ERR_HIP;
}

}  // namespace snls

// Punctuation mask from token ids: mask[i] = 1 iff ids[i] is in the
// punctuation id set P (the indicator I(x_i in P) of Eq. 7).
//
// Every workgroup stages the sorted set in LDS once and then covers a
// grid-stride range of tokens, four ids per thread per step (16-byte loads),
// each found by a binary search over the staged set.  The kernel streams the
// ids once (HBM-bound).
#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ uint8_t in_sorted(const int32_t *s, int n, int32_t x) {
  int lo = 0, hi = n;  // first element >= x
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (s[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return (lo < n && s[lo] == x) ? 1 : 0;
}

__global__ __launch_bounds__(256) void punct_mask_kernel(const int32_t *__restrict__ ids, int64_t n,
                                                         const int32_t *__restrict__ pset, int n_punct,
                                                         uint8_t *__restrict__ mask) {
  extern __shared__ int32_t sp[];
  for (int j = threadIdx.x; j < n_punct; j += 256) sp[j] = pset[j];
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * 256 * 4;
  for (int64_t i0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; i0 < n; i0 += stride) {
    if (i0 + 4 <= n && (reinterpret_cast<uintptr_t>(ids + i0) & 15) == 0) {
      const int4 v = *reinterpret_cast<const int4 *>(ids + i0);
      const uint32_t packed = (uint32_t)in_sorted(sp, n_punct, v.x) | ((uint32_t)in_sorted(sp, n_punct, v.y) << 8) |
                              ((uint32_t)in_sorted(sp, n_punct, v.z) << 16) |
                              ((uint32_t)in_sorted(sp, n_punct, v.w) << 24);
      if ((reinterpret_cast<uintptr_t>(mask + i0) & 3) == 0) {
        *reinterpret_cast<uint32_t *>(mask + i0) = packed;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) mask[i0 + e] = (uint8_t)(packed >> (8 * e));
      }
    } else {
      for (int64_t i = i0; i < i0 + 4 && i < n; ++i) mask[i] = in_sorted(sp, n_punct, ids[i]);
    }
  }
}

hipError_t launch_punct_mask(const int32_t *ids, int64_t n, const int32_t *pset, int n_punct, uint8_t *mask,
                             hipStream_t s) {
  const int64_t groups = (n + 1023) / 1024;
  const unsigned grid = (unsigned)(groups < 4096 ? groups : 4096);
  timing_begin("phsa_punct_mask", s);
  hipLaunchKernelGGL(punct_mask_kernel, dim3(grid), dim3(256), (size_t)n_punct * sizeof(int32_t), s, ids, n, pset,
                     n_punct, mask);
  timing_end(s);
  return hipGetLastError();
}

}  // namespace phsa

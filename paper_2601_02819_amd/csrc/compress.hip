// Block representatives: for each (b, g, t) the m keys of block t are pooled
// into M = lambda * mean(K) + (1 - lambda) * mean(K at punctuation), or the
// plain mean when the block holds no punctuation (Eq. 6-8 and the fallback
// under Eq. 7).
//
// Both kernels below are a single streaming pass over K (HBM-bound).  The
// per-head kernel takes one workgroup per (t, g, b): the block's m rows of d
// elements are read with 16-byte loads, d / VEC threads cover a row, the 256
// threads cover 256 * VEC / d rows at a time, and the per-thread float32 partial
// sums meet in LDS.
#include "common.h"
#include "launch.h"

namespace phsa {

template <typename T, int D>
__global__ __launch_bounds__(256) void compress_kernel(const T *__restrict__ K, const uint8_t *__restrict__ punct,
                                                       float *__restrict__ Kc, int Lk, int Hkv, int m, int T_blocks,
                                                       float lambda) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int TPR = D / VEC;          // threads per key row
  constexpr int NG = 256 / TPR;         // rows in flight
  __shared__ float red_all[NG][D];
  __shared__ float red_p[NG][D];
  __shared__ int s_npunct;

  const int t = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int c0 = (tid % TPR) * VEC;
  const int rg = tid / TPR;
  if (tid == 0) s_npunct = 0;
  __syncthreads();

  const uint8_t *pm = punct + (int64_t)b * Lk + (int64_t)t * m;
  float s_all[VEC], s_p[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) s_all[v] = s_p[v] = 0.f;
  int my_punct = 0;
  for (int r = rg; r < m; r += NG) {
    const int64_t row = (int64_t)b * Lk + (int64_t)t * m + r;
    const T *src = K + (row * Hkv + g) * D + c0;
    const uint4 raw = *reinterpret_cast<const uint4 *>(src);
    const T *vals = reinterpret_cast<const T *>(&raw);
    const bool is_p = pm[r] != 0;
    if (is_p && c0 == 0) ++my_punct;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      const float x = to_f32<T>(vals[v]);
      s_all[v] += x;
      s_p[v] += is_p ? x : 0.f;
    }
  }
#pragma unroll
  for (int v = 0; v < VEC; ++v) {
    red_all[rg][c0 + v] = s_all[v];
    red_p[rg][c0 + v] = s_p[v];
  }
  if (my_punct) atomicAdd(&s_npunct, my_punct);
  __syncthreads();
  const int np = s_npunct;
  for (int c = tid; c < D; c += 256) {
    float a = 0.f, p = 0.f;
#pragma unroll 8
    for (int x = 0; x < NG; ++x) {
      a += red_all[x][c];
      p += red_p[x][c];
    }
    const float M0 = a / (float)m;
    const float M = np > 0 ? lambda * M0 + (1.f - lambda) * (p / (float)np) : M0;
    Kc[(((int64_t)b * Hkv + g) * T_blocks + t) * D + c] = M;
  }
}

// All KV heads of a block at once: a token's Hkv * D keys are one contiguous
// row of CV 16-byte vectors, and a block's m rows are one contiguous run.  A
// workgroup takes RG = 256 / CV consecutive blocks of one sequence (CV >= 256:
// one block, CV / 256 vectors per thread); thread (rg, cv) sums vector cv over
// all m rows of its block on its own, U loads in flight, so no partial sums
// meet anywhere.  A wave lies inside one block: the block's punctuation flags
// are one ballot per 64 rows and every row's flag is a wave-uniform bit.
template <typename T, int CV>
__global__ __launch_bounds__(256) void compress_rows_kernel(const T *__restrict__ K, const uint8_t *__restrict__ punct,
                                                            float *__restrict__ Kc, int Lk, int Hkv, int D, int m,
                                                            int T_blocks, float lambda) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int RG = CV >= 256 ? 1 : 256 / CV;  // blocks per workgroup
  constexpr int CPT = CV >= 256 ? CV / 256 : 1;  // vectors per thread
  constexpr int U = 8;                           // rows in flight per thread
  static_assert(CV >= 64 && (CV >= 256 ? CV % 256 == 0 : 256 % CV == 0), "row vectors");

  const int tid = threadIdx.x, lane = tid & 63;
  const int rg = __builtin_amdgcn_readfirstlane(tid / (CV >= 256 ? 256 : CV));
  const int cv0 = CV >= 256 ? tid : tid % CV;
  const int b = blockIdx.y, t = blockIdx.x * RG + rg;
  if (t >= T_blocks) return;
  const uint8_t *pm = punct + (int64_t)b * Lk + (int64_t)t * m;
  const T *src = K + ((int64_t)b * Lk + (int64_t)t * m) * CV * VEC + cv0 * VEC;
  float s_all[CPT][VEC], s_p[CPT][VEC];
#pragma unroll
  for (int c = 0; c < CPT; ++c)
#pragma unroll
    for (int v = 0; v < VEC; ++v) s_all[c][v] = s_p[c][v] = 0.f;
  int np = 0;  // punctuation tokens of the block
  for (int r64 = 0; r64 < m; r64 += 64) {
    const uint64_t pmask = __ballot(r64 + lane < m && pm[r64 + lane] != 0);
    np += __popcll(pmask);
    const int n = min(64, m - r64);
    for (int u0 = 0; u0 < n; u0 += U) {
      uint4 raw[U][CPT];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < CPT; ++c)
          raw[u][c] = u0 + u < n ? *reinterpret_cast<const uint4 *>(src + (int64_t)(r64 + u0 + u) * CV * VEC + c * 256 * VEC)
                                 : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool isp = (pmask >> (u0 + u)) & 1;  // rows past n have a clear bit
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
          const T *vals = reinterpret_cast<const T *>(&raw[u][c]);
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            const float x = to_f32<T>(vals[v]);
            s_all[c][v] += x;
            s_p[c][v] += isp ? x : 0.f;
          }
        }
      }
    }
  }
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int e = (cv0 + c * 256) * VEC;  // g * D + feature of the first element
    const int g = e / D, f = e - g * D;    // D is a multiple of VEC: one head per vector
    float M[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      const float M0 = s_all[c][v] / (float)m;
      M[v] = np > 0 ? lambda * M0 + (1.f - lambda) * (s_p[c][v] / (float)np) : M0;
    }
    float *dst = Kc + (((int64_t)b * Hkv + g) * T_blocks + t) * D + f;
#pragma unroll
    for (int v = 0; v < VEC; v += 4) *reinterpret_cast<float4 *>(dst + v) = make_float4(M[v], M[v + 1], M[v + 2], M[v + 3]);
  }
}

template <typename T, int D>
static hipError_t launch_compress_t(const Geom &g, const void *K, const uint8_t *punct, float *Kc, hipStream_t s) {
  timing_begin("phsa_compress", s);
  const int cv = g.Hkv * D * (int)sizeof(T) / 16;  // 16-byte vectors per token row
  // short blocks: the per-head kernel's workgroups would carry m * D elements
  // each (4 KB at m = 16), too little to hide a launch; at m >= 64 the two run
  // at the same rate (the per-head kernel slightly ahead)
  if (g.m < 64 && (cv == 64 || cv == 128 || cv == 256 || cv == 512)) {
    const int rg = cv >= 256 ? 1 : 256 / cv;
    const dim3 grid((g.T + rg - 1) / rg, g.B);
    const T *Kt = static_cast<const T *>(K);
    if (cv == 64)
      hipLaunchKernelGGL((compress_rows_kernel<T, 64>), grid, dim3(256), 0, s, Kt, punct, Kc, g.Lk, g.Hkv, D, g.m, g.T,
                         g.lambda);
    else if (cv == 128)
      hipLaunchKernelGGL((compress_rows_kernel<T, 128>), grid, dim3(256), 0, s, Kt, punct, Kc, g.Lk, g.Hkv, D, g.m, g.T,
                         g.lambda);
    else if (cv == 256)
      hipLaunchKernelGGL((compress_rows_kernel<T, 256>), grid, dim3(256), 0, s, Kt, punct, Kc, g.Lk, g.Hkv, D, g.m, g.T,
                         g.lambda);
    else
      hipLaunchKernelGGL((compress_rows_kernel<T, 512>), grid, dim3(256), 0, s, Kt, punct, Kc, g.Lk, g.Hkv, D, g.m, g.T,
                         g.lambda);
  } else {
    const dim3 grid(g.T, g.Hkv, g.B);
    hipLaunchKernelGGL((compress_kernel<T, D>), grid, dim3(256), 0, s, static_cast<const T *>(K), punct, Kc, g.Lk,
                       g.Hkv, g.m, g.T, g.lambda);
  }
  timing_end(s);
  return hipGetLastError();
}

hipError_t launch_compress(const Geom &g, const void *K, const uint8_t *punct, float *Kc, hipStream_t s) {
  if (g.dtype == 0) {
    return g.d == 128 ? launch_compress_t<bf16_t, 128>(g, K, punct, Kc, s)
                      : launch_compress_t<bf16_t, 64>(g, K, punct, Kc, s);
  }
  return g.d == 128 ? launch_compress_t<float, 128>(g, K, punct, Kc, s)
                    : launch_compress_t<float, 64>(g, K, punct, Kc, s);
}

}  // namespace phsa

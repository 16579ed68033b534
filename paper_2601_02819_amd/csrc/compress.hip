// Block representatives: for each (b, g, t) the m keys of block t are pooled
// into M = lambda * mean(K) + (1 - lambda) * mean(K at punctuation), or the
// plain mean when the block holds no punctuation (Eq. 6-8 and the fallback
// under Eq. 7).
//
// One workgroup per (t, g, b).  The block's m rows of d elements are read with
// 16-byte loads: d / VEC threads cover a row, the 256 threads cover 256 * VEC / d
// rows at a time, and the per-thread float32 partial sums meet in LDS.  The
// kernel is a single streaming pass over K (HBM-bound).
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

template <typename T, int D>
static hipError_t launch_compress_t(const Geom &g, const void *K, const uint8_t *punct, float *Kc, hipStream_t s) {
  dim3 grid(g.T, g.Hkv, g.B);
  timing_begin("phsa_compress", s);
  hipLaunchKernelGGL((compress_kernel<T, D>), grid, dim3(256), 0, s, static_cast<const T *>(K), punct, Kc, g.Lk,
                     g.Hkv, g.m, g.T, g.lambda);
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

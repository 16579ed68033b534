// Sparse attention forward/backward for float32 tensors (Eq. 10-11), token-major.
//
// float32 inputs are held to a 1e-4 tolerance, which bf16 matrix cores cannot
// meet, so this path runs on the vector ALUs in float32.  One wave per
// (b, h, query row): lane = key within a 64-key slice of a selected block,
// an online softmax runs over the selected blocks, and the P.V / dS.K
// products use the lane = feature mapping through LDS.  The backward adds
// dK/dV with float32 atomics.  It targets small problems (the 1k-token fp32
// workload); the bf16 path is the throughput path.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {


__device__ __forceinline__ bool slot_ok_f(int t, int cur, int T) { return t >= 0 && t <= cur && t < T; }

template <int D>
__global__ __launch_bounds__(64) void attn_fwd_fp32_kernel(const float *__restrict__ Q, const float *__restrict__ K,
                                                           const float *__restrict__ V, const int32_t *__restrict__ sel,
                                                           float *__restrict__ O, float *__restrict__ LSE, Geom gm) {
  constexpr int NC = D / 64;
  __shared__ float qs[D];
  __shared__ float ps[64];
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z, lane = threadIdx.x;
  const int g = h / gm.G;
  const int pos = gm.q_pos0 + i, cur = pos / gm.m;
  for (int c = lane; c < D; c += 64) qs[c] = Q[(((int64_t)b * gm.Lq + i) * gm.Hq + h) * D + c];
  __syncthreads();
  float mrun = -INFINITY, lrun = 0.f, acc[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) acc[j] = 0.f;
  const int32_t *srow = sel + (((int64_t)b * gm.Hkv + g) * gm.Lq + i) * gm.ksel;
  for (int s = 0; s < gm.ksel; ++s) {
    const int t = srow[s];
    if (!slot_ok_f(t, cur, gm.T)) continue;
    for (int kb = 0; kb < gm.m; kb += 64) {
      const int key = t * gm.m + kb + lane;
      const bool ok = (kb + lane < gm.m) && key <= pos;
      float sc = -INFINITY;
      if (ok) {
        const float *kr = K + (((int64_t)b * gm.Lk + key) * gm.Hkv + g) * D;
        float d0 = 0.f;
        for (int c = 0; c < D; ++c) d0 = fmaf(qs[c], kr[c], d0);
        sc = d0 * gm.scale;
      }
      const float mx = wave_max(sc);
      const float newm = fmaxf(mrun, mx);
      if (newm == -INFINITY) continue;  // nothing visible in this slice yet (uniform)
      const float alpha = mrun == -INFINITY ? 0.f : expf(mrun - newm);
      const float p = ok ? expf(sc - newm) : 0.f;
      lrun = lrun * alpha + wave_sum(p);
      ps[lane] = p;
      __syncthreads();
      const int nk = min(64, gm.m - kb);
#pragma unroll
      for (int j = 0; j < NC; ++j) {
        float a = acc[j] * alpha;
        for (int k = 0; k < nk; ++k)
          a = fmaf(ps[k], V[(((int64_t)b * gm.Lk + t * gm.m + kb + k) * gm.Hkv + g) * D + lane + 64 * j], a);
        acc[j] = a;
      }
      __syncthreads();
      mrun = newm;
    }
  }
  const float inv = lrun > 0.f ? 1.f / lrun : 0.f;
#pragma unroll
  for (int j = 0; j < NC; ++j) O[(((int64_t)b * gm.Lq + i) * gm.Hq + h) * D + lane + 64 * j] = acc[j] * inv;
  if (lane == 0) LSE[((int64_t)b * gm.Hq + h) * gm.Lq + i] = lrun > 0.f ? mrun + logf(lrun) : -INFINITY;
}

__global__ void zero_kernel(float *__restrict__ p, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n; x += (int64_t)gridDim.x * blockDim.x)
    p[x] = 0.f;
}

template <int D>
__global__ __launch_bounds__(64) void attn_bwd_fp32_kernel(const float *__restrict__ Q, const float *__restrict__ K,
                                                           const float *__restrict__ V, const float *__restrict__ dO,
                                                           const float *__restrict__ LSE,
                                                           const float *__restrict__ Dvec,
                                                           const int32_t *__restrict__ sel, float *__restrict__ dQ,
                                                           float *__restrict__ dK, float *__restrict__ dV, Geom gm) {
  constexpr int NC = D / 64;
  __shared__ float qs[D], dos[D];
  __shared__ float ps[64], dss[64];
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z, lane = threadIdx.x;
  const int g = h / gm.G;
  const int pos = gm.q_pos0 + i, cur = pos / gm.m;
  const int64_t qrow = (((int64_t)b * gm.Lq + i) * gm.Hq + h) * D;
  for (int c = lane; c < D; c += 64) {
    qs[c] = Q[qrow + c];
    dos[c] = dO[qrow + c];
  }
  const float lse = LSE[((int64_t)b * gm.Hq + h) * gm.Lq + i];
  const float dd = Dvec[((int64_t)b * gm.Lq + i) * gm.Hq + h];
  __syncthreads();
  float dq[NC];
#pragma unroll
  for (int j = 0; j < NC; ++j) dq[j] = 0.f;
  const int32_t *srow = sel + (((int64_t)b * gm.Hkv + g) * gm.Lq + i) * gm.ksel;
  for (int s = 0; s < gm.ksel; ++s) {
    const int t = srow[s];
    if (!slot_ok_f(t, cur, gm.T)) continue;
    for (int kb = 0; kb < gm.m; kb += 64) {
      const int key = t * gm.m + kb + lane;
      const bool ok = (kb + lane < gm.m) && key <= pos;
      float p = 0.f, ds = 0.f;
      if (ok) {
        const int64_t kv = (((int64_t)b * gm.Lk + key) * gm.Hkv + g) * D;
        float sdot = 0.f, pdot = 0.f;
        for (int c = 0; c < D; ++c) {
          sdot = fmaf(qs[c], K[kv + c], sdot);
          pdot = fmaf(dos[c], V[kv + c], pdot);
        }
        p = expf(sdot * gm.scale - lse);
        ds = p * (pdot - dd);
      }
      ps[lane] = p;
      dss[lane] = ds;
      __syncthreads();
      const int nk = min(64, gm.m - kb);
      for (int k = 0; k < nk; ++k) {
        const int kk = t * gm.m + kb + k;
        if (kk > pos) break;
        const int64_t kv = (((int64_t)b * gm.Lk + kk) * gm.Hkv + g) * D;
#pragma unroll
        for (int j = 0; j < NC; ++j) {
          const int c = lane + 64 * j;
          dq[j] = fmaf(dss[k], K[kv + c], dq[j]);
          atomicAdd(&dV[kv + c], ps[k] * dos[c]);
          atomicAdd(&dK[kv + c], gm.scale * dss[k] * qs[c]);
        }
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int j = 0; j < NC; ++j) dQ[qrow + lane + 64 * j] = dq[j] * gm.scale;
}

hipError_t launch_attn_fwd_fp32(const Geom &g, const float *Q, const float *K, const float *V, const int32_t *sel,
                                float *O, float *LSE, hipStream_t s) {
  dim3 grid(g.Lq, g.Hq, g.B);
  timing_begin("phsa_attn_fwd_fp32", s);
  if (g.d == 128)
    hipLaunchKernelGGL(attn_fwd_fp32_kernel<128>, grid, dim3(64), 0, s, Q, K, V, sel, O, LSE, g);
  else
    hipLaunchKernelGGL(attn_fwd_fp32_kernel<64>, grid, dim3(64), 0, s, Q, K, V, sel, O, LSE, g);
  timing_end(s);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_fp32(const Geom &g, const float *Q, const float *K, const float *V, const float *O,
                                const float *dO, const float *LSE, const int32_t *sel, float *dQ, float *dK, float *dV,
                                float *Dvec, hipStream_t s) {
  hipError_t e = launch_bwd_pre(g, O, dO, Dvec, s);
  if (e != hipSuccess) return e;
  const int64_t nkv = (int64_t)g.B * g.Lk * g.Hkv * g.d;
  hipLaunchKernelGGL(zero_kernel, dim3(1024), dim3(256), 0, s, dK, nkv);
  hipLaunchKernelGGL(zero_kernel, dim3(1024), dim3(256), 0, s, dV, nkv);
  dim3 grid(g.Lq, g.Hq, g.B);
  timing_begin("phsa_attn_bwd_fp32", s);
  if (g.d == 128)
    hipLaunchKernelGGL(attn_bwd_fp32_kernel<128>, grid, dim3(64), 0, s, Q, K, V, dO, LSE, Dvec, sel, dQ, dK, dV, g);
  else
    hipLaunchKernelGGL(attn_bwd_fp32_kernel<64>, grid, dim3(64), 0, s, Q, K, V, dO, LSE, Dvec, sel, dQ, dK, dV, g);
  timing_end(s);
  return hipGetLastError();
}

}  // namespace phsa

// One decode step with a block KV cache: each of B sequences has one new
// query at position Lk - 1 (its key/value are already in the cache), scores
// the cache's T block representatives, selects, and attends over the chosen
// blocks (Eq. 8, Algorithm 1 selection, Eq. 10-11).  All three kernels are
// memory-bound: the representatives and the selected K/V blocks are each
// read once.
//
//   decode_select  : one workgroup per (b, g).  Waves score blocks with
//                    coalesced 512-byte reads of K_comp rows and a wave sum;
//                    wave 0 then takes the top-k by successive maxima of the
//                    strict order (score desc, block asc), each round looking
//                    only below the previous winner.
//   decode_attn    : one workgroup per (slot, b, g): the block's K/V tile is
//                    staged in LDS as float32, each wave does one head's
//                    softmax over the 64 keys, and the partial (o / l, m, l)
//                    goes to the workspace.
//   decode_combine : one wave per (b, g) merges the partials.
#include <float.h>
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool beats_d(float s1, int t1, float s2, int t2) {
  return s1 > s2 || (s1 == s2 && t1 < t2);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void decode_select_kernel(const T *__restrict__ Q, const float *__restrict__ Kc,
                                                            int32_t *__restrict__ sel, Geom gm) {
  extern __shared__ float sc[];  // [T]
  __shared__ float qsum[D];
  const int bg = blockIdx.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int c = tid; c < D; c += 256) {
    float a = 0.f;
    for (int hh = 0; hh < gm.G; ++hh) a += to_f32<T>(Q[((int64_t)b * gm.Hq + g * gm.G + hh) * D + c]);
    qsum[c] = a;
  }
  __syncthreads();
  const int cur = gm.T - 1;
  const int lo = max(0, cur - gm.window / gm.m);
  const float *kc = Kc + (int64_t)bg * gm.T * D;
  for (int t = gm.n_init + wave; t < lo; t += 4) {
    float a = 0.f;
#pragma unroll
    for (int c = lane; c < D; c += 64) a = fmaf(qsum[c], kc[(int64_t)t * D + c], a);
    a = wave_sum(a);
    if (lane == 0) sc[t] = a * gm.scale;
  }
  __syncthreads();
  if (wave != 0) return;

  const int nc = max(0, lo - gm.n_init);
  const int npick = min(gm.top_k, nc);
  float ps = FLT_MAX;  // previous winner (strictly better than everything left)
  int pt = -1;
  int mine = 0x7fffffff;
  for (int p = 0; p < npick; ++p) {
    float bs = -FLT_MAX;
    int bt = 0x7fffffff;
    for (int t = gm.n_init + lane; t < lo; t += 64) {
      const float s = sc[t];
      if (beats_d(ps, pt, s, t) && beats_d(s, t, bs, bt)) {
        bs = s;
        bt = t;
      }
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float os = __shfl_xor(bs, o, 64);
      const int ot = __shfl_xor(bt, o, 64);
      if (beats_d(os, ot, bs, bt)) {
        bs = os;
        bt = ot;
      }
    }
    if (lane == p) mine = bt;
    ps = bs;
    pt = bt;
  }
  // ascending order of the picks: rank = number of smaller picks
  int rank = 0;
  for (int j = 0; j < npick; ++j) rank += (__shfl(mine, j, 64) < mine);
  int32_t *out = sel + (int64_t)bg * gm.ksel;
  const int ni = min(gm.n_init, cur + 1);
  const int lstart = max(lo, ni);
  const int nlocal = cur - lstart + 1;
  if (lane < ni) out[lane] = lane;
  if (lane < npick) out[ni + rank] = mine;
  if (lane < nlocal) out[ni + npick + lane] = lstart + lane;
  for (int x = ni + npick + nlocal + lane; x < gm.ksel; x += 64) out[x] = -1;
}

template <typename T, int D>
__global__ __launch_bounds__(256) void decode_attn_kernel(const T *__restrict__ Q, const T *__restrict__ K,
                                                          const T *__restrict__ V, const int32_t *__restrict__ sel,
                                                          float *__restrict__ part, Geom gm) {
  __shared__ float Kf[64][D + 1];
  __shared__ float Vf[64][D];
  __shared__ float ps[8][64];
  __shared__ float qf[8][D];
  __shared__ float mls[8][2];
  const int slot = blockIdx.x, bg = blockIdx.y, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cur = gm.T - 1, pos = gm.Lk - 1;
  const int t = sel[(int64_t)bg * gm.ksel + slot];
  if (t < 0 || t > cur || t >= gm.T) return;
  constexpr int VEC = 16 / sizeof(T);
  for (int x = tid; x < 64 * D / VEC; x += 256) {
    const int kk = x / (D / VEC), c = (x % (D / VEC)) * VEC;
    const int64_t src = (((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g) * D + c;
    const uint4 rk = *reinterpret_cast<const uint4 *>(K + src);
    const uint4 rv = *reinterpret_cast<const uint4 *>(V + src);
    const T *pk = reinterpret_cast<const T *>(&rk);
    const T *pv = reinterpret_cast<const T *>(&rv);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      Kf[kk][c + e] = to_f32<T>(pk[e]);
      Vf[kk][c + e] = to_f32<T>(pv[e]);
    }
  }
  for (int x = tid; x < gm.G * D; x += 256) qf[x / D][x % D] = to_f32<T>(Q[((int64_t)b * gm.Hq + g * gm.G) * D + x]);
  __syncthreads();
  for (int hh = wave; hh < gm.G; hh += 4) {
    float a = 0.f;
#pragma unroll 8
    for (int c = 0; c < D; ++c) a = fmaf(qf[hh][c], Kf[lane][c], a);
    const float s = (t * 64 + lane) <= pos ? a * gm.scale : -INFINITY;
    const float m = wave_max(s);
    const float p = expf(s - m);
    const float l = wave_sum(p);
    ps[hh][lane] = p;
    if (lane == 0) {
      mls[hh][0] = m;
      mls[hh][1] = l;
    }
  }
  __syncthreads();
  for (int x = tid; x < gm.G * D; x += 256) {
    const int hh = x / D, c = x - hh * D;
    float o = 0.f;
#pragma unroll 8
    for (int k = 0; k < 64; ++k) o = fmaf(ps[hh][k], Vf[k][c], o);
    float *dst = part + (((int64_t)bg * gm.ksel + slot) * gm.G + hh) * (D + 2);
    dst[c] = o / mls[hh][1];
    if (c == 0) {
      dst[D] = mls[hh][0];
      dst[D + 1] = mls[hh][1];
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(const int32_t *__restrict__ sel,
                                                             const float *__restrict__ part, T *__restrict__ O,
                                                             float *__restrict__ LSE, Geom gm) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int bg = blockIdx.x * 4 + wave;
  if (bg >= gm.B * gm.Hkv) return;
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int cur = gm.T - 1;
  const int tl = lane < gm.ksel ? sel[(int64_t)bg * gm.ksel + lane] : -1;
  const uint64_t valid = __ballot(tl >= 0 && tl <= cur && tl < gm.T);
  for (int e = lane; e < gm.G * D; e += 64) {
    const int hh = e / D, c = e - hh * D;
    float M = -INFINITY;
    for (uint64_t v = valid; v; v &= v - 1) {
      const int s = __ffsll((long long)v) - 1;
      M = fmaxf(M, part[(((int64_t)bg * gm.ksel + s) * gm.G + hh) * (D + 2) + D]);
    }
    float L = 0.f, acc = 0.f;
    for (uint64_t v = valid; v; v &= v - 1) {
      const int s = __ffsll((long long)v) - 1;
      const float *p = part + (((int64_t)bg * gm.ksel + s) * gm.G + hh) * (D + 2);
      const float w = p[D + 1] * expf(p[D] - M);
      L += w;
      acc = fmaf(w, p[c], acc);
    }
    O[((int64_t)b * gm.Hq + g * gm.G + hh) * D + c] = from_f32<T>(L > 0.f ? acc / L : 0.f);
    if (c == 0) LSE[(int64_t)b * gm.Hq + g * gm.G + hh] = L > 0.f ? M + logf(L) : -INFINITY;
  }
}

template <typename T, int D>
static hipError_t launch_decode_t(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc,
                                  int32_t *sel, void *O, float *LSE, float *part, hipStream_t s) {
  timing_begin("phsa_decode_select", s);
  hipLaunchKernelGGL((decode_select_kernel<T, D>), dim3(g.B * g.Hkv), dim3(256), (size_t)g.T * sizeof(float), s,
                     static_cast<const T *>(Q), Kc, sel, g);
  timing_end(s);
  timing_begin("phsa_decode_attn", s);
  hipLaunchKernelGGL((decode_attn_kernel<T, D>), dim3(g.ksel, g.B * g.Hkv), dim3(256), 0, s,
                     static_cast<const T *>(Q), static_cast<const T *>(K), static_cast<const T *>(V), sel, part, g);
  timing_end(s);
  timing_begin("phsa_decode_combine", s);
  hipLaunchKernelGGL((decode_combine_kernel<T, D>), dim3((g.B * g.Hkv + 3) / 4), dim3(256), 0, s, sel, part,
                     static_cast<T *>(O), LSE, g);
  timing_end(s);
  return hipGetLastError();
}

hipError_t launch_decode(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc, int32_t *sel,
                         void *O, float *LSE, float *part, hipStream_t s) {
  if (g.dtype == 0)
    return g.d == 128 ? launch_decode_t<bf16_t, 128>(g, Q, K, V, Kc, sel, O, LSE, part, s)
                      : launch_decode_t<bf16_t, 64>(g, Q, K, V, Kc, sel, O, LSE, part, s);
  return g.d == 128 ? launch_decode_t<float, 128>(g, Q, K, V, Kc, sel, O, LSE, part, s)
                    : launch_decode_t<float, 64>(g, Q, K, V, Kc, sel, O, LSE, part, s);
}

}  // namespace phsa

// Sparse attention forward, bf16 (Eq. 10-11; Algorithm 1 attention step).
//
// Work is key-block-major.  Every query row selects its own blocks, so the
// only operand that many rows share is a key/value block.  A workgroup takes
// one work unit = one (b, g, t) block plus up to unit_tokens entries of the
// list of rows that selected it, keeps K_t (row-major) and V_t (transposed)
// in LDS for the whole unit, and streams the rows through it in chunks of
// 64 MFMA rows (64 / G tokens x G heads of the group):
//
//   S = Q_chunk K_t^T            16x16x32 bf16 MFMA, fp32 accumulate
//   m = rowmax(S), P = exp(S - m), l = rowsum(P)   (token-level causal mask)
//   O_part = (P V_t) / l          16x16x32 bf16 MFMA
//
// and writes, per (row, slot), the partial output O_part (bf16) and its
// (m, l) pair (log2 units).  A second kernel merges the at most Ksel
// partials of each row into the exact softmax over the union:
//   M = max_s m_s,  L = sum_s l_s 2^(m_s - M),  O = sum_s (l_s 2^(m_s - M) / L) O_part_s,
//   LSE = (M + log2 L) ln 2.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool slot_ok(int t, int cur, int T) { return t >= 0 && t <= cur && t < T; }

template <int D, int G>
__global__ __launch_bounds__(256) void attn_fwd_sparse_kernel(const bf16_t *__restrict__ Q,
                                                              const bf16_t *__restrict__ K,
                                                              const bf16_t *__restrict__ V, Geom gm, IndexWs ix,
                                                              bf16_t *__restrict__ opart, float2 *__restrict__ ml) {
  constexpr int CT = 64 / G;   // query tokens per chunk
  constexpr int KP = D + 8;    // padded LDS row (elements) of K and Q tiles
  constexpr int VP = 64 + 8;   // padded LDS row of the transposed V tile and of P
  constexpr int VPR = D / 8;   // 16-byte vectors per row
  __shared__ __attribute__((aligned(16))) bf16_t Ks[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VP];
  __shared__ __attribute__((aligned(16))) bf16_t Qs[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Ps[4][16 * VP];
  __shared__ int ent[CT];

  const int u = blockIdx.x;
  if (u >= ix.totals[1]) return;
  const int2 unit = ix.units[u];
  const int bgt = unit.x, e0 = unit.y;
  const int n_ent = min(ix.cnt[bgt] - e0, ix.unit_tokens);
  const int bg = bgt / gm.T, t = bgt - bg * gm.T;
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  const int32_t *list = ix.tok + ix.off[bgt] + e0;

  for (int x = tid; x < 64 * VPR; x += 256) {
    const int kk = x / VPR, c = (x % VPR) * 8;
    const int64_t grow = ((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g;
    *reinterpret_cast<uint4 *>(&Ks[kk * KP + c]) = *reinterpret_cast<const uint4 *>(K + grow * D + c);
    const uint4 vv = *reinterpret_cast<const uint4 *>(V + grow * D + c);
    const bf16_t *ve = reinterpret_cast<const bf16_t *>(&vv);
#pragma unroll
    for (int e = 0; e < 8; ++e) Vt[(c + e) * VP + kk] = ve[e];
  }
  const float sl2 = gm.scale * kLog2e;
  const int key0 = t * 64;

  for (int c0 = 0; c0 < n_ent; c0 += CT) {
    const int ntok = min(CT, n_ent - c0);
    __syncthreads();
    if (tid < CT) ent[tid] = tid < ntok ? list[c0 + tid] : -1;
    __syncthreads();
    for (int x = tid; x < 64 * VPR; x += 256) {
      const int r = x / VPR, c = (x % VPR) * 8;
      const int e = ent[r / G];
      uint4 qv = make_uint4(0u, 0u, 0u, 0u);
      if (e >= 0)
        qv = *reinterpret_cast<const uint4 *>(Q + (((int64_t)b * gm.Lq + (e >> 6)) * gm.Hq + g * G + (r % G)) * D + c);
      *reinterpret_cast<uint4 *>(&Qs[r * KP + c]) = qv;
    }
    __syncthreads();

    // S for this wave's 16 rows x 64 keys
    f32x4 s[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) s[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int arow = wave * 16 + l16;
#pragma unroll
    for (int kb = 0; kb < D; kb += 32) {
      const bf16x8 a = load_bf16x8(&Qs[arow * KP + kb + kq]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) s[nt] = mfma16x16x32(a, load_bf16x8(&Ks[(nt * 16 + l16) * KP + kb + kq]), s[nt]);
    }

    float mrow[4], lrow[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = wave * 16 + q4 * 4 + r;
      const int e = ent[row / G];
      const int pos = e >= 0 ? gm.q_pos0 + (e >> 6) : -1;
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int key = key0 + nt * 16 + l16;
        const float v = key <= pos ? s[nt][r] * sl2 : -INFINITY;
        s[nt][r] = v;
        mx = fmaxf(mx, v);
      }
      mx = max16(mx);
      if (mx == -INFINITY) mx = 0.f;
      float l = 0.f;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const float p = exp2f(s[nt][r] - mx);
        s[nt][r] = p;
        l += p;
      }
      mrow[r] = mx;
      lrow[r] = sum16(l);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) Ps[wave][(q4 * 4 + r) * VP + nt * 16 + l16] = f32_to_bf16(s[nt][r]);
    __syncthreads();

    f32x4 o[D / 16];
#pragma unroll
    for (int nt = 0; nt < D / 16; ++nt) o[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 64; kb += 32) {
      const bf16x8 a = load_bf16x8(&Ps[wave][l16 * VP + kb + kq]);
#pragma unroll
      for (int nt = 0; nt < D / 16; ++nt) o[nt] = mfma16x16x32(a, load_bf16x8(&Vt[(nt * 16 + l16) * VP + kb + kq]), o[nt]);
    }

#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = wave * 16 + q4 * 4 + r;
      const int e = ent[row / G];
      if (l16 == 0 && e >= 0)
        ml[(((int64_t)bg * gm.Lq + (e >> 6)) * gm.ksel + (e & 63)) * G + row % G] = make_float2(mrow[r], lrow[r]);
      const float inv = lrow[r] > 0.f ? 1.f / lrow[r] : 0.f;
#pragma unroll
      for (int nt = 0; nt < D / 16; ++nt) Qs[row * KP + nt * 16 + l16] = f32_to_bf16(o[nt][r] * inv);
    }
    __syncthreads();
    for (int x = lane; x < 16 * VPR; x += 64) {
      const int row = wave * 16 + x / VPR, c = (x % VPR) * 8;
      const int e = ent[row / G];
      if (e >= 0)
        *reinterpret_cast<uint4 *>(opart + ((((int64_t)bg * gm.Lq + (e >> 6)) * gm.ksel + (e & 63)) * G + row % G) * D + c) =
            *reinterpret_cast<const uint4 *>(&Qs[row * KP + c]);
    }
  }
}

// One wave per (b, g, query row): merge the row's per-slot partials.
template <int D, int G>
__global__ __launch_bounds__(256) void attn_fwd_combine_kernel(const int32_t *__restrict__ sel,
                                                               const bf16_t *__restrict__ opart,
                                                               const float2 *__restrict__ ml, bf16_t *__restrict__ O,
                                                               float *__restrict__ LSE, Geom gm) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t x = (int64_t)blockIdx.x * 4 + wave;  // bg * Lq + i
  if (x >= (int64_t)gm.B * gm.Hkv * gm.Lq) return;
  const int bg = (int)(x / gm.Lq), i = (int)(x - (int64_t)bg * gm.Lq);
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int cur = (gm.q_pos0 + i) / gm.m;
  const int tl = lane < gm.ksel ? sel[x * gm.ksel + lane] : -1;
  const uint64_t valid = __ballot(slot_ok(tl, cur, gm.T));
  const int64_t base = x * gm.ksel;
  for (int e = lane * 4; e < G * D; e += 256) {
    const int hh = e / D, c = e - hh * D;
    float M = -INFINITY;
    for (uint64_t v = valid; v; v &= v - 1) M = fmaxf(M, ml[(base + __ffsll((long long)v) - 1) * G + hh].x);
    float L = 0.f, acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, acc3 = 0.f;
    for (uint64_t v = valid; v; v &= v - 1) {
      const int64_t sl = base + __ffsll((long long)v) - 1;
      const float2 q = ml[sl * G + hh];
      const float w = q.y * exp2f(q.x - M);
      L += w;
      const uint2 raw = *reinterpret_cast<const uint2 *>(opart + (sl * G + hh) * D + c);
      const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw);
      acc0 = fmaf(w, bf16_to_f32(pv[0]), acc0);
      acc1 = fmaf(w, bf16_to_f32(pv[1]), acc1);
      acc2 = fmaf(w, bf16_to_f32(pv[2]), acc2);
      acc3 = fmaf(w, bf16_to_f32(pv[3]), acc3);
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    bf16_t outv[4] = {f32_to_bf16(acc0 * inv), f32_to_bf16(acc1 * inv), f32_to_bf16(acc2 * inv),
                      f32_to_bf16(acc3 * inv)};
    *reinterpret_cast<uint2 *>(O + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + c) =
        *reinterpret_cast<const uint2 *>(outv);
    if (c == 0) LSE[((int64_t)b * gm.Hq + g * G + hh) * gm.Lq + i] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  }
}

template <int D, int G>
static hipError_t launch_fwd_t(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel,
                               void *O, float *LSE, const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  timing_begin("phsa_attn_fwd_sparse", s);
  hipLaunchKernelGGL((attn_fwd_sparse_kernel<D, G>), dim3((unsigned)ix.units_max), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     g, ix, static_cast<bf16_t *>(opart), ml);
  timing_end(s);
  const int64_t rows = (int64_t)g.B * g.Hkv * g.Lq;
  timing_begin("phsa_attn_fwd_combine", s);
  hipLaunchKernelGGL((attn_fwd_combine_kernel<D, G>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, sel,
                     static_cast<const bf16_t *>(opart), ml, static_cast<bf16_t *>(O), LSE, g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_fwd_d(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel,
                               void *O, float *LSE, const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_fwd_t<D, 1>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s);
    case 2: return launch_fwd_t<D, 2>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s);
    case 4: return launch_fwd_t<D, 4>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s);
    default: return launch_fwd_t<D, 8>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s);
  }
}

hipError_t launch_attn_fwd(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel,
                           void *O, float *LSE, const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  hipError_t e = launch_build_index(g, sel, ix, s);
  if (e != hipSuccess) return e;
  return g.d == 128 ? launch_fwd_d<128>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s)
                    : launch_fwd_d<64>(g, Q, K, V, sel, O, LSE, ix, opart, ml, s);
}

}  // namespace phsa

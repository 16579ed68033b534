// Sparse attention backward, bf16, with the selection held fixed.
//
// With s_ij = scale * q_i.k_j, P_ij = exp(s_ij - LSE_i), D_i = dO_i . O_i:
//   dV_j = sum_i P_ij dO_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dQ_i = scale * sum_j dS_ij k_j
//   dK_j = scale * sum_i dS_ij q_i
// where i ranges over the query rows (all heads of the group) that selected
// the block of key j and are causally allowed to see j.
//
// Like the forward, the main kernel is key-block-major over the inverted
// index.  A work unit keeps K_t and V_t in LDS and its 64 x d dK_t / dV_t
// accumulators in registers (wave w owns keys 16w..16w+15), and streams the
// unit's query rows through in chunks of 64 MFMA rows.  Per chunk, per wave:
//   S^T  = K_w Q^T,  dP^T = V_w dO^T          (keys x rows; 16x16x32 MFMA)
//   P^T, dS^T elementwise from LSE and D
//   dV_w += P^T dO,  dK_w += dS^T Q           (rows contracted; transposed Q, dO tiles)
//   dQ_rows = dS K_t                          (keys contracted over all 4 waves)
// dQ leaves as one bf16 partial per (row, slot), summed by a per-row kernel.
// dK/dV leave directly (bf16) when the unit covers its whole block, else as
// float32 partials that a per-block kernel sums; blocks nobody selected get
// zeros from that kernel too.
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool slot_ok_b(int t, int cur, int T) { return t >= 0 && t <= cur && t < T; }

// D = rowsum(dO * O) per (b, h, i), float32.
template <typename T, int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const T *__restrict__ O, const T *__restrict__ dO,
                                                      float *__restrict__ Dvec, Geom gm) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (b, i, h)
  if (x >= (int64_t)gm.B * gm.Lq * gm.Hq) return;
  const int h = (int)(x % gm.Hq);
  const int64_t bi = x / gm.Hq;
  const int i = (int)(bi % gm.Lq), b = (int)(bi / gm.Lq);
  const T *o = O + x * D;
  const T *d = dO + x * D;
  float acc = 0.f;
  constexpr int V = 16 / sizeof(T);
  for (int c = 0; c < D; c += V) {
    const uint4 ro = *reinterpret_cast<const uint4 *>(o + c);
    const uint4 rd = *reinterpret_cast<const uint4 *>(d + c);
    const T *po = reinterpret_cast<const T *>(&ro);
    const T *pd = reinterpret_cast<const T *>(&rd);
#pragma unroll
    for (int e = 0; e < V; ++e) acc = fmaf(to_f32<T>(po[e]), to_f32<T>(pd[e]), acc);
  }
  Dvec[((int64_t)b * gm.Hq + h) * gm.Lq + i] = acc;
}

template <int D, int G>
__global__ __launch_bounds__(256) void attn_bwd_sparse_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ V,
    const bf16_t *__restrict__ dO, const float *__restrict__ LSE, const float *__restrict__ Dvec, Geom gm, IndexWs ix,
    bf16_t *__restrict__ dqpart, bf16_t *__restrict__ dK, bf16_t *__restrict__ dV, float *__restrict__ dkvpart) {
  constexpr int CT = 64 / G;
  constexpr int KP = D + 8;   // row-major tiles [64][KP]
  constexpr int RP = 64 + 8;  // transposed tiles [D][RP] and P/dS tiles [.][RP]
  constexpr int VPR = D / 8;
  constexpr int NT = D / 16;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[D * RP];
  __shared__ __attribute__((aligned(16))) bf16_t Qs[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[64 * KP];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[D * RP];
  __shared__ __attribute__((aligned(16))) bf16_t dOt[D * RP];
  __shared__ __attribute__((aligned(16))) bf16_t PTs[4][16 * RP];
  __shared__ __attribute__((aligned(16))) bf16_t dSTs[4][16 * RP];
  __shared__ __attribute__((aligned(16))) bf16_t dSs[64 * RP];
  __shared__ float lse_s[64], dd_s[64];
  __shared__ int pos_s[64];
  __shared__ int ent[CT];

  const int u = blockIdx.x;
  if (u >= ix.totals[1]) return;
  const int2 unit = ix.units[u];
  const int bgt = unit.x, e0 = unit.y;
  const int cnt = ix.cnt[bgt];
  const int n_ent = min(cnt - e0, ix.unit_tokens);
  const bool whole_block = (e0 == 0) && (n_ent == cnt);
  const int bg = bgt / gm.T, t = bgt - bg * gm.T;
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  const int32_t *list = ix.tok + ix.off[bgt] + e0;

  for (int x = tid; x < 64 * VPR; x += 256) {
    const int kk = x / VPR, c = (x % VPR) * 8;
    const int64_t grow = ((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g;
    const uint4 kv = *reinterpret_cast<const uint4 *>(K + grow * D + c);
    *reinterpret_cast<uint4 *>(&Ks[kk * KP + c]) = kv;
    *reinterpret_cast<uint4 *>(&Vs[kk * KP + c]) = *reinterpret_cast<const uint4 *>(V + grow * D + c);
    const bf16_t *ke = reinterpret_cast<const bf16_t *>(&kv);
#pragma unroll
    for (int e = 0; e < 8; ++e) Kt[(c + e) * RP + kk] = ke[e];
  }

  f32x4 dk[NT], dv[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) dk[n] = dv[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float sl2 = gm.scale * kLog2e;
  const int key_base = t * 64 + wave * 16 + q4 * 4;  // key of accumulator element r is key_base + r

  for (int c0 = 0; c0 < n_ent; c0 += CT) {
    const int ntok = min(CT, n_ent - c0);
    __syncthreads();
    if (tid < CT) ent[tid] = tid < ntok ? list[c0 + tid] : -1;
    __syncthreads();
    for (int x = tid; x < 64 * VPR; x += 256) {
      const int r = x / VPR, c = (x % VPR) * 8;
      const int e = ent[r / G];
      uint4 qv = make_uint4(0u, 0u, 0u, 0u), dv4 = make_uint4(0u, 0u, 0u, 0u);
      if (e >= 0) {
        const int64_t src = (((int64_t)b * gm.Lq + (e >> 6)) * gm.Hq + g * G + (r % G)) * D + c;
        qv = *reinterpret_cast<const uint4 *>(Q + src);
        dv4 = *reinterpret_cast<const uint4 *>(dO + src);
      }
      *reinterpret_cast<uint4 *>(&Qs[r * KP + c]) = qv;
      *reinterpret_cast<uint4 *>(&dOs[r * KP + c]) = dv4;
      const bf16_t *qe = reinterpret_cast<const bf16_t *>(&qv);
      const bf16_t *de = reinterpret_cast<const bf16_t *>(&dv4);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        Qt[(c + k) * RP + r] = qe[k];
        dOt[(c + k) * RP + r] = de[k];
      }
    }
    if (tid < 64) {
      const int e = ent[tid / G];
      if (e >= 0) {
        const int i = e >> 6, h = g * G + tid % G;
        lse_s[tid] = LSE[((int64_t)b * gm.Hq + h) * gm.Lq + i] * kLog2e;
        dd_s[tid] = Dvec[((int64_t)b * gm.Hq + h) * gm.Lq + i];
        pos_s[tid] = gm.q_pos0 + i;
      } else {
        lse_s[tid] = 0.f;
        dd_s[tid] = 0.f;
        pos_s[tid] = -1;
      }
    }
    __syncthreads();

    // S^T and dP^T: this wave's 16 keys x 64 rows
    f32x4 st[4], dpt[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) st[n] = dpt[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int krow = wave * 16 + l16;
#pragma unroll
    for (int kb = 0; kb < D; kb += 32) {
      const bf16x8 ak = load_bf16x8(&Ks[krow * KP + kb + kq]);
      const bf16x8 av = load_bf16x8(&Vs[krow * KP + kb + kq]);
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        st[n] = mfma16x16x32(ak, load_bf16x8(&Qs[(n * 16 + l16) * KP + kb + kq]), st[n]);
        dpt[n] = mfma16x16x32(av, load_bf16x8(&dOs[(n * 16 + l16) * KP + kb + kq]), dpt[n]);
      }
    }
    // elementwise: lane holds rows n*16 + l16, keys key_base + r
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int row = n * 16 + l16;
      const float lse2 = lse_s[row], dd = dd_s[row];
      const int pos = pos_s[row];
      bf16_t dsq[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = (key_base + r) <= pos ? exp2f(st[n][r] * sl2 - lse2) : 0.f;
        const float ds = p * (dpt[n][r] - dd);
        PTs[wave][(q4 * 4 + r) * RP + row] = f32_to_bf16(p);
        dsq[r] = f32_to_bf16(ds);
        dSTs[wave][(q4 * 4 + r) * RP + row] = dsq[r];
      }
      *reinterpret_cast<uint2 *>(&dSs[row * RP + wave * 16 + q4 * 4]) = *reinterpret_cast<const uint2 *>(dsq);
    }
    __syncthreads();

    // dV += P^T dO, dK += dS^T Q (contract over the 64 chunk rows)
#pragma unroll
    for (int kb = 0; kb < 64; kb += 32) {
      const bf16x8 ap = load_bf16x8(&PTs[wave][l16 * RP + kb + kq]);
      const bf16x8 as = load_bf16x8(&dSTs[wave][l16 * RP + kb + kq]);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        dv[n] = mfma16x16x32(ap, load_bf16x8(&dOt[(n * 16 + l16) * RP + kb + kq]), dv[n]);
        dk[n] = mfma16x16x32(as, load_bf16x8(&Qt[(n * 16 + l16) * RP + kb + kq]), dk[n]);
      }
    }
    // dQ for rows 16w..16w+15 = dS (rows x 64 keys) K (64 keys x D)
    f32x4 dq[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) dq[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 64; kb += 32) {
      const bf16x8 a = load_bf16x8(&dSs[(wave * 16 + l16) * RP + kb + kq]);
#pragma unroll
      for (int n = 0; n < NT; ++n) dq[n] = mfma16x16x32(a, load_bf16x8(&Kt[(n * 16 + l16) * RP + kb + kq]), dq[n]);
    }
    // stage scaled dQ rows of this wave in Qs (all reads of Qs are done) and write them out
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = wave * 16 + q4 * 4 + r;
#pragma unroll
      for (int n = 0; n < NT; ++n) Qs[row * KP + n * 16 + l16] = f32_to_bf16(dq[n][r] * gm.scale);
    }
    __syncthreads();
    for (int x = lane; x < 16 * VPR; x += 64) {
      const int row = wave * 16 + x / VPR, c = (x % VPR) * 8;
      const int e = ent[row / G];
      if (e >= 0)
        *reinterpret_cast<uint4 *>(dqpart + ((((int64_t)bg * gm.Lq + (e >> 6)) * gm.ksel + (e & 63)) * G + row % G) * D + c) =
            *reinterpret_cast<const uint4 *>(&Qs[row * KP + c]);
    }
  }

  // dK (scaled) / dV of this wave's 16 keys.
  if (whole_block) {
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = wave * 16 + q4 * 4 + r;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        Ks[kk * KP + n * 16 + l16] = f32_to_bf16(dk[n][r] * gm.scale);
        Vs[kk * KP + n * 16 + l16] = f32_to_bf16(dv[n][r]);
      }
    }
    __syncthreads();
    for (int x = tid; x < 64 * VPR; x += 256) {
      const int kk = x / VPR, c = (x % VPR) * 8;
      const int64_t grow = ((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g;
      *reinterpret_cast<uint4 *>(dK + grow * D + c) = *reinterpret_cast<const uint4 *>(&Ks[kk * KP + c]);
      *reinterpret_cast<uint4 *>(dV + grow * D + c) = *reinterpret_cast<const uint4 *>(&Vs[kk * KP + c]);
    }
  } else {
    float *pk = dkvpart + (int64_t)u * 2 * 64 * D;
    float *pv = pk + 64 * D;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int kk = wave * 16 + q4 * 4 + r;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        pk[kk * D + n * 16 + l16] = dk[n][r] * gm.scale;
        pv[kk * D + n * 16 + l16] = dv[n][r];
      }
    }
  }
}

// Per (b, g, t): sum float32 partials of multi-unit blocks; zero unselected blocks.
template <int D>
__global__ __launch_bounds__(256) void dkv_finalize_kernel(const float *__restrict__ dkvpart, bf16_t *__restrict__ dK,
                                                           bf16_t *__restrict__ dV, Geom gm, IndexWs ix) {
  const int bgt = blockIdx.x;
  const int u0 = ix.uoff[bgt], u1 = ix.uoff[bgt + 1];
  if (u1 - u0 == 1) return;  // written by the sparse kernel
  const int bg = bgt / gm.T, t = bgt - bg * gm.T;
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  for (int x = threadIdx.x; x < 64 * D; x += 256) {
    const int kk = x / D, c = x - kk * D;
    float sk = 0.f, sv = 0.f;
    for (int u = u0; u < u1; ++u) {
      sk += dkvpart[(int64_t)u * 2 * 64 * D + x];
      sv += dkvpart[(int64_t)u * 2 * 64 * D + 64 * D + x];
    }
    const int64_t dst = (((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g) * D + c;
    dK[dst] = f32_to_bf16(sk);
    dV[dst] = f32_to_bf16(sv);
  }
}

// One wave per (b, g, query row): dQ = sum over valid slots of the partials.
template <int D, int G>
__global__ __launch_bounds__(256) void dq_combine_kernel(const int32_t *__restrict__ sel,
                                                         const bf16_t *__restrict__ dqpart, bf16_t *__restrict__ dQ,
                                                         Geom gm) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t x = (int64_t)blockIdx.x * 4 + wave;
  if (x >= (int64_t)gm.B * gm.Hkv * gm.Lq) return;
  const int bg = (int)(x / gm.Lq), i = (int)(x - (int64_t)bg * gm.Lq);
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int cur = (gm.q_pos0 + i) / gm.m;
  const int tl = lane < gm.ksel ? sel[x * gm.ksel + lane] : -1;
  const uint64_t valid = __ballot(slot_ok_b(tl, cur, gm.T));
  const int64_t base = x * gm.ksel;
  for (int e = lane * 4; e < G * D; e += 256) {
    const int hh = e / D, c = e - hh * D;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    for (uint64_t v = valid; v; v &= v - 1) {
      const int64_t sl = base + __ffsll((long long)v) - 1;
      const uint2 raw = *reinterpret_cast<const uint2 *>(dqpart + (sl * G + hh) * D + c);
      const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw);
      a0 += bf16_to_f32(pv[0]);
      a1 += bf16_to_f32(pv[1]);
      a2 += bf16_to_f32(pv[2]);
      a3 += bf16_to_f32(pv[3]);
    }
    bf16_t outv[4] = {f32_to_bf16(a0), f32_to_bf16(a1), f32_to_bf16(a2), f32_to_bf16(a3)};
    *reinterpret_cast<uint2 *>(dQ + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + c) =
        *reinterpret_cast<const uint2 *>(outv);
  }
}

template <int D, int G>
static hipError_t launch_bwd_t(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                               const float *LSE, const int32_t *sel, void *dQ, void *dK, void *dV, const IndexWs &ix,
                               const float *Dvec, void *dqpart, float *dkvpart, hipStream_t s) {
  timing_begin("phsa_attn_bwd_sparse", s);
  hipLaunchKernelGGL((attn_bwd_sparse_kernel<D, G>), dim3((unsigned)ix.units_max), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     static_cast<const bf16_t *>(dO), LSE, Dvec, g, ix, static_cast<bf16_t *>(dqpart),
                     static_cast<bf16_t *>(dK), static_cast<bf16_t *>(dV), dkvpart);
  timing_end(s);
  timing_begin("phsa_attn_bwd_dkv_finalize", s);
  hipLaunchKernelGGL((dkv_finalize_kernel<D>), dim3(g.B * g.Hkv * g.T), dim3(256), 0, s, dkvpart,
                     static_cast<bf16_t *>(dK), static_cast<bf16_t *>(dV), g, ix);
  timing_end(s);
  const int64_t rows = (int64_t)g.B * g.Hkv * g.Lq;
  timing_begin("phsa_attn_bwd_dq_combine", s);
  hipLaunchKernelGGL((dq_combine_kernel<D, G>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, sel,
                     static_cast<const bf16_t *>(dqpart), static_cast<bf16_t *>(dQ), g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_bwd_d(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                               const float *LSE, const int32_t *sel, void *dQ, void *dK, void *dV, const IndexWs &ix,
                               const float *Dvec, void *dqpart, float *dkvpart, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_bwd_t<D, 1>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s);
    case 2: return launch_bwd_t<D, 2>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s);
    case 4: return launch_bwd_t<D, 4>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s);
    default: return launch_bwd_t<D, 8>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s);
  }
}

template <typename T, int D>
static void launch_pre(const Geom &g, const void *O, const void *dO, float *Dvec, hipStream_t s) {
  const int64_t n = (int64_t)g.B * g.Lq * g.Hq;
  timing_begin("phsa_attn_bwd_pre", s);
  hipLaunchKernelGGL((bwd_pre_kernel<T, D>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     static_cast<const T *>(O), static_cast<const T *>(dO), Dvec, g);
  timing_end(s);
}

hipError_t launch_bwd_pre(const Geom &g, const void *O, const void *dO, float *Dvec, hipStream_t s) {
  if (g.dtype == 0) {
    if (g.d == 128) launch_pre<bf16_t, 128>(g, O, dO, Dvec, s);
    else launch_pre<bf16_t, 64>(g, O, dO, Dvec, s);
  } else {
    if (g.d == 128) launch_pre<float, 128>(g, O, dO, Dvec, s);
    else launch_pre<float, 64>(g, O, dO, Dvec, s);
  }
  return hipGetLastError();
}

hipError_t launch_attn_bwd(const Geom &g, const void *Q, const void *K, const void *V, const void *O,
                           const void *dO, const float *LSE, const int32_t *sel, void *dQ, void *dK, void *dV,
                           const IndexWs &ix, float *Dvec, void *dqpart, float *dkvpart, hipStream_t s) {
  hipError_t e = launch_bwd_pre(g, O, dO, Dvec, s);
  if (e != hipSuccess) return e;
  e = launch_build_index(g, sel, ix, s);
  if (e != hipSuccess) return e;
  return g.d == 128 ? launch_bwd_d<128>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s)
                    : launch_bwd_d<64>(g, Q, K, V, dO, LSE, sel, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, s);
}

}  // namespace phsa

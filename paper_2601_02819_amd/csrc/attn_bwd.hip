// Sparse attention backward, bf16, with the selection held fixed.
//
// With s_ij = scale * q_i.k_j, P_ij = exp(s_ij - LSE_i), D_i = dO_i . O_i:
//   dV_j = sum_i P_ij dO_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dQ_i = scale * sum_j dS_ij k_j
//   dK_j = scale * sum_i dS_ij q_i
// where i ranges over the query rows (all heads of the group) that selected
// the block of key j and are causally allowed to see j.  With blocks of 16 or
// 32 tokens a 64-key tile holds several blocks; a list entry's quarter mask
// says which 16-key quarters its row selected (wave w's keys are quarter w).
//
// Like the forward, the main kernel is key-block-major over the inverted
// index.  A work unit keeps K_t and V_t in LDS (wave w owns keys
// 16w..16w+15) and the dK^T / dV^T accumulators of its keys in registers, and streams the unit's query rows through in
// chunks of 64 MFMA rows; the next chunk's gathered Q / dO rows are fetched
// into registers while the current chunk computes.  Per chunk, per wave:
//   S = Q K_w^T,  dP = dO V_w^T           (64 rows x 16 keys)
//   P, dS elementwise from LSE and D
//   dV_w^T += dO^T P,  dK_w^T += Q^T dS   (features x 16 keys; rows contracted)
//   dQ^T = K_t^T dS^T                     (features x 16 rows; all 64 keys)
// The S / dP accumulator layout is reused directly as the row-contracted
// operand (row tiles {4q..4q+3} and {16+4q..16+4q+3}); dO^T, Q^T and K_t^T
// come from the row-major tiles through transposing LDS loads, and dS
// reaches the other waves through one [key][row] LDS tile.  dQ leaves as one
// bf16 partial per list entry, stored in list order (a unit writes one
// contiguous run, non-temporal: only the merge reads it), and a per-row
// kernel sums a row's partials.  dK/dV leave
// directly (bf16) when the unit covers its whole block, else as float32
// partials that a per-block kernel sums; blocks nobody selected get zeros
// from that kernel too.
//
// The softmax scale rides in the exponent: the kernel computes P' = scale * P
// (its LSE is lowered by log2(scale)), so dS' = P' (dP - D) = scale * dS is
// already what dK and dQ need, and dV, summed from P', is divided by the scale
// once per unit.  A row that did not select a wave's quarter gets LSE = +inf in
// that wave (its weights are 2^-inf = 0), and the causal test runs only in
// chunks that reach past the first row's position.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace phsa {

// D = rowsum(dO * O) per (b, i, h), float32, stored [B, Lq, Hq] (workspace
// layout).  TPR threads cover one row with
// 16-byte loads (coalesced), then reduce with lane shuffles.
template <typename T, int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(const T *__restrict__ O, const T *__restrict__ dO,
                                                      float *__restrict__ Dvec, Geom gm) {
  constexpr int V = 16 / sizeof(T);
  constexpr int TPR = D / V;           // threads per row (8..32)
  const int64_t x = ((int64_t)blockIdx.x * 256 + threadIdx.x) / TPR;  // row (b, i, h)
  const int c = (threadIdx.x % TPR) * V;
  const bool ok = x < (int64_t)gm.B * gm.Lq * gm.Hq;
  float acc = 0.f;
  if (ok) {
    const uint4 ro = *reinterpret_cast<const uint4 *>(O + x * D + c);
    const uint4 rd = *reinterpret_cast<const uint4 *>(dO + x * D + c);
    const T *po = reinterpret_cast<const T *>(&ro);
    const T *pd = reinterpret_cast<const T *>(&rd);
#pragma unroll
    for (int e = 0; e < V; ++e) acc = fmaf(to_f32<T>(po[e]), to_f32<T>(pd[e]), acc);
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) acc += __shfl_xor(acc, o, 64);
  if (ok && c == 0) Dvec[x] = acc;  // [B, Lq, Hq], the row order of O
}

// P' and dS' of one 16-row tile (lane (q, j): rows 4q..4q+3, key j); CAUSAL
// zeroes the weights of keys past a row's position.
template <bool CAUSAL>
__device__ __forceinline__ void bwd_p_ds(f32x4 &s, f32x4 &dp, const float4 lse4, const float4 dd4, const int4 pos4,
                                         int key, float sl2, bf16_t dsq[4]) {
  const float lsev[4] = {lse4.x, lse4.y, lse4.z, lse4.w};
  const float ddv[4] = {dd4.x, dd4.y, dd4.z, dd4.w};
  const int posv[4] = {pos4.x, pos4.y, pos4.z, pos4.w};
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float p = __builtin_amdgcn_exp2f(fmaf(s[r], sl2, -lsev[r]));
    if (CAUSAL) p = key <= posv[r] ? p : 0.f;
    const float ds = p * (dp[r] - ddv[r]);
    s[r] = p;
    dp[r] = ds;
    dsq[r] = f32_to_bf16(ds);
  }
}

template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_bwd_sparse_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ V,
    const bf16_t *__restrict__ dO, const float *__restrict__ LSE, const float *__restrict__ Dvec, Geom gm, IndexWs ix,
    bf16_t *__restrict__ dqpart, bf16_t *__restrict__ dK, bf16_t *__restrict__ dV, float *__restrict__ dkvpart,
    const float *__restrict__ bkv) {
  constexpr int CT = 64 / G;
  // Row-major [row][d] tiles.  The pitch decides the banks of the 16-byte
  // fragment reads (rows 16m + l16, chunk q4) and of the transposing reads: with
  // D + 16 elements (288 bytes) both are nearly conflict-free, with D + 8 they
  // conflict.  Q, dO and K (read transposed every chunk) get D + 16; V, read
  // only as one row fragment per wave per chunk, is unpadded and swizzled
  // (swz), which holds the workgroup under 80 KB (two per CU).
  constexpr int KPQ = D + 16;
  // pitch of the [key][row] dS tile; the 8-element pad of its 64 rows holds the
  // chunk's per-wave LSE: row 16w + 4mt + q, as 4 floats, those of rows
  // 16mt + 4q .. +3 in wave w
  constexpr int RP = 64 + 8;
  constexpr int VPR = D / 8;
  constexpr int NV = 64 * VPR / 256;
  constexpr int KB = D / 32;
  constexpr int NT = D / 16;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[64 * KPQ];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[64 * D];
  __shared__ __attribute__((aligned(16))) bf16_t Qs[64 * KPQ];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[64 * KPQ];
  __shared__ __attribute__((aligned(16))) bf16_t dSt[64 * RP];
  __shared__ __attribute__((aligned(16))) float dd_s[64];
  __shared__ __attribute__((aligned(16))) int pos_s[64];

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
  // list position of the unit's first entry, read once (a load inside the chunk loop
  // would make the wait for it also wait for the prefetched rows)
  const int64_t list0 = (int64_t)ix.off[bgt] + e0;
  const int32_t *list = ix.tok + list0;
  const int64_t krow0 = ((int64_t)b * gm.Lk + (int64_t)t * 64) * gm.Hkv + g;  // global row of key 0
  // the group's first head of sequence b; a row's head h, query i is at i * Hq * D + (h - gG) * D
  const int64_t qb0 = ((int64_t)b * gm.Lq * gm.Hq + g * G) * D;
  const int hqd = gm.Hq * D;
  const float *lse_b = LSE + ((int64_t)b * gm.Hq + g * G) * gm.Lq;  // [G][Lq] of the group
  const float *dd_b = Dvec + (int64_t)b * gm.Lq * gm.Hq + g * G;     // [Lq][Hq] from the group's first head

  for (int x = tid; x < 64 * VPR; x += 256) {
    const int kk = x / VPR, c = (x % VPR) * 8;
    const int64_t src = (krow0 + (int64_t)kk * gm.Hkv) * D + c;
    *reinterpret_cast<uint4 *>(&Ks[kk * KPQ + c]) = *reinterpret_cast<const uint4 *>(K + src);
    *reinterpret_cast<uint4 *>(&Vs[swz<D>(kk, c)]) = *reinterpret_cast<const uint4 *>(V + src);
  }
  // dK^T / dV^T accumulators: lane (q, j) holds feature 16nt + 4q + r of key 16w + j
  f32x4 dkt[NT], dvt[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) dkt[n] = dvt[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Row gather, pipelined two deep: the list entries of chunk c + 2 are read
  // while the rows of chunk c + 1 are fetched, which is while chunk c computes.
  // Rows past the list's end fetch the last entry's row again (finite values
  // whose weights are zero: their LSE is +inf).
  int ne[NV], nrow = -1;               // list entries of the next chunk to fetch
  u32x4 pq[NV], pd[NV];
  float plse = 0.f, pdd = 0.f;
  int ppos = 0;
  auto load_entries = [&](int c0) {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int tk = ((tid + 256 * k) / VPR) / G;
      ne[k] = list[min(c0 + tk, n_ent - 1)];
    }
    const int tk = tid / G;
    nrow = (tid < 64 && c0 + tk < n_ent) ? list[c0 + tk] : -1;
  };
  auto fetch_rows = [&]() {
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int v = tid + 256 * k, r = v / VPR, c = (v % VPR) * 8;
      const int64_t src = qb0 + (int64_t)(ne[k] >> 10) * hqd + ((r % G) * D + c);
      pq[k] = *reinterpret_cast<const u32x4 *>(Q + src);
      pd[k] = *reinterpret_cast<const u32x4 *>(dO + src);
    }
    if (tid < 64) {
      if (nrow >= 0) {
        const int i = nrow >> 10;
        plse = lse_b[(tid % G) * gm.Lq + i];  // scaled when staged, so nothing waits here
        pdd = dd_b[i * gm.Hq + tid % G];
        ppos = (gm.q_pos0 + i) | (((nrow >> 6) & 15) << 27);  // position, and the quarters the row attends to
      } else {
        plse = 0.f;
        pdd = 0.f;
        ppos = 0;  // no quarter: nothing allowed
      }
    }
  };
  load_entries(0);
  fetch_rows();
  load_entries(CT);

  const float sl2 = gm.scale * kLog2e;
  const float lsc = __log2f(gm.scale);       // P' = scale * P
  const float inv_scale = 1.f / gm.scale;
  const int key = t * 64 + wave * 16 + l16;  // the key whose S column this lane holds

  for (int c0 = 0; c0 < n_ent; c0 += CT) {
    __syncthreads();  // previous chunk is done with Qs, dOs, dSt and the row tables
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int v = tid + 256 * k, r = v / VPR, c = (v % VPR) * 8;
      *reinterpret_cast<u32x4 *>(&Qs[r * KPQ + c]) = pq[k];
      *reinterpret_cast<u32x4 *>(&dOs[r * KPQ + c]) = pd[k];
    }
    if (tid < 64) {
      const float l = plse * kLog2e - lsc;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        reinterpret_cast<float *>(&dSt[(w * 16 + (tid >> 2)) * RP + 64])[tid & 3] =
            (ppos >> (27 + w)) & 1 ? l : INFINITY;
      dd_s[tid] = pdd;
      pos_s[tid] = ppos & 0x7ffffff;
    }
    __syncthreads();
    if (c0 + CT < n_ent) {
      fetch_rows();
      load_entries(c0 + 2 * CT);
    }

    // S and dP: 64 rows (4 tiles) x this wave's 16 keys; lane (q, j) holds rows 16mt + 4q + r of key j
    f32x4 s[4], dp[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) s[mt] = dp[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const bf16x8 kf = load_bf16x8(&Ks[(wave * 16 + l16) * KPQ + kb * 32 + kq]);
      const bf16x8 vf = load_bf16x8(&Vs[swz<D>(wave * 16 + l16, kb * 32 + kq)]);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        s[mt] = mfma16x16x32(load_bf16x8(&Qs[(mt * 16 + l16) * KPQ + kb * 32 + kq]), kf, s[mt]);
        dp[mt] = mfma16x16x32(load_bf16x8(&dOs[(mt * 16 + l16) * KPQ + kb * 32 + kq]), vf, dp[mt]);
      }
    }
    // P' and dS'; dS' also goes to LDS as [key][row] for the dQ product.  The
    // chunk's rows ascend: when the first one sees all of the wave's 16 keys,
    // every row does.
    const bool causal = __builtin_amdgcn_readfirstlane(pos_s[0]) < t * 64 + wave * 16 + 15;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int r0 = mt * 16 + q4 * 4;
      const float4 lse4 = *reinterpret_cast<const float4 *>(&dSt[(wave * 16 + mt * 4 + q4) * RP + 64]);
      const float4 dd4 = *reinterpret_cast<const float4 *>(&dd_s[r0]);
      const int4 pos4 = *reinterpret_cast<const int4 *>(&pos_s[r0]);
      bf16_t dsq[4];
      if (causal)
        bwd_p_ds<true>(s[mt], dp[mt], lse4, dd4, pos4, key, sl2, dsq);
      else
        bwd_p_ds<false>(s[mt], dp[mt], lse4, dd4, pos4, key, sl2, dsq);
      *reinterpret_cast<uint2 *>(&dSt[(wave * 16 + l16) * RP + r0]) = *reinterpret_cast<const uint2 *>(dsq);
    }
    // rows {4q..4q+3} and {16+4q..16+4q+3} (+32) as the K-operand of the row contractions
    const bf16x8 pb0 = pack_bf16x8(s[0], s[1]), pb1 = pack_bf16x8(s[2], s[3]);
    const bf16x8 sb0 = pack_bf16x8(dp[0], dp[1]), sb1 = pack_bf16x8(dp[2], dp[3]);
    // dV^T += dO^T P,  dK^T += Q^T dS   (feature tiles x this wave's keys)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      dvt[nt] = mfma16x16x32(lds_col8(dOs, KPQ, q4 * 4, 16 + q4 * 4, nt * 16, l16), pb0, dvt[nt]);
      dvt[nt] = mfma16x16x32(lds_col8(dOs, KPQ, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), pb1, dvt[nt]);
      dkt[nt] = mfma16x16x32(lds_col8(Qs, KPQ, q4 * 4, 16 + q4 * 4, nt * 16, l16), sb0, dkt[nt]);
      dkt[nt] = mfma16x16x32(lds_col8(Qs, KPQ, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), sb1, dkt[nt]);
    }
    __syncthreads();  // dSt complete

    // dQ^T = K^T dS^T for chunk rows 16w..16w+15 (all 64 keys)
    const int row = wave * 16 + l16;
    f32x4 dqt[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) dqt[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const bf16x8 bs = lds_col8(dSt, RP, kb * 32 + kq, kb * 32 + kq + 4, wave * 16, l16);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        dqt[nt] = mfma16x16x32(lds_col8(Ks, KPQ, kb * 32 + kq, kb * 32 + kq + 4, nt * 16, l16), bs, dqt[nt]);
    }
    // The wave's 16 dQ rows (chunk rows 16w..16w+15) are one contiguous run of
    // the list-ordered partial buffer: stage them in this wave's rows of Qs
    // (free after the dK product) and write full 16-byte lanes.
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16_t o4[4] = {f32_to_bf16(dqt[nt][0]), f32_to_bf16(dqt[nt][1]), f32_to_bf16(dqt[nt][2]),
                            f32_to_bf16(dqt[nt][3])};
      *reinterpret_cast<uint2 *>(&Qs[row * KPQ + nt * 16 + q4 * 4]) = *reinterpret_cast<const uint2 *>(o4);
    }
    wave_lds_sync();
    {
      const int64_t run0 = (list0 + c0) * G + wave * 16;  // first row of this wave
      const int nrows = min(CT, n_ent - c0) * G - wave * 16;                // valid rows of this wave
      // every lane stores (rows past the chunk's end go to the discard row), so the
      // number of stores per chunk is fixed and the waits for the prefetched rows
      // need not wait for them
      const int64_t discard = ix.discard;
#pragma unroll
      for (int k = 0; k < 16 * VPR / 64; ++k) {
        const int v = lane + 64 * k, r = v / VPR, cc = (v % VPR) * 8;
        const int64_t row = r < nrows ? run0 + r : discard;
        st_stream16(dqpart + row * D + cc, &Qs[(wave * 16 + r) * KPQ + cc]);
      }
    }
  }

  // this wave's keys: lane (q, j) holds features 16nt + 4q .. +3 of key 16w + j
  const int kk = wave * 16 + l16;
  if (whole_block) {
    const int64_t dst = (krow0 + (int64_t)kk * gm.Hkv) * D + q4 * 4;
    // the band's contribution to these keys (a band geometry), already scaled;
    // all of it is loaded before any is used, so the loads overlap
    f32x4 ak[NT], av[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) ak[nt] = av[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (bkv) {
      const float *bk = bkv + (int64_t)bgt * 2 * 64 * D + kk * D + q4 * 4;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        ak[nt] = *reinterpret_cast<const f32x4 *>(bk + nt * 16);
        av[nt] = *reinterpret_cast<const f32x4 *>(bk + 64 * D + nt * 16);
      }
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16_t k4[4] = {f32_to_bf16(dkt[nt][0] + ak[nt][0]), f32_to_bf16(dkt[nt][1] + ak[nt][1]),
                            f32_to_bf16(dkt[nt][2] + ak[nt][2]), f32_to_bf16(dkt[nt][3] + ak[nt][3])};
      const bf16_t v4[4] = {f32_to_bf16(fmaf(dvt[nt][0], inv_scale, av[nt][0])),
                            f32_to_bf16(fmaf(dvt[nt][1], inv_scale, av[nt][1])),
                            f32_to_bf16(fmaf(dvt[nt][2], inv_scale, av[nt][2])),
                            f32_to_bf16(fmaf(dvt[nt][3], inv_scale, av[nt][3]))};
      *reinterpret_cast<uint2 *>(dK + dst + nt * 16) = *reinterpret_cast<const uint2 *>(k4);
      *reinterpret_cast<uint2 *>(dV + dst + nt * 16) = *reinterpret_cast<const uint2 *>(v4);
    }
  } else {
    float *pk = dkvpart + (int64_t)u * 2 * 64 * D + kk * D + q4 * 4;
    float *pv = pk + 64 * D;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      *reinterpret_cast<float4 *>(pk + nt * 16) = make_float4(dkt[nt][0], dkt[nt][1], dkt[nt][2], dkt[nt][3]);
      *reinterpret_cast<float4 *>(pv + nt * 16) =
          make_float4(dvt[nt][0] * inv_scale, dvt[nt][1] * inv_scale, dvt[nt][2] * inv_scale, dvt[nt][3] * inv_scale);
    }
  }
}

// Per (b, g, t) of the index's compact list (blocks with zero or several work
// units): sum the float32 partials of its units, or zeros for a block nobody
// selected; a band geometry adds the band's float32 dK/dV of the tile (bkv).
// Each block's 2 x 64 x d outputs are split over kFinSplit workgroups; each
// thread owns 4 consecutive features (16-byte loads).  A fixed grid of
// kFinGrid x kFinSplit workgroups walks the list, kFinGrid blocks apart.
constexpr int kFinSplit = 16;
constexpr int kFinGrid = 512;
template <int D>
__global__ __launch_bounds__(256) void dkv_finalize_kernel(const float *__restrict__ dkvpart,
                                                           const float *__restrict__ bkv, bf16_t *__restrict__ dK,
                                                           bf16_t *__restrict__ dV, Geom gm, IndexWs ix) {
  constexpr int PER = 64 * D / kFinSplit;  // elements of dK (and of dV) per workgroup
  for (int j = blockIdx.x; j < ix.totals[2]; j += gridDim.x) {
    const int bgt = ix.fin[j];
    const int u0 = ix.uoff[bgt], u1 = ix.uoff[bgt + 1];
    const int bg = bgt / gm.T, t = bgt - bg * gm.T;
    const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
    for (int x = blockIdx.y * PER + threadIdx.x * 4; x < (int)(blockIdx.y + 1) * PER; x += 256 * 4) {
      const int kk = x / D, c = x - kk * D;
      float4 sk = make_float4(0.f, 0.f, 0.f, 0.f), sv = sk;
      if (bkv) {
        sk = *reinterpret_cast<const float4 *>(bkv + (int64_t)bgt * 2 * 64 * D + x);
        sv = *reinterpret_cast<const float4 *>(bkv + (int64_t)bgt * 2 * 64 * D + 64 * D + x);
      }
      for (int u = u0; u < u1; ++u) {
        const float4 a = *reinterpret_cast<const float4 *>(dkvpart + (int64_t)u * 2 * 64 * D + x);
        const float4 v = *reinterpret_cast<const float4 *>(dkvpart + (int64_t)u * 2 * 64 * D + 64 * D + x);
        sk.x += a.x; sk.y += a.y; sk.z += a.z; sk.w += a.w;
        sv.x += v.x; sv.y += v.y; sv.z += v.z; sv.w += v.w;
      }
      const int64_t dst = (((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g) * D + c;
      const bf16_t k4[4] = {f32_to_bf16(sk.x), f32_to_bf16(sk.y), f32_to_bf16(sk.z), f32_to_bf16(sk.w)};
      const bf16_t v4[4] = {f32_to_bf16(sv.x), f32_to_bf16(sv.y), f32_to_bf16(sv.z), f32_to_bf16(sv.w)};
      *reinterpret_cast<uint2 *>(dK + dst) = *reinterpret_cast<const uint2 *>(k4);
      *reinterpret_cast<uint2 *>(dV + dst) = *reinterpret_cast<const uint2 *>(v4);
    }
  }
}

// dQ = sum over a row's valid slots of the partials.  Half a wave per
// (b, g, query row), 8 features per lane (16-byte loads); the row's list
// positions come in one load (RowSlots), then up to 16 partials are loaded
// together and summed in slot order.
template <int D, int G>
__global__ __launch_bounds__(256) void dq_combine_kernel(const int32_t *__restrict__ pmap,
                                                         const bf16_t *__restrict__ dqpart, bf16_t *__restrict__ dQ,
                                                         Geom gm) {
  constexpr int U = 16;  // slots whose partials are in flight together
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int64_t x = ((int64_t)blockIdx.x * 4 + wave) * 2 + half;
  const bool row_ok = x < (int64_t)gm.B * gm.Hkv * gm.Lq;
  const int64_t xr = row_ok ? x : 0;
  const int bg = (int)(xr / gm.Lq), i = (int)(xr - (int64_t)bg * gm.Lq);
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const RowSlots rs(pmap, xr * gm.ksel, row_ok, gm.ksel, half, l32);
  const int ns = rs.slots();
  // Every lane runs the feature loop: the slot positions are shuffled from
  // lanes of the half-wave.  With G * D < 256 features, lanes past them only
  // take part in the shuffles.
  for (int e0 = 0; e0 < G * D; e0 += 256) {
    const int e = e0 + l32 * 8;
    const bool act = e < G * D;
    const int hh = act ? e / D : 0, c = act ? e - hh * D : 0;
    float a[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) a[k] = 0.f;
    for (int s0 = 0; s0 < ns; s0 += U) {
      uint4 raw[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int s = s0 + k;
        const int p = s < ns ? rs.pos(s, half) : -1;
        raw[k] = act && p >= 0 ? ld_stream16(dqpart + ((int64_t)p * G + hh) * D + c) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw[k]);
#pragma unroll
        for (int j = 0; j < 8; ++j) a[j] += bf16_to_f32(pv[j]);
      }
    }
    if (!row_ok || !act) continue;
    bf16_t outv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) outv[k] = f32_to_bf16(a[k]);
    *reinterpret_cast<uint4 *>(dQ + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + c) =
        *reinterpret_cast<const uint4 *>(outv);
  }
}

template <int D, int G>
static hipError_t launch_bwd_t(const Geom &g, const void *Q, const void *K, const void *V, const void *O,
                               const void *dO, const float *LSE, void *dQ, void *dK, void *dV, const IndexWs &ix,
                               float *Dvec, void *dqpart, float *dkvpart, float *bkv, hipStream_t s) {
  if (g.band) {  // the band's dK/dV tiles first: the sparse epilogue adds them
    const hipError_t e = launch_bwd_band_dkv(g, Q, K, V, dO, LSE, Dvec, ix, bkv, dkvpart, s);
    if (e != hipSuccess) return e;
  }
  const float *bk = g.band ? bkv : nullptr;
  timing_begin("phsa_attn_bwd_sparse", s);
  hipLaunchKernelGGL((attn_bwd_sparse_kernel<D, G>), dim3((unsigned)ix.units_max), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     static_cast<const bf16_t *>(dO), LSE, Dvec, g, ix, static_cast<bf16_t *>(dqpart),
                     static_cast<bf16_t *>(dK), static_cast<bf16_t *>(dV), dkvpart, bk);
  timing_end(s);
  timing_begin("phsa_attn_bwd_dkv_finalize", s);
  hipLaunchKernelGGL((dkv_finalize_kernel<D>), dim3(std::min(g.B * g.Hkv * g.T, kFinGrid), kFinSplit), dim3(256), 0, s,
                     dkvpart, bk,
                     static_cast<bf16_t *>(dK), static_cast<bf16_t *>(dV), g, ix);
  timing_end(s);
  if (g.band) {  // the band's dQ kernel merges every row's dQ itself
    const hipError_t e = launch_bwd_band_dq(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  const int64_t rows = (int64_t)g.B * g.Hkv * g.Lq;
  timing_begin("phsa_attn_bwd_dq_combine", s);
  hipLaunchKernelGGL((dq_combine_kernel<D, G>), dim3((unsigned)((rows + 7) / 8)), dim3(256), 0, s, ix.pmap,
                     static_cast<const bf16_t *>(dqpart), static_cast<bf16_t *>(dQ), g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_bwd_d(const Geom &g, const void *Q, const void *K, const void *V, const void *O,
                               const void *dO, const float *LSE, void *dQ, void *dK, void *dV, const IndexWs &ix,
                               float *Dvec, void *dqpart, float *dkvpart, float *bkv, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_bwd_t<D, 1>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s);
    case 2: return launch_bwd_t<D, 2>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s);
    case 4: return launch_bwd_t<D, 4>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s);
    default: return launch_bwd_t<D, 8>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s);
  }
}

template <typename T, int D>
static void launch_pre(const Geom &g, const void *O, const void *dO, float *Dvec, hipStream_t s) {
  const int64_t n = (int64_t)g.B * g.Lq * g.Hq * (D / (16 / sizeof(T)));  // threads
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
                           const void *dO, const float *LSE, const int32_t *sel, void *dQ,
                           void *dK, void *dV, const IndexWs &ix, float *Dvec, void *dqpart, float *dkvpart,
                           float *bkv, bool reuse_index, hipStream_t s) {
  hipError_t e = launch_bwd_pre(g, O, dO, Dvec, s);
  if (e != hipSuccess) return e;
  if (!reuse_index) {
    e = launch_build_index(g, sel, ix, s);
    if (e != hipSuccess) return e;
  }
  return g.d == 128 ? launch_bwd_d<128>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s)
                    : launch_bwd_d<64>(g, Q, K, V, O, dO, LSE, dQ, dK, dV, ix, Dvec, dqpart, dkvpart, bkv, s);
}

}  // namespace phsa

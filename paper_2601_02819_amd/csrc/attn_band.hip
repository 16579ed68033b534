// The forced blocks as dense attention (the "band"), bf16.
//
// Algorithm 1 always keeps the init blocks 0 .. n_init - 1 and the local
// window, blocks max(0, cur - w/m) .. cur, of every query row: the keys
// [0, n_init m) up to the row and [A(i), pos(i)] with
//   A(i) = max(cur - w/m, min(n_init, cur + 1)) * m
// (w = 0: the row's own block).  Every row shares the init keys and
// neighbouring rows share most of their windows.  In the key-block-major
// sparse kernels each (row, forced tile) pair would gather the row and leave
// a partial; here the forced keys are attended densely instead:
//   forward, dQ : query-major.  A workgroup holds 128 (forward) or 64 (dQ)
//                 (token, head) MFMA rows of consecutive tokens in registers
//                 and streams the 64-key tiles of their forced keys (the init
//                 tiles, then the window tiles) through LDS, each copied from
//                 global memory straight into LDS while the previous one is
//                 used, with an online softmax (forward) or the dQ
//                 accumulation (backward).  Both run after their sparse
//                 kernel and merge their rows themselves: a row's sparse
//                 partials in slot order, then its band result, whose slot
//                 (list position band_base + row) follows the row's sparse
//                 entries; that is the order of the per-row merge kernels
//                 used without a band, so the results are the same bits.
//   dK, dV      : key-major.  A workgroup holds one 64-key tile (wave w owns
//                 keys 16w..16w+15: their K and V fragments and the dK, dV
//                 accumulators in registers) and streams the contiguous rows
//                 whose forced keys reach into it, each 64-row chunk of Q and
//                 dO copied straight into LDS while the previous one is used; it writes
//                 the tile's float32 dK/dV to bkv, which the sparse backward's
//                 epilogue and the dK/dV finalize add to the sparse part.  An
//                 init tile is reached by every later row: its rows are split
//                 into segments, one workgroup each, whose float32 sums a
//                 reduction adds up into bkv in segment order.
// Only rows that hold all their forced blocks (bflag, set by the index) take
// part; other rows keep every block in the sparse kernels.  Operand layouts
// and the transposing LDS reads are those of the sparse kernels (attn_fwd.hip,
// attn_bwd.hip).
#include <math.h>

#include <algorithm>

#include "common.h"
#include "launch.h"

namespace phsa {

// First key of the band of the query at position pos (selection blocks of gm.sm tokens).
__device__ __forceinline__ int band_first_key(const Geom &gm, int pos) {
  const int cur = pos / gm.sm;
  return max(max(0, cur - gm.window / gm.sm), min(gm.n_init, cur + 1)) * gm.sm;
}

// Keys of the init blocks: a band row attends to [0, init_end) up to itself
// and to its local window [A(i), pos(i)] (A(i) >= init_end once the row is
// past the init blocks).
__device__ __forceinline__ int init_end_key(const Geom &gm) { return gm.n_init * gm.sm; }
__device__ __forceinline__ bool forced_key(int key, int pos, int a, int init_end) {
  return key <= pos && (key < init_end || key >= a);
}

// The 64-key tiles a query-major workgroup visits: the init tiles it reaches,
// then the window tiles past them.  Tile j of ntile is tile_of(j).
struct TileSeq {
  int nit, kt_b, ntile;
  __device__ __forceinline__ TileSeq(int kt_lo, int kt_hi, int init_end) {
    nit = min((init_end + 63) / 64, kt_hi + 1);
    kt_b = max(kt_lo, nit);
    ntile = nit + max(0, kt_hi - kt_b + 1);
  }
  __device__ __forceinline__ int tile_of(int j) const { return j < nit ? j : kt_b + (j - nit); }
};

// ---------------------------------------------------------------- forward
template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_fwd_band_kernel(const bf16_t *__restrict__ Q,
                                                               const bf16_t *__restrict__ K,
                                                               const bf16_t *__restrict__ V, Geom gm, IndexWs ix,
                                                               const bf16_t *__restrict__ opart,
                                                               const float2 *__restrict__ ml, bf16_t *__restrict__ O,
                                                               float *__restrict__ LSE) {
  constexpr int RT = 2;                  // 16-row chunks per wave
  constexpr int TOK = 4 * RT * 16 / G;   // tokens per workgroup
  constexpr int SP = D + 8;
  constexpr int VPR = D / 8, KB = D / 32, NT = D / 16;
  constexpr int TILE = 64 * D;           // one K or V tile (swizzled rows, no padding)
  static_assert(4 * 16 * SP <= 2 * TILE, "output staging fits a tile buffer");
  // two buffers of a K tile and a V tile: tile kt is read from one while tile
  // kt + 1 is copied into the other; two distinct arrays, so that the
  // compiler can tell the copies into one from the reads of the other.  The
  // output staging of the epilogue reuses KV0.
  __shared__ __attribute__((aligned(16))) bf16_t KV0[2 * TILE];
  __shared__ __attribute__((aligned(16))) bf16_t KV1[2 * TILE];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  // query tiles of one XCD are consecutive (they share most key tiles)
  const int item = xcd_item(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int qt = item % gridDim.x, bg = item / gridDim.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int i0 = qt * TOK, i1 = min(i0 + TOK, gm.Lq) - 1;
  const uint8_t *bf = ix.bflag + (int64_t)bg * gm.Lq;

  // the rows of this lane: chunk c, MFMA row (wave RT + c) 16 + l16
  int pos[RT], a0[RT];
  bool ok[RT];
  bf16x8 qf[RT][KB];
#pragma unroll
  for (int c = 0; c < RT; ++c) {
    const int r = (wave * RT + c) * 16 + l16;
    const int tok = i0 + r / G, h = r % G;
    const int ti = min(tok, i1);
    ok[c] = tok <= i1 && bf[ti] != 0;
    pos[c] = gm.q_pos0 + ti;
    a0[c] = band_first_key(gm, pos[c]);
    const bf16_t *src = Q + (((int64_t)b * gm.Lq + ti) * gm.Hq + g * G + h) * D;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) qf[c][kb] = load_bf16x8(src + kb * 32 + kq);
  }
  // a workgroup without band rows attends to no tile, but still merges its rows
  const bool any_band = __syncthreads_or(ok[0] || ok[RT - 1]);
  const int kt_lo = band_first_key(gm, gm.q_pos0 + i0) / 64, kt_hi = (gm.q_pos0 + i1) / 64;
  const int a_last = band_first_key(gm, gm.q_pos0 + i1), pos_first = gm.q_pos0 + i0;
  const int init_end = init_end_key(gm);
  TileSeq seq(kt_lo, kt_hi, init_end);
  if (!any_band) seq.ntile = 0;

  const float sl2 = gm.scale * kLog2e;
  // the row sums l accumulate on the matrix cores: an all-ones A operand
  // against the same P^T fragments as O, so l sums the bf16 weights that O sums
  float mrun[RT];
  f32x4 o[RT][NT], lacc[RT];
  const bf16x8 ones = __builtin_bit_cast(bf16x8, v8i16{0x3f80, 0x3f80, 0x3f80, 0x3f80, 0x3f80, 0x3f80, 0x3f80, 0x3f80});
#pragma unroll
  for (int c = 0; c < RT; ++c) {
    mrun[c] = -INFINITY;
    lacc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) o[c][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // Tile kt + 1 is copied into the other buffer while tile kt is used (issued
  // before the use, a whole tile ahead); one barrier per tile then publishes
  // it and ends every wave's reads of tile kt.
  const int64_t head0 = (int64_t)b * gm.Lk * gm.Hkv * D + (int64_t)g * D;
  const int kstride = gm.Hkv * D;  // elements between consecutive keys of a head
  auto key_row = [kstride](int r) { return r * kstride; };
  auto issue = [&](int kt, bf16_t *buf) {
    const int64_t t0 = head0 + (int64_t)kt * 64 * kstride;
    tile_dma<D>(K + t0, key_row, buf, wave, lane);
    tile_dma<D>(V + t0, key_row, buf + TILE, wave, lane);
  };
  auto step = [&](int j, const bf16_t *Ks, bf16_t *nxt) {
    if (j + 1 < seq.ntile) issue(seq.tile_of(j + 1), nxt);
    const bf16_t *Vs = Ks + TILE;
    const int key0 = seq.tile_of(j) * 64;
    // S^T = K Q^T for both chunks (every K fragment read from LDS feeds both)
    f32x4 sa[RT][4];
#pragma unroll
    for (int c = 0; c < RT; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) sa[c][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bf16x8 kfr = load_bf16x8(&Ks[swz<D>(j * 16 + l16, kb * 32 + kq)]);
#pragma unroll
        for (int c = 0; c < RT; ++c) sa[c][j] = mfma16x16x32(kfr, qf[c][kb], sa[c][j]);
      }
    // Tiles inside every row's forced keys (all but the first and last one or
    // two) need no mask: rows outside the band compute values that are discarded.
    const bool interior = key0 + 63 <= pos_first && (key0 + 63 < init_end || key0 >= a_last);
    bf16x8 pb[RT][2];
    float fs[RT];
#pragma unroll
    for (int c = 0; c < RT; ++c) {
      f32x4 (&st)[4] = sa[c];
      if (!interior) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = key0 + j * 16 + q4 * 4 + r;
            st[j][r] = (ok[c] && forced_key(key, pos[c], a0[c], init_end)) ? st[j][r] : -INFINITY;
          }
      }
      // IEEE maximum (v_maximum3_f32): no quieting pass over the accumulators
      // first; the scores are finite or -inf
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        mx = __builtin_elementwise_maximum(__builtin_elementwise_maximum(mx, st[j][0]),
                                           __builtin_elementwise_maximum(st[j][1], __builtin_elementwise_maximum(st[j][2], st[j][3])));
      mx = max_xor32(max_xor16(mx));
      mx *= sl2;
      // The reference maximum moves only when some row's maximum rises by more
      // than 2^8 (or is first set): weights stay below 2^8, far inside bf16
      // and float32, and most tiles skip the rescaling of O and l.
      float f = 1.f;
      if (__any(mx > mrun[c] + 8.f)) {
        const float mn = fmaxf(mrun[c], mx);
        f = mn == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(mrun[c] - mn);  // 0 when the row had no key yet
        mrun[c] = mn;
      }
      const float mref = mrun[c] == -INFINITY ? 0.f : mrun[c];  // no key of the row yet: every weight is 0
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) st[j][r] = __builtin_amdgcn_exp2f(fmaf(st[j][r], sl2, -mref));
      fs[c] = f;
      pb[c][0] = pack_bf16x8(st[0], st[1]);
      pb[c][1] = pack_bf16x8(st[2], st[3]);
    }
    // O^T = O^T f (a uniform branch, rarely taken) ...
    if (__any(fs[0] != 1.f || fs[RT - 1] != 1.f)) {
#pragma unroll
      for (int c = 0; c < RT; ++c) {
        lacc[c] *= fs[c];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) o[c][nt] *= fs[c];
      }
    }
    // ... + V^T P^T for both chunks (every V^T fragment feeds both)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16x8 v0 = lds_col8_sw<D>(Vs, q4 * 4, 16 + q4 * 4, nt * 16, l16);
      const bf16x8 v1 = lds_col8_sw<D>(Vs, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16);
#pragma unroll
      for (int c = 0; c < RT; ++c) {
        o[c][nt] = mfma16x16x32(v0, pb[c][0], o[c][nt]);
        o[c][nt] = mfma16x16x32(v1, pb[c][1], o[c][nt]);
      }
    }
#pragma unroll
    for (int c = 0; c < RT; ++c) {
      lacc[c] = mfma16x16x32(ones, pb[c][0], lacc[c]);
      lacc[c] = mfma16x16x32(ones, pb[c][1], lacc[c]);
    }
    dma_wait();
    lds_barrier();
  };
  if (seq.ntile > 0) issue(seq.tile_of(0), KV0);
  dma_wait();
  lds_barrier();
  for (int j = 0; j < seq.ntile; j += 2) {
    step(j, KV0, KV1);
    if (j + 1 < seq.ntile) step(j + 1, KV1, KV0);
  }

  // The merge of the workgroup's rows (Eq. 10-11 across the row's partials),
  // fused here: the sparse kernel's partials of a row are folded in slot
  // order, then this kernel's band partial, whose slot follows them (the order
  // of the per-row merge kernel).  Every wave has passed the loop's last
  // barrier, so the tile buffers hold the band results: rows 0..63 in KV0,
  // 64..127 in KV1, each as a bf16 row of O, then (m, l) and the band flag.
  auto orow = [&](int r) -> bf16_t * { return (r < 64 ? KV0 : KV1) + (r & 63) * SP; };
  auto mls = [&](int r) -> float2 * { return reinterpret_cast<float2 *>((r < 64 ? KV0 : KV1) + 64 * SP) + (r & 63); };
  auto oks = [&](int r) -> int * {
    return reinterpret_cast<int *>(reinterpret_cast<float2 *>((r < 64 ? KV0 : KV1) + 64 * SP) + 64) + (r & 63);
  };
  static_assert(64 * SP * sizeof(bf16_t) + 64 * (sizeof(float2) + sizeof(int)) <= 2 * TILE * sizeof(bf16_t),
                "band results fit a tile buffer");
#pragma unroll
  for (int c = 0; c < RT; ++c) {
    const int r = (wave * RT + c) * 16 + l16;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16_t o4[4] = {f32_to_bf16(o[c][nt][0]), f32_to_bf16(o[c][nt][1]), f32_to_bf16(o[c][nt][2]),
                            f32_to_bf16(o[c][nt][3])};
      *reinterpret_cast<uint2 *>(orow(r) + nt * 16 + q4 * 4) = *reinterpret_cast<const uint2 *>(o4);
    }
    if (q4 == 0) {
      *mls(r) = make_float2(mrun[c], lacc[c][0]);
      *oks(r) = ok[c] ? 1 : 0;
    }
  }
  __syncthreads();
  // half a wave per token (its G heads), 8 features per lane, as in the merge
  // kernel; each half-wave merges NP tokens at a time (t, t + 8, ...), so that
  // their partials are in flight together (this kernel holds only 8 waves per
  // CU: eight tokens with two slots each in flight took the merge of the
  // paper's geometry from 2.67 to 2.45 ms, one token with sixteen slots was
  // the slowest)
  constexpr int U = 2;                           // slots per token whose partials are in flight together
  constexpr int NP = TOK >= 64 ? 8 : TOK / 8;  // tokens per half-wave at a time
  static_assert(TOK % (8 * NP) == 0, "token groups");
  const int half = lane >> 5, l32 = lane & 31;
  // a token's list positions are loaded while the previous tokens' partials are
  auto load_pos = [&](int t, int &pa, int &pb) {
    const int i = i0 + t;
    const bool row_ok = i <= i1;
    const int64_t base = ((int64_t)bg * gm.Lq + (row_ok ? i : i0)) * gm.ksel;
    pa = (row_ok && l32 < gm.ksel) ? ix.pmap[base + l32] : -1;
    pb = (row_ok && l32 + 32 < gm.ksel) ? ix.pmap[base + l32 + 32] : -1;
  };
  int pa[NP], pb[NP];
#pragma unroll
  for (int u = 0; u < NP; ++u) load_pos(wave * 2 + half + 8 * u, pa[u], pb[u]);
  for (int t0 = 0; t0 < TOK; t0 += 8 * NP) {
    RowSlots rs[NP];
    int ns = 0;
#pragma unroll
    for (int u = 0; u < NP; ++u) {
      rs[u] = RowSlots(pa[u], pb[u], half);
      ns = max(ns, rs[u].slots());
    }
    if (t0 + 8 * NP < TOK) {
#pragma unroll
      for (int u = 0; u < NP; ++u) load_pos(t0 + 8 * NP + wave * 2 + half + 8 * u, pa[u], pb[u]);
    }
    // every lane runs the feature loop: the slot positions are shuffled from
    // lanes of the half-wave; with G * D < 256 features, lanes past them only
    // take part in the shuffles
    for (int e0 = 0; e0 < G * D; e0 += 256) {
      const int e = e0 + l32 * 8;
      const bool act = e < G * D;
      const int hh = act ? e / D : 0, cc = act ? e - hh * D : 0;
      float M[NP], L[NP], a[NP][8];
#pragma unroll
      for (int u = 0; u < NP; ++u) {
        M[u] = -INFINITY;
        L[u] = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) a[u][k] = 0.f;
      }
      for (int s0 = 0; s0 < ns; s0 += U) {
        float2 q[NP][U];
        uint4 raw[NP][U];
#pragma unroll
        for (int k = 0; k < U; ++k)
#pragma unroll
          for (int u = 0; u < NP; ++u) {
            const int s = s0 + k;
            const int p = s < ns ? rs[u].pos(s, half) : -1;
            const bool sp = act && p >= 0 && p < ix.band_base;  // a sparse partial (not the band slot)
            q[u][k] = sp ? ml[(int64_t)p * G + hh] : make_float2(-INFINITY, 0.f);
            raw[u][k] = sp ? ld_stream16(opart + ((int64_t)p * G + hh) * D + cc) : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
        for (int k = 0; k < U; ++k)
#pragma unroll
          for (int u = 0; u < NP; ++u) fold_partial(M[u], L[u], a[u], q[u][k], raw[u][k]);
      }
#pragma unroll
      for (int u = 0; u < NP; ++u) {
        const int t = t0 + wave * 2 + half + 8 * u, i = i0 + t;
        const bool row_ok = i <= i1;
        const int r = t * G + hh;
        if (!row_ok || !act) continue;
        if (*oks(r)) fold_partial(M[u], L[u], a[u], *mls(r), *reinterpret_cast<const uint4 *>(orow(r) + cc));
        const float inv = L[u] > 0.f ? 1.f / L[u] : 0.f;
        bf16_t outv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) outv[k] = f32_to_bf16(a[u][k] * inv);
        *reinterpret_cast<uint4 *>(O + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + cc) =
            *reinterpret_cast<const uint4 *>(outv);
        if (cc == 0)
          LSE[((int64_t)b * gm.Hq + g * G + hh) * gm.Lq + i] = L[u] > 0.f ? (M[u] + log2f(L[u])) * kLn2 : -INFINITY;
      }
    }
  }
}

// ---------------------------------------------------------------- backward: dQ
template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_bwd_band_dq_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ V,
    const bf16_t *__restrict__ dO, const float *__restrict__ LSE, const float *__restrict__ Dvec, Geom gm,
    IndexWs ix, const bf16_t *__restrict__ dqpart, bf16_t *__restrict__ dQ) {
  constexpr int RT = 1;                  // one 16-row chunk per wave (registers)
  constexpr int TOK = 4 * RT * 16 / G;
  constexpr int SP = D + 8;
  constexpr int VPR = D / 8, KB = D / 32, NT = D / 16;
  constexpr int TILE = 64 * D;           // one K or V tile (swizzled rows, no padding)
  static_assert(4 * 16 * SP <= 2 * TILE, "output staging fits a tile buffer");
  // the tile buffers of the forward kernel: tile kt + 1 is copied from global
  // memory straight into one while tile kt is read from the other
  __shared__ __attribute__((aligned(16))) bf16_t KV0[2 * TILE];
  __shared__ __attribute__((aligned(16))) bf16_t KV1[2 * TILE];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  // query tiles of one XCD are consecutive (they share most key tiles)
  const int item = xcd_item(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int qt = item % gridDim.x, bg = item / gridDim.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int i0 = qt * TOK, i1 = min(i0 + TOK, gm.Lq) - 1;
  const uint8_t *bf = ix.bflag + (int64_t)bg * gm.Lq;

  int pos[RT], a0[RT];
  bool ok[RT];
  float lse2[RT], dd[RT];
  bf16x8 qf[RT][KB], df[RT][KB];
#pragma unroll
  for (int c = 0; c < RT; ++c) {
    const int r = (wave * RT + c) * 16 + l16;
    const int tok = i0 + r / G, h = g * G + r % G;
    const int ti = min(tok, i1);
    ok[c] = tok <= i1 && bf[ti] != 0;
    pos[c] = gm.q_pos0 + ti;
    a0[c] = band_first_key(gm, pos[c]);
    lse2[c] = LSE[((int64_t)b * gm.Hq + h) * gm.Lq + ti] * kLog2e;
    dd[c] = Dvec[((int64_t)b * gm.Lq + ti) * gm.Hq + h];
    const int64_t src = (((int64_t)b * gm.Lq + ti) * gm.Hq + h) * D;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      qf[c][kb] = load_bf16x8(Q + src + kb * 32 + kq);
      df[c][kb] = load_bf16x8(dO + src + kb * 32 + kq);
    }
  }
  // a workgroup without band rows attends to no tile, but still merges its rows
  const bool any_band = __syncthreads_or(ok[0]);
  const int kt_lo = band_first_key(gm, gm.q_pos0 + i0) / 64, kt_hi = (gm.q_pos0 + i1) / 64;
  const int a_last = band_first_key(gm, gm.q_pos0 + i1), pos_first = gm.q_pos0 + i0;
  const int init_end = init_end_key(gm);
  TileSeq seq(kt_lo, kt_hi, init_end);
  if (!any_band) seq.ntile = 0;

  const float sl2 = gm.scale * kLog2e;
  f32x4 dq[RT][NT];
#pragma unroll
  for (int c = 0; c < RT; ++c)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) dq[c][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int64_t head0 = (int64_t)b * gm.Lk * gm.Hkv * D + (int64_t)g * D;
  const int kstride = gm.Hkv * D;  // elements between consecutive keys of a head
  auto key_row = [kstride](int r) { return r * kstride; };
  auto issue = [&](int kt, bf16_t *buf) {
    const int64_t t0 = head0 + (int64_t)kt * 64 * kstride;
    tile_dma<D>(K + t0, key_row, buf, wave, lane);
    tile_dma<D>(V + t0, key_row, buf + TILE, wave, lane);
  };
  auto step = [&](int jt, const bf16_t *Ks, bf16_t *nxt) {
    if (jt + 1 < seq.ntile) issue(seq.tile_of(jt + 1), nxt);
    const bf16_t *Vs = Ks + TILE;
    const int key0 = seq.tile_of(jt) * 64;
    const bool interior = key0 + 63 <= pos_first && (key0 + 63 < init_end || key0 >= a_last);
#pragma unroll
    for (int c = 0; c < RT; ++c) {
      // S^T = K Q^T and dP^T = V dO^T: lane (q, j) holds keys 16 jt + 4 q + r of row j
      f32x4 st[4], dp[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) st[j] = dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          st[j] = mfma16x16x32(load_bf16x8(&Ks[swz<D>(j * 16 + l16, kb * 32 + kq)]), qf[c][kb], st[j]);
          dp[j] = mfma16x16x32(load_bf16x8(&Vs[swz<D>(j * 16 + l16, kb * 32 + kq)]), df[c][kb], dp[j]);
        }
      // interior tiles (inside every row's band) need no mask: rows outside
      // the band compute values that are discarded.  A masked score is -inf
      // and its weight 2^-inf = 0.
      if (!interior) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = key0 + j * 16 + q4 * 4 + r;
            st[j][r] = (ok[c] && forced_key(key, pos[c], a0[c], init_end)) ? st[j][r] : -INFINITY;
          }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(st[j][r], sl2, -lse2[c]));
          dp[j][r] = p * (dp[j][r] - dd[c]);
        }
      // dQ^T += K^T dS^T
      const bf16x8 sb0 = pack_bf16x8(dp[0], dp[1]), sb1 = pack_bf16x8(dp[2], dp[3]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        dq[c][nt] = mfma16x16x32(lds_col8_sw<D>(Ks, q4 * 4, 16 + q4 * 4, nt * 16, l16), sb0, dq[c][nt]);
        dq[c][nt] = mfma16x16x32(lds_col8_sw<D>(Ks, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), sb1, dq[c][nt]);
      }
    }
    dma_wait();
    lds_barrier();
  };
  if (seq.ntile > 0) issue(seq.tile_of(0), KV0);
  dma_wait();
  lds_barrier();
  for (int jt = 0; jt < seq.ntile; jt += 2) {
    step(jt, KV0, KV1);
    if (jt + 1 < seq.ntile) step(jt + 1, KV1, KV0);
  }

  // The dQ merge of the workgroup's rows, fused here: the sparse kernel's dQ
  // partials of a row are summed in slot order, then this kernel's band dQ
  // (rounded to bf16 like a partial), whose slot follows them: the order of
  // the per-row merge kernel.  Every wave has passed the loop's last barrier,
  // so KV0 holds the band results: a bf16 row of dQ per MFMA row, then the
  // band flags.
  int *oks = reinterpret_cast<int *>(KV0 + 64 * SP);
  static_assert(64 * SP * sizeof(bf16_t) + 64 * sizeof(int) <= 2 * TILE * sizeof(bf16_t), "band dQ fits a tile buffer");
#pragma unroll
  for (int c = 0; c < RT; ++c) {
    const int r = (wave * RT + c) * 16 + l16;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16_t o4[4] = {f32_to_bf16(dq[c][nt][0] * gm.scale), f32_to_bf16(dq[c][nt][1] * gm.scale),
                            f32_to_bf16(dq[c][nt][2] * gm.scale), f32_to_bf16(dq[c][nt][3] * gm.scale)};
      *reinterpret_cast<uint2 *>(&KV0[r * SP + nt * 16 + q4 * 4]) = *reinterpret_cast<const uint2 *>(o4);
    }
    if (q4 == 0) oks[r] = ok[c] ? 1 : 0;
  }
  __syncthreads();
  // half a wave per token (its G heads), 8 features per lane, all of the
  // half-wave's tokens at once (t, t + 8, ...), two slots of each in flight
  constexpr int U = 2;
  constexpr int NP = TOK / 8;
  static_assert(TOK % 8 == 0 && NP >= 1, "tokens per half-wave");
  const int half = lane >> 5, l32 = lane & 31;
  RowSlots rs[NP];
  int ns = 0;
#pragma unroll
  for (int u = 0; u < NP; ++u) {
    const int i = i0 + wave * 2 + half + 8 * u;
    const bool row_ok = i <= i1;
    rs[u] = RowSlots(ix.pmap, ((int64_t)bg * gm.Lq + (row_ok ? i : i0)) * gm.ksel, row_ok, gm.ksel, half, l32);
    ns = max(ns, rs[u].slots());
  }
  // every lane runs the feature loop (the slot positions are shuffled from
  // lanes of the half-wave); with G * D < 256, lanes past the features only shuffle
  for (int e0 = 0; e0 < G * D; e0 += 256) {
    const int e = e0 + l32 * 8;
    const bool act = e < G * D;
    const int hh = act ? e / D : 0, cc = act ? e - hh * D : 0;
    float a[NP][8];
#pragma unroll
    for (int u = 0; u < NP; ++u)
#pragma unroll
      for (int k = 0; k < 8; ++k) a[u][k] = 0.f;
    for (int s0 = 0; s0 < ns; s0 += U) {
      uint4 raw[NP][U];
#pragma unroll
      for (int k = 0; k < U; ++k)
#pragma unroll
        for (int u = 0; u < NP; ++u) {
          const int s = s0 + k;
          const int p = s < ns ? rs[u].pos(s, half) : -1;
          raw[u][k] = (act && p >= 0 && p < ix.band_base) ? ld_stream16(dqpart + ((int64_t)p * G + hh) * D + cc)
                                                           : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
      for (int k = 0; k < U; ++k)
#pragma unroll
        for (int u = 0; u < NP; ++u) {
          const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw[u][k]);
#pragma unroll
          for (int j = 0; j < 8; ++j) a[u][j] += bf16_to_f32(pv[j]);
        }
    }
#pragma unroll
    for (int u = 0; u < NP; ++u) {
      const int t = wave * 2 + half + 8 * u, i = i0 + t;
      if (i > i1 || !act) continue;
      const int r = t * G + hh;
      if (oks[r]) {
        const bf16_t *pv = &KV0[r * SP + cc];
#pragma unroll
        for (int j = 0; j < 8; ++j) a[u][j] += bf16_to_f32(pv[j]);
      }
      bf16_t outv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) outv[k] = f32_to_bf16(a[u][k]);
      *reinterpret_cast<uint4 *>(dQ + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + cc) =
          *reinterpret_cast<const uint4 *>(outv);
    }
  }
}

// ---------------------------------------------------------------- backward: dK, dV
// One workgroup per (b, g, 64-key tile kt, row segment).  The rows whose
// forced keys reach into the tile are tokens kt 64 - q_pos0 .. (the last token
// with A(i) <= kt 64 + 63), or every later token for an init tile; they stream
// through in chunks of 64 MFMA rows (64 / G tokens, heads inner).  Work item x
// of a (b, g) is tile kt0 + x / nseg, segment x % nseg (tokens seg_tok seg ..
// seg_tok (seg + 1) - 1); the tile's float32 dK, dV go to slot
// ((b, g) out_tiles + kt) nseg + seg of out.
template <int D, int G>
__global__ __launch_bounds__(256, 2) void attn_bwd_band_dkv_kernel(
    const bf16_t *__restrict__ Q, const bf16_t *__restrict__ K, const bf16_t *__restrict__ V,
    const bf16_t *__restrict__ dO, const float *__restrict__ LSE, const float *__restrict__ Dvec, Geom gm, IndexWs ix,
    int kt0, int nseg, int seg_tok, int out_tiles, float *__restrict__ out) {
  constexpr int CT = 64 / G;             // tokens per chunk
  constexpr int KB = D / 32, NT = D / 16;
  constexpr int TILE = 64 * D;           // one chunk's Q or dO rows (swizzled, no padding)
  // two buffers of a chunk's Q and dO rows: chunk c + 1 is copied from global
  // memory straight into one while chunk c is read from the other (two
  // distinct arrays, so that the compiler can tell the copies from the reads)
  __shared__ __attribute__((aligned(16))) bf16_t QD0[2 * TILE];
  __shared__ __attribute__((aligned(16))) bf16_t QD1[2 * TILE];
  // per buffer, the chunk's rows: LSE (log2 units; +inf outside the band), D,
  // position (-1 outside the band) and band start
  __shared__ __attribute__((aligned(16))) float lse_s[2][64];
  __shared__ __attribute__((aligned(16))) float dd_s[2][64];
  __shared__ __attribute__((aligned(16))) int pos_s[2][64];
  __shared__ __attribute__((aligned(16))) int a_s[2][64];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  // key tiles of one XCD are consecutive (they share most rows)
  const int item = xcd_item(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  const int xi = item % gridDim.x, bg = item / gridDim.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int kt = kt0 + xi / nseg, seg = xi % nseg;
  const uint8_t *bf = ix.bflag + (int64_t)bg * gm.Lq;
  const int key0 = kt * 64;
  const int init_end = init_end_key(gm);
  // rows: from the first token that sees key0 to the last whose window starts
  // by key0 + 63 (every later token, for a tile holding init keys), within the
  // segment
  int r_lo = max(0, key0 - gm.q_pos0);
  int r_hi = gm.Lq - 1;
  if (key0 >= init_end) {
    const int cmax = (key0 + 63) / gm.sm + gm.window / gm.sm;
    r_hi = min(r_hi, (cmax + 1) * gm.sm - 1 - gm.q_pos0);
  }
  r_lo = max(r_lo, seg * seg_tok);
  r_hi = min(r_hi, seg * seg_tok + seg_tok - 1);

  // the wave's keys 16w..16w+15 of K and V as B operands, in registers for the whole tile
  bf16x8 kf[KB], vf[KB];
  {
    const int64_t src = (((int64_t)b * gm.Lk + key0 + wave * 16 + l16) * gm.Hkv + g) * D + kq;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      kf[kb] = load_bf16x8(K + src + kb * 32);
      vf[kb] = load_bf16x8(V + src + kb * 32);
    }
  }
  f32x4 dkt[NT], dvt[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) dkt[n] = dvt[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const float sl2 = gm.scale * kLog2e;
  const int key = key0 + wave * 16 + l16;  // the key whose S column this lane holds
  // Chunk c0's rows are tokens c0 + r / G, heads r % G (tokens past r_hi repeat
  // the last one and are masked).  Q and dO rows of a token's G heads are one
  // contiguous run.
  const int64_t head0 = ((int64_t)b * gm.Lq * gm.Hq + g * G) * D;
  auto issue = [&](int c0, bf16_t *buf) {
    auto row_off = [&](int r) { return ((int64_t)min(c0 + r / G, r_hi) * gm.Hq + r % G) * D; };
    tile_dma<D>(Q + head0, row_off, buf, wave, lane);
    tile_dma<D>(dO + head0, row_off, buf + TILE, wave, lane);
  };
  // thread r < 64 loads row r's LSE, D, band flag of a chunk into registers;
  // they reach LDS after the chunk before it has been computed
  float plse = 0.f, pdd = 0.f;
  int ptok = 0, pflag = 0;
  auto load_row = [&](int c0) {
    if (tid < 64) {
      const int tok = c0 + tid / G, h = g * G + tid % G;
      const int ti = min(tok, r_hi);
      plse = LSE[((int64_t)b * gm.Hq + h) * gm.Lq + ti];
      pdd = Dvec[((int64_t)b * gm.Lq + ti) * gm.Hq + h];
      pflag = bf[ti];
      ptok = tok;
    }
  };
  auto store_row = [&](int sb) {
    if (tid < 64) {
      const int ti = min(ptok, r_hi);
      const bool in_band = ptok <= r_hi && pflag != 0;
      lse_s[sb][tid] = in_band ? plse * kLog2e : INFINITY;  // rows outside the band: weight 2^-inf = 0
      dd_s[sb][tid] = pdd;
      pos_s[sb][tid] = in_band ? gm.q_pos0 + ti : -1;
      a_s[sb][tid] = band_first_key(gm, gm.q_pos0 + ti);
    }
  };

  auto step = [&](int c0, const bf16_t *Qs, bf16_t *nxt, int sb) {
    const bool more = c0 + CT <= r_hi;
    if (more) {
      issue(c0 + CT, nxt);
      load_row(c0 + CT);
    }
    const bf16_t *dOs = Qs + TILE;
    // the chunk's tokens ascend, and so do their positions and band starts:
    // when the first token sees the wave's last key and the last token's
    // window starts by its first key (or the keys are init keys), every key of
    // the wave is forced for every row of the chunk
    const int wk0 = key0 + wave * 16;
    const int pos_first = gm.q_pos0 + c0, a_last = band_first_key(gm, gm.q_pos0 + min(c0 + CT - 1, r_hi));
    const bool interior = wk0 + 15 <= pos_first && (wk0 + 15 < init_end || wk0 >= a_last);

    // S and dP: 64 rows (4 tiles) x this wave's 16 keys; lane (q, j) holds rows 16 mt + 4 q + r of key j
    f32x4 s[4], dp[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) s[mt] = dp[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        s[mt] = mfma16x16x32(load_bf16x8(&Qs[swz<D>(mt * 16 + l16, kb * 32 + kq)]), kf[kb], s[mt]);
        dp[mt] = mfma16x16x32(load_bf16x8(&dOs[swz<D>(mt * 16 + l16, kb * 32 + kq)]), vf[kb], dp[mt]);
      }
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int r0 = mt * 16 + q4 * 4;
      const float4 lse4 = *reinterpret_cast<const float4 *>(&lse_s[sb][r0]);
      const float4 dd4 = *reinterpret_cast<const float4 *>(&dd_s[sb][r0]);
      const float lsev[4] = {lse4.x, lse4.y, lse4.z, lse4.w};
      const float ddv[4] = {dd4.x, dd4.y, dd4.z, dd4.w};
      if (interior) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[mt][r], sl2, -lsev[r]));
          s[mt][r] = p;
          dp[mt][r] = p * (dp[mt][r] - ddv[r]);
        }
      } else {
        const int4 pos4 = *reinterpret_cast<const int4 *>(&pos_s[sb][r0]);
        const int4 a4 = *reinterpret_cast<const int4 *>(&a_s[sb][r0]);
        const int posv[4] = {pos4.x, pos4.y, pos4.z, pos4.w};
        const int av[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool in = forced_key(key, posv[r], av[r], init_end);
          const float p = __builtin_amdgcn_exp2f(in ? fmaf(s[mt][r], sl2, -lsev[r]) : -INFINITY);
          s[mt][r] = p;
          dp[mt][r] = p * (dp[mt][r] - ddv[r]);
        }
      }
    }
    const bf16x8 pb0 = pack_bf16x8(s[0], s[1]), pb1 = pack_bf16x8(s[2], s[3]);
    const bf16x8 sb0 = pack_bf16x8(dp[0], dp[1]), sb1 = pack_bf16x8(dp[2], dp[3]);
    // dV^T += dO^T P,  dK^T += Q^T dS   (feature tiles x this wave's keys)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      dvt[nt] = mfma16x16x32(lds_col8_sw<D>(dOs, q4 * 4, 16 + q4 * 4, nt * 16, l16), pb0, dvt[nt]);
      dvt[nt] = mfma16x16x32(lds_col8_sw<D>(dOs, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), pb1, dvt[nt]);
      dkt[nt] = mfma16x16x32(lds_col8_sw<D>(Qs, q4 * 4, 16 + q4 * 4, nt * 16, l16), sb0, dkt[nt]);
      dkt[nt] = mfma16x16x32(lds_col8_sw<D>(Qs, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), sb1, dkt[nt]);
    }
    if (more) store_row(sb ^ 1);  // the other buffer's rows were last read before the previous barrier
    dma_wait();
    lds_barrier();
  };
  if (r_lo <= r_hi) {
    issue(r_lo, QD0);
    load_row(r_lo);
    store_row(0);
  }
  dma_wait();
  lds_barrier();
  for (int c0 = r_lo; c0 <= r_hi; c0 += 2 * CT) {
    step(c0, QD0, QD1, 0);
    if (c0 + CT <= r_hi) step(c0 + CT, QD1, QD0, 1);
  }
  // the tile's dK (scaled) and dV: lane (q, j) holds features 16 nt + 4 q .. +3 of key 16 w + j
  float *pk = out + (((int64_t)bg * out_tiles + kt) * nseg + seg) * 2 * 64 * D + (wave * 16 + l16) * D + q4 * 4;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    *reinterpret_cast<float4 *>(pk + nt * 16) =
        make_float4(dkt[nt][0] * gm.scale, dkt[nt][1] * gm.scale, dkt[nt][2] * gm.scale, dkt[nt][3] * gm.scale);
    *reinterpret_cast<float4 *>(pk + 64 * D + nt * 16) = make_float4(dvt[nt][0], dvt[nt][1], dvt[nt][2], dvt[nt][3]);
  }
}

// Sums the row segments of each init tile (in segment order) into bkv:
// workgroup (tile of a (b, g), part) adds 1024 consecutive floats of the
// tile's 2 x 64 x d.
template <int D>
__global__ __launch_bounds__(256) void band_init_reduce_kernel(const float *__restrict__ seg_sums, float *__restrict__ bkv,
                                                                Geom gm, int nit, int nseg) {
  constexpr int PER = 2 * 64 * D;
  const int bgk = blockIdx.x, bg = bgk / nit, kt = bgk - bg * nit;
  const int x = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (x >= PER) return;
  const float *src = seg_sums + (int64_t)bgk * nseg * PER + x;
  float4 acc = *reinterpret_cast<const float4 *>(src);
  for (int sg = 1; sg < nseg; ++sg) {
    const float4 v = *reinterpret_cast<const float4 *>(src + (int64_t)sg * PER);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  *reinterpret_cast<float4 *>(bkv + ((int64_t)bg * gm.T + kt) * PER + x) = acc;
}

// ---------------------------------------------------------------- launchers
template <int D, int G>
static hipError_t fwd_band_t(const Geom &g, const void *Q, const void *K, const void *V, const IndexWs &ix,
                             const void *opart, const float2 *ml, void *O, float *LSE, hipStream_t s) {
  constexpr int TOK = 128 / G;
  timing_begin("phsa_attn_fwd_band", s);
  hipLaunchKernelGGL((attn_fwd_band_kernel<D, G>), dim3((g.Lq + TOK - 1) / TOK, g.B * g.Hkv), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     g, ix, static_cast<const bf16_t *>(opart), ml, static_cast<bf16_t *>(O), LSE);
  timing_end(s);
  return hipGetLastError();
}

// Init tiles that every row reaches are split into segments of about
// kInitSegTokens tokens, at most T / nit per tile so that their float32 sums
// fit in the sparse backward's dK/dV partial buffer, which they borrow.
constexpr int kInitSegTokens = 1024;

int band_init_tiles(const Geom &g) { return std::min((g.n_init * g.sm + 63) / 64, g.T); }

int band_init_segments(const Geom &g) {
  const int nit = band_init_tiles(g);
  if (nit == 0) return 0;
  return std::max(1, std::min((g.Lq + kInitSegTokens - 1) / kInitSegTokens, g.T / nit));
}

template <int D, int G>
static hipError_t bwd_band_dkv_t(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                                 const float *LSE, const float *Dvec, const IndexWs &ix, float *bkv, float *seg_sums,
                                 hipStream_t s) {
  const bf16_t *q = static_cast<const bf16_t *>(Q), *k = static_cast<const bf16_t *>(K);
  const bf16_t *v = static_cast<const bf16_t *>(V), *dout = static_cast<const bf16_t *>(dO);
  const int nit = band_init_tiles(g), R = g.B * g.Hkv;
  if (nit > 0) {
    const int nseg = band_init_segments(g), seg_tok = (g.Lq + nseg - 1) / nseg;
    timing_begin("phsa_attn_bwd_band_dkv_init", s);
    hipLaunchKernelGGL((attn_bwd_band_dkv_kernel<D, G>), dim3(nit * nseg, R), dim3(256), 0, s, q, k, v, dout, LSE,
                       Dvec, g, ix, 0, nseg, seg_tok, nit, seg_sums);
    timing_end(s);
    timing_begin("phsa_attn_bwd_band_init_reduce", s);
    hipLaunchKernelGGL((band_init_reduce_kernel<D>), dim3(R * nit, (2 * 64 * D + 1023) / 1024), dim3(256), 0, s,
                       static_cast<const float *>(seg_sums), bkv, g, nit, nseg);
    timing_end(s);
  }
  if (g.T > nit) {
    timing_begin("phsa_attn_bwd_band_dkv", s);
    hipLaunchKernelGGL((attn_bwd_band_dkv_kernel<D, G>), dim3(g.T - nit, R), dim3(256), 0, s, q, k, v, dout, LSE, Dvec,
                       g, ix, nit, 1, g.Lq, g.T, bkv);
    timing_end(s);
  }
  return hipGetLastError();
}

template <int D, int G>
static hipError_t bwd_band_dq_t(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                                const float *LSE, const float *Dvec, const IndexWs &ix, const void *dqpart, void *dQ,
                                hipStream_t s) {
  constexpr int TOKQ = 64 / G;
  timing_begin("phsa_attn_bwd_band_dq", s);
  hipLaunchKernelGGL((attn_bwd_band_dq_kernel<D, G>), dim3((g.Lq + TOKQ - 1) / TOKQ, g.B * g.Hkv), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     static_cast<const bf16_t *>(dO), LSE, Dvec, g, ix, static_cast<const bf16_t *>(dqpart),
                     static_cast<bf16_t *>(dQ));
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t fwd_band_d(const Geom &g, const void *Q, const void *K, const void *V, const IndexWs &ix,
                             const void *opart, const float2 *ml, void *O, float *LSE, hipStream_t s) {
  switch (g.G) {
    case 1: return fwd_band_t<D, 1>(g, Q, K, V, ix, opart, ml, O, LSE, s);
    case 2: return fwd_band_t<D, 2>(g, Q, K, V, ix, opart, ml, O, LSE, s);
    case 4: return fwd_band_t<D, 4>(g, Q, K, V, ix, opart, ml, O, LSE, s);
    default: return fwd_band_t<D, 8>(g, Q, K, V, ix, opart, ml, O, LSE, s);
  }
}

template <int D>
static hipError_t bwd_band_dkv_d(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                                 const float *LSE, const float *Dvec, const IndexWs &ix, float *bkv, float *seg_sums,
                                 hipStream_t s) {
  switch (g.G) {
    case 1: return bwd_band_dkv_t<D, 1>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s);
    case 2: return bwd_band_dkv_t<D, 2>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s);
    case 4: return bwd_band_dkv_t<D, 4>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s);
    default: return bwd_band_dkv_t<D, 8>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s);
  }
}

template <int D>
static hipError_t bwd_band_dq_d(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                                const float *LSE, const float *Dvec, const IndexWs &ix, const void *dqpart, void *dQ,
                                hipStream_t s) {
  switch (g.G) {
    case 1: return bwd_band_dq_t<D, 1>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
    case 2: return bwd_band_dq_t<D, 2>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
    case 4: return bwd_band_dq_t<D, 4>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
    default: return bwd_band_dq_t<D, 8>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
  }
}

hipError_t launch_fwd_band(const Geom &g, const void *Q, const void *K, const void *V, const IndexWs &ix,
                           const void *opart, const float2 *ml, void *O, float *LSE, hipStream_t s) {
  return g.d == 128 ? fwd_band_d<128>(g, Q, K, V, ix, opart, ml, O, LSE, s)
                    : fwd_band_d<64>(g, Q, K, V, ix, opart, ml, O, LSE, s);
}

hipError_t launch_bwd_band_dkv(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                               const float *LSE, const float *Dvec, const IndexWs &ix, float *bkv, float *seg_sums,
                               hipStream_t s) {
  return g.d == 128 ? bwd_band_dkv_d<128>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s)
                    : bwd_band_dkv_d<64>(g, Q, K, V, dO, LSE, Dvec, ix, bkv, seg_sums, s);
}

hipError_t launch_bwd_band_dq(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                              const float *LSE, const float *Dvec, const IndexWs &ix, const void *dqpart, void *dQ,
                              hipStream_t s) {
  return g.d == 128 ? bwd_band_dq_d<128>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s)
                    : bwd_band_dq_d<64>(g, Q, K, V, dO, LSE, Dvec, ix, dqpart, dQ, s);
}

}  // namespace phsa

// Relevance scoring + block selection (Eq. 8 logits; Algorithm 1 block
// selection with forced init / local blocks, causal block mask, top-k and
// Unique).
//
// float32 inputs (select_kernel): one workgroup per (64-query tile, b*Hkv + g).  Lane r of every wave owns
// query row i0 + r; the group's query heads are summed once into a float32
// register vector (sum_h q_h . M = (sum_h q_h) . M), so a block costs one
// d-long dot product per row.  Representative keys stream through LDS in
// chunks of 64 blocks; wave w scores blocks 16w..16w+15 of each chunk with
// broadcast LDS reads and keeps a sorted register list of its best KMAX
// (score, block) pairs.  The four per-wave lists are merged in LDS, the
// winners are put in ascending block order together with the forced blocks,
// and the row is written out padded with -1.
//
// Order: score descending, then block index ascending (a strict total order,
// so every row has one answer).
#include <float.h>

#include <type_traits>

#include "common.h"
#include "launch.h"

// Selection workgroups for k <= 16: 4 waves (128 rows) with one (hi, lo)
// chunk buffer take 80 KB of LDS, so two workgroups share a CU and one's
// VALU-heavy phases (bar, final rank) overlap the other's MFMA chunks.  (One
// 8-wave workgroup per CU with double-buffered chunks, 160 KB, keeps all its
// waves in the same phase: 0.78 -> 0.70 ms at 4 x 32k, 1.78 -> 1.59 ms at
// T = 2048 with 16-token blocks.)
#ifndef PHSA_SEL_NW
#define PHSA_SEL_NW 4      // waves per selection workgroup (k <= 16)
#endif
#ifndef PHSA_SEL_DB
#define PHSA_SEL_DB false  // double-buffered pass 2 (k <= 16)
#endif
#ifndef PHSA_SEL_SLACK
#define PHSA_SEL_SLACK 112 // list capacity beyond 4 k entries
#endif
#ifndef PHSA_SEL_CH
#define PHSA_SEL_CH 64     // blocks per staged chunk (a multiple of 16)
#endif

namespace phsa {

// Maximum over the 16 lanes of a row, every lane getting it: DPP moves inside
// the row (lane ^ 1, lane ^ 2, then the mirrored half row and row), no LDS.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float a) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp_move<0xB1>(v));   // quad_perm [1, 0, 3, 2]
  v = fmaxf(v, dpp_move<0x4E>(v));   // quad_perm [2, 3, 0, 1]
  v = fmaxf(v, dpp_move<0x141>(v));  // row_half_mirror
  return fmaxf(v, dpp_move<0x140>(v));  // row_mirror
}

__device__ __forceinline__ bool beats(float s1, int t1, float s2, int t2) {
  return s1 > s2 || (s1 == s2 && t1 < t2);
}

// The query tile and (b, g) of a workgroup of a (query tiles, B * Hkv) grid,
// longest first: a tile's causal blocks grow with its index, so the last tiles
// are dispatched first and the short ones fill in behind them.
struct TileOrder {
  int tile, bg;
  __device__ __forceinline__ TileOrder() {
    const int lin = blockIdx.x + blockIdx.y * gridDim.x;
    bg = lin % gridDim.y;
    tile = gridDim.x - 1 - lin / gridDim.y;
  }
};

// Writes one row of sel: the forced init blocks, the npick picks (sorted here
// into ascending order, in place) and the local blocks, padded with -1.
__device__ __forceinline__ void emit_row(int32_t *__restrict__ out, int *pk, int npick, int cur, const Geom &gm) {
  for (int a = 1; a < npick; ++a) {  // insertion sort, at most top_k items
    const int x = pk[a];
    int c = a - 1;
    while (c >= 0 && pk[c] > x) {
      pk[c + 1] = pk[c];
      --c;
    }
    pk[c + 1] = x;
  }
  const int lo = max(0, cur - gm.window / gm.m);
  const int ni = min(gm.n_init, cur + 1);
  int n = 0;
  for (int t = 0; t < ni; ++t) out[n++] = t;
  for (int a = 0; a < npick; ++a) out[n++] = pk[a];
  for (int t = max(lo, ni); t <= cur; ++t) out[n++] = t;
  for (; n < gm.ksel; ++n) out[n] = -1;
}

// Merge the four waves' sorted (score, block) lists of each row through LDS,
// take the k best (score descending, block ascending) and write the row:
// forced init blocks, the picks and the local blocks in ascending order,
// padded with -1.  Every thread of the workgroup calls this (it holds a
// barrier); lanes with `active` set write their row.  smem must hold the four
// lists (4 * 64 * KMAX (score, block) pairs).
template <int KMAX>
__device__ __forceinline__ void finish_rows(const float (&ls)[KMAX], const int (&lt)[KMAX], unsigned char *smem,
                                            int (*picks)[KMAX], bool active, int i, int cur, int bg,
                                            int32_t *__restrict__ sel, const Geom &gm) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __syncthreads();
  float *list_s = reinterpret_cast<float *>(smem);
  int *list_t = reinterpret_cast<int *>(smem) + 4 * 64 * KMAX;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    list_s[(wave * 64 + lane) * KMAX + k] = ls[k];
    list_t[(wave * 64 + lane) * KMAX + k] = lt[k];
  }
  __syncthreads();
  if (!active) return;
  int head[4] = {0, 0, 0, 0};
  int npick = 0;
  for (int p = 0; p < gm.top_k && p < KMAX; ++p) {
    int bw = -1;
    float bs = -FLT_MAX;
    int bt = 0x7fffffff;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      if (head[w] < KMAX) {
        const float s = list_s[(w * 64 + lane) * KMAX + head[w]];
        const int t = list_t[(w * 64 + lane) * KMAX + head[w]];
        if (t != 0x7fffffff && beats(s, t, bs, bt)) {
          bw = w;
          bs = s;
          bt = t;
        }
      }
    }
    if (bw < 0) break;
#pragma unroll
    for (int w = 0; w < 4; ++w) head[w] += (w == bw);
    picks[lane][npick++] = bt;
  }
  emit_row(sel + ((int64_t)bg * gm.Lq + i) * gm.ksel, picks[lane], npick, cur, gm);
}

template <typename T, int D, int KMAX>
__global__ __launch_bounds__(256) void select_kernel(const T *__restrict__ Q, const float *__restrict__ Kc,
                                                     int32_t *__restrict__ sel, Geom gm) {
  constexpr int CH = 64;                               // blocks per LDS chunk
  constexpr int LIST_BYTES = 4 * 64 * KMAX * 8;        // four wave lists
  constexpr int CHUNK_BYTES = CH * D * 4;
  constexpr int BUF = LIST_BYTES > CHUNK_BYTES ? LIST_BYTES : CHUNK_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[BUF];
  __shared__ int picks[64][KMAX];
  float *kc_s = reinterpret_cast<float *>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const TileOrder wo;
  const int bg = wo.bg, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int i = wo.tile * 64 + lane;
  const bool row_ok = i < gm.Lq;
  const int pos = gm.q_pos0 + (row_ok ? i : gm.Lq - 1);
  const int cur = pos / gm.m;
  const int lo = max(0, cur - gm.window / gm.m);       // first local block
  // candidate blocks of this row: n_init <= t < lo
  const int last_i = min(wo.tile * 64 + 63, gm.Lq - 1);
  const int t_end = max(0, (gm.q_pos0 + last_i) / gm.m - gm.window / gm.m);  // max lo over the tile

  float q[D];
#pragma unroll
  for (int c = 0; c < D; ++c) q[c] = 0.f;
  if (row_ok) {
    for (int hh = 0; hh < gm.G; ++hh) {
      const T *src = Q + (((int64_t)b * gm.Lq + i) * gm.Hq + g * gm.G + hh) * D;
#pragma unroll
      for (int c = 0; c < D; c += 16 / sizeof(T)) {
        const uint4 raw = *reinterpret_cast<const uint4 *>(src + c);
        const T *v = reinterpret_cast<const T *>(&raw);
#pragma unroll
        for (int e = 0; e < 16 / (int)sizeof(T); ++e) q[c + e] += to_f32<T>(v[e]);
      }
    }
  }

  float ls[KMAX];
  int lt[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    ls[k] = -FLT_MAX;
    lt[k] = 0x7fffffff;
  }

  const float *kc_bg = Kc + (int64_t)bg * gm.T * D;
  if (gm.top_k > 0) {
    for (int t0 = gm.n_init; t0 < t_end; t0 += CH) {
      const int nblk = min(CH, gm.T - t0);
      __syncthreads();
      for (int e = tid * 4; e < nblk * D; e += 256 * 4)
        *reinterpret_cast<float4 *>(kc_s + e) = *reinterpret_cast<const float4 *>(kc_bg + (int64_t)t0 * D + e);
      __syncthreads();
      for (int tt = wave * 16; tt < wave * 16 + 16; ++tt) {
        const int t = t0 + tt;
        if (t >= t_end) break;
        const float *kr = kc_s + tt * D;
        float acc0 = 0.f, acc1 = 0.f, acc2 = 0.f, acc3 = 0.f;
#pragma unroll
        for (int c = 0; c < D; c += 4) {
          const float4 kv = *reinterpret_cast<const float4 *>(kr + c);
          acc0 = fmaf(q[c], kv.x, acc0);
          acc1 = fmaf(q[c + 1], kv.y, acc1);
          acc2 = fmaf(q[c + 2], kv.z, acc2);
          acc3 = fmaf(q[c + 3], kv.w, acc3);
        }
        float s = ((acc0 + acc1) + (acc2 + acc3)) * gm.scale;
        int ct = t;
        if (row_ok && t < lo && beats(s, ct, ls[KMAX - 1], lt[KMAX - 1])) {
#pragma unroll
          for (int k = 0; k < KMAX; ++k) {
            const bool bt = beats(s, ct, ls[k], lt[k]);
            const float os = ls[k];
            const int ot = lt[k];
            ls[k] = bt ? s : os;
            lt[k] = bt ? ct : ot;
            s = bt ? os : s;
            ct = bt ? ot : ct;
          }
        }
      }
    }
  }

  finish_rows<KMAX>(ls, lt, smem, picks, wave == 0 && row_ok, i, cur, bg, sel, gm);
}

// Softmax-sum selection (PHSA_FLAG_SELECT_SOFTMAX_SUM): Eq. 8's softmax is
// taken per query head over the complete blocks 0..cur-1 of the row's causal
// past, and a block's group score is the sum of its G head probabilities,
// ranked as s = log2 sum_h 2^(x_h - lse_h) with x_h the head's logit in log2
// units and lse_h the head's log2 normaliser.
//
// A lane owns one (query row, head) pair: 64 / G rows per workgroup, lane l
// holding row l / G and head l % G, whose query (scaled by scale * log2 e)
// stays in registers.  Representatives stream through LDS in chunks of 64
// blocks as in select_kernel, wave w scoring blocks 16w..16w+15 of a chunk.
//   pass 1: every lane keeps a running (max, sum) of 2^x over t < cur; the
//           four waves' states are merged through LDS into lse_h.
//   pass 2: the candidate blocks are scored again, the G lanes of a row
//           combine their terms by shuffles (shifted by their maximum, so no
//           term underflows), and every lane inserts the row's score into
//           its sorted list (the G lanes of a row hold identical lists).
// Costs two d-long dot products per (row, head, block), 2G times those of the
// summed-logit kernel.
template <typename T, int D, int KMAX>
__global__ __launch_bounds__(256) void select_softmax_kernel(const T *__restrict__ Q, const float *__restrict__ Kc,
                                                             int32_t *__restrict__ sel, Geom gm) {
  constexpr int CH = 64;
  constexpr int LIST_BYTES = 4 * 64 * KMAX * 8;
  constexpr int CHUNK_BYTES = CH * D * 4;
  constexpr int BUF = LIST_BYTES > CHUNK_BYTES ? LIST_BYTES : CHUNK_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[BUF];
  __shared__ int picks[64][KMAX];
  __shared__ float wmax[4][64], wsum[4][64];
  float *kc_s = reinterpret_cast<float *>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = gm.G, R = 64 / G;                      // rows per workgroup
  const TileOrder wo;
  const int bg = wo.bg, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int hh = lane % G;
  const int i = wo.tile * R + lane / G;
  const bool row_ok = i < gm.Lq;
  const int pos = gm.q_pos0 + (row_ok ? i : gm.Lq - 1);
  const int cur = pos / gm.m;
  const int lo = max(0, cur - gm.window / gm.m);
  const int last_i = min(wo.tile * R + R - 1, gm.Lq - 1);
  const int cur_max = (gm.q_pos0 + last_i) / gm.m;     // normaliser blocks: t < cur
  const int t_end = max(0, cur_max - gm.window / gm.m);  // candidates: n_init <= t < lo

  float q[D];
  {
    const float f = gm.scale * kLog2e;
    const T *src = Q + (((int64_t)b * gm.Lq + (row_ok ? i : gm.Lq - 1)) * gm.Hq + g * G + hh) * D;
#pragma unroll
    for (int c = 0; c < D; c += 16 / sizeof(T)) {
      const uint4 raw = *reinterpret_cast<const uint4 *>(src + c);
      const T *v = reinterpret_cast<const T *>(&raw);
#pragma unroll
      for (int e = 0; e < 16 / (int)sizeof(T); ++e) q[c + e] = to_f32<T>(v[e]) * f;
    }
  }
  const float *kc_bg = Kc + (int64_t)bg * gm.T * D;
  auto load_chunk = [&](int t0, int nblk) {
    __syncthreads();
    for (int e = tid * 4; e < nblk * D; e += 256 * 4)
      *reinterpret_cast<float4 *>(kc_s + e) = *reinterpret_cast<const float4 *>(kc_bg + (int64_t)t0 * D + e);
    __syncthreads();
  };
  auto dot = [&](int tt) {
    const float *kr = kc_s + tt * D;
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int c = 0; c < D; c += 4) {
      const float4 kv = *reinterpret_cast<const float4 *>(kr + c);
      a0 = fmaf(q[c], kv.x, a0);
      a1 = fmaf(q[c + 1], kv.y, a1);
      a2 = fmaf(q[c + 2], kv.z, a2);
      a3 = fmaf(q[c + 3], kv.w, a3);
    }
    return (a0 + a1) + (a2 + a3);
  };

  float ls[KMAX];
  int lt[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    ls[k] = -FLT_MAX;
    lt[k] = 0x7fffffff;
  }

  if (gm.top_k > 0 && t_end > gm.n_init) {
    // pass 1: per-head log2 normaliser over blocks 0..cur-1
    float mx = -INFINITY, sm = 0.f;
    for (int t0 = 0; t0 < cur_max; t0 += CH) {
      load_chunk(t0, min(CH, gm.T - t0));
      for (int tt = wave * 16; tt < wave * 16 + 16; ++tt) {
        const int t = t0 + tt;
        if (t >= cur_max) break;
        const float x = dot(tt);
        if (t < cur) {
          if (x > mx) {
            sm = sm * exp2f(mx - x) + 1.f;
            mx = x;
          } else {
            sm += exp2f(x - mx);
          }
        }
      }
    }
    wmax[wave][lane] = mx;
    wsum[wave][lane] = sm;
    __syncthreads();
    float gmx = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) gmx = fmaxf(gmx, wmax[w][lane]);
    float gsum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      if (wsum[w][lane] > 0.f) gsum += wsum[w][lane] * exp2f(wmax[w][lane] - gmx);
    const float lse = gsum > 0.f ? gmx + log2f(gsum) : 0.f;  // rows with cur = 0 have no candidates

    // pass 2: group scores of the candidates and the running top-k
    for (int t0 = gm.n_init; t0 < t_end; t0 += CH) {
      load_chunk(t0, min(CH, gm.T - t0));
      for (int tt = wave * 16; tt < wave * 16 + 16; ++tt) {
        const int t = t0 + tt;
        if (t >= t_end) break;
        const float y = dot(tt) - lse;
        float ymax = y;
        for (int o = 1; o < G; o <<= 1) ymax = fmaxf(ymax, __shfl_xor(ymax, o, 64));
        float e = exp2f(y - ymax);
        for (int o = 1; o < G; o <<= 1) e += __shfl_xor(e, o, 64);
        float sc = ymax + log2f(e);
        int ct = t;
        if (row_ok && t < lo && beats(sc, ct, ls[KMAX - 1], lt[KMAX - 1])) {
#pragma unroll
          for (int k = 0; k < KMAX; ++k) {
            const bool bt = beats(sc, ct, ls[k], lt[k]);
            const float os = ls[k];
            const int ot = lt[k];
            ls[k] = bt ? sc : os;
            lt[k] = bt ? ct : ot;
            sc = bt ? os : sc;
            ct = bt ? ot : ct;
          }
        }
      }
    }
  }
  finish_rows<KMAX>(ls, lt, smem, picks, wave == 0 && row_ok && hh == 0, i, cur, bg, sel, gm);
}

// Softmax-sum selection on the matrix cores (bf16 inputs; mode of
// select_softmax_kernel).  A workgroup holds 64 (query token, head) pairs,
// 64 / G tokens with their heads inner; wave w owns pairs 16w..16w+15 as one
// 16-row MFMA tile.  A pair's query is scaled to log2 units and split into
// bf16 hi + lo like the representatives (select_split_kernel), and the three
// chains hi.hi + hi.lo + lo.hi give its logits to about 2^-17 relative.  In
// the accumulator layout lane (q4, l16) holds pairs 4 q4 + r of its tile for
// blocks t0 + 16 nt + l16: the G heads of a token sit in the same lane (G <= 4)
// or in lanes q4 and q4 ^ 1 (G = 8), so a token's group score
// log2 sum_h 2^(x_h - lse_h) is formed without LDS, and the 16 lanes of a
// quarter-wave see all blocks of their tokens, each a fixed residue mod 16.
//   pass 1: the complete causal blocks t < cur: a running (max, sum) of 2^x per
//           lane and pair, merged over the 16 lanes: the log2 normaliser lse.
//   pass 2: the candidates' group scores; each lane keeps the best two of its
//           stripe per token.  A token's 32 stripe tops are 32 distinct
//           blocks, so the largest v with at least k of them >= v (the bar)
//           lies at or below the token's k-th best score.
//   pass 3: the group scores again; those >= bar are appended to the token's
//           LDS list (slots from an LDS counter: about k + 3 per token on
//           random inputs).  A list that could overflow with the next chunk
//           (many equal scores) is cut to its k best first.
//   final:  the k best of each list (score descending, block ascending) by
//           counting ranks, so the order of arrival does not matter.
// Scores of passes 2 and 3 come from identical instruction sequences on the
// same data, so they are bitwise equal and the bar never drops a winner.
template <int D, int G, int KMAX>
__global__ __launch_bounds__(256) void select_softmax_mfma_kernel(const bf16_t *__restrict__ Q,
                                                                  const bf16_t *__restrict__ Mh_g,
                                                                  const bf16_t *__restrict__ Ml_g,
                                                                  int32_t *__restrict__ sel, Geom gm) {
  constexpr int CH = 64;
  constexpr int NTOK = 64 / G;            // tokens per workgroup
  constexpr int GL = G < 4 ? G : 4;       // heads of a token within one lane
  constexpr int TPL = 4 / GL;             // tokens per lane (lanes q4 even only when G = 8)
  constexpr int LPT = 256 / NTOK;         // threads per token when ranking
  constexpr int CAP = KMAX + CH;          // list slots per token: k best + one chunk
  constexpr int MP = D + 16;              // 16-byte fragment reads of 16 rows are conflict-free
  constexpr int KB = D / 32;
  constexpr int NL = CH * D / (256 * 8);
  constexpr int BUF = 2 * CH * MP * 2;
  __shared__ __attribute__((aligned(16))) unsigned char smem[BUF];
  __shared__ float2 cand[NTOK][CAP];      // (score, block as int bits), unordered
  __shared__ int ccnt[NTOK];
  __shared__ int picks[NTOK][KMAX];
  __shared__ float bar_s[NTOK];
  bf16_t *Mh = reinterpret_cast<bf16_t *>(smem);
  bf16_t *Ml = Mh + CH * MP;
  float *tops = reinterpret_cast<float *>(smem);   // bar and cuts: [NTOK][32] / [NTOK][2 KMAX]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  const TileOrder wo;
  const int bg = wo.bg, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int i0 = wo.tile * NTOK;
  const int last_i = min(i0 + NTOK - 1, gm.Lq - 1);
  const int cur_max = (gm.q_pos0 + last_i) / gm.m;
  const int t_end = max(0, cur_max - gm.window / gm.m);
  const int k = gm.top_k;

  // A operand: pair 16 w + l16 (token (16 w + l16) / G, head l16 % G)
  bf16x8 ah[KB], al[KB];
  {
    const float f = gm.scale * kLog2e;
    const int p = wave * 16 + l16;
    const int i = min(i0 + p / G, gm.Lq - 1);
    const bf16_t *src = Q + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + p % G) * D;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const uint4 raw = *reinterpret_cast<const uint4 *>(src + kb * 32 + kq);
      const bf16_t *v = reinterpret_cast<const bf16_t *>(&raw);
      bf16_t hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = bf16_to_f32(v[e]) * f;
        hi[e] = f32_to_bf16(x);
        lo[e] = f32_to_bf16(x - bf16_to_f32(hi[e]));
      }
      ah[kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(hi));
      al[kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(lo));
    }
  }
  // accumulator row r of this lane: pair 16 w + 4 q4 + r; its token and bounds
  const int tok0 = (wave * 16 + q4 * 4) / G;   // first token of this lane's rows
  int cur_r[4], lo_t[TPL];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + (wave * 16 + q4 * 4 + r) / G;
    cur_r[r] = i < gm.Lq ? (gm.q_pos0 + i) / gm.m : 0;
  }
#pragma unroll
  for (int u = 0; u < TPL; ++u) {
    const int i = i0 + tok0 + u;
    lo_t[u] = i < gm.Lq ? max(0, (gm.q_pos0 + i) / gm.m - gm.window / gm.m) : 0;
  }

  const bf16_t *mh_bg = Mh_g + (int64_t)bg * gm.T * D;
  const bf16_t *ml_bg = Ml_g + (int64_t)bg * gm.T * D;
  uint4 ph[NL], pl[NL];
  auto fetch = [&](int t0) {
    const int nblk = min(CH, gm.T - t0);
#pragma unroll
    for (int x = 0; x < NL; ++x) {
      const int e = (tid + 256 * x) * 8, row = e / D, c = e % D;
      const int64_t off = (int64_t)(t0 + row) * D + c;
      ph[x] = row < nblk ? *reinterpret_cast<const uint4 *>(mh_bg + off) : make_uint4(0u, 0u, 0u, 0u);
      pl[x] = row < nblk ? *reinterpret_cast<const uint4 *>(ml_bg + off) : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int x = 0; x < NL; ++x) {
      const int e = (tid + 256 * x) * 8, row = e / D, c = e % D;
      *reinterpret_cast<uint4 *>(&Mh[row * MP + c]) = ph[x];
      *reinterpret_cast<uint4 *>(&Ml[row * MP + c]) = pl[x];
    }
  };
  // exact logits of the staged chunk: acc[nt][r] = x(pair 16 w + 4 q4 + r, block t0 + 16 nt + l16)
  auto scores = [&](f32x4 (&acc)[4]) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      bf16x8 bh[4], bl[4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        bh[nt] = load_bf16x8(&Mh[(nt * 16 + l16) * MP + kb * 32 + kq]);
        bl[nt] = load_bf16x8(&Ml[(nt * 16 + l16) * MP + kb * 32 + kq]);
      }
      // each chain over the 4 accumulators in turn (consecutive MFMAs independent;
      // every accumulator still takes hi.hi, hi.lo, lo.hi of each kb in that order)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma16x16x32(ah[kb], bh[nt], acc[nt]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma16x16x32(ah[kb], bl[nt], acc[nt]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[nt] = mfma16x16x32(al[kb], bh[nt], acc[nt]);
    }
  };
  // one pass over the chunks of [ta, tb): body(t0, acc) after the scores
  auto sweep = [&](int ta, int tb, auto body) {
    fetch(ta);
    for (int t0 = ta; t0 < tb; t0 += CH) {
      __syncthreads();
      stage();
      __syncthreads();
      if (t0 + CH < tb) fetch(t0 + CH);
      f32x4 acc[4];
      scores(acc);
      body(t0, acc);
    }
  };
  float lse[4];
  // group score of token u of this lane for block t0 + 16 nt + l16 (all lanes call this)
  auto group = [&](const f32x4 &a, int u) {
    float m = a[u * GL] - lse[u * GL];
#pragma unroll
    for (int r = 1; r < GL; ++r) m = fmaxf(m, a[u * GL + r] - lse[u * GL + r]);
    if (G == 8) m = fmaxf(m, __shfl_xor(m, 16, 64));
    float e = 0.f;
#pragma unroll
    for (int r = 0; r < GL; ++r) e += __builtin_amdgcn_exp2f(a[u * GL + r] - lse[u * GL + r] - m);
    if (G == 8) e += __shfl_xor(e, 16, 64);
    return m + __builtin_amdgcn_logf(e);   // e in [1, G]
  };
  const bool lane_tok = G < 8 || (q4 & 1) == 0;   // lanes that hold whole tokens

  if (tid < NTOK) ccnt[tid] = 0;
  if (k > 0 && t_end > gm.n_init) {
    // ---- pass 1: log2 normaliser of every pair over blocks 0 .. cur - 1
    float mx[4], sm[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      mx[r] = -INFINITY;
      sm[r] = 0.f;
    }
    sweep(0, cur_max, [&](int t0, f32x4 (&acc)[4]) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float cm = -INFINITY;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          if (t0 + nt * 16 + l16 < cur_r[r]) cm = fmaxf(cm, acc[nt][r]);
        const float nm = fmaxf(mx[r], cm);
        if (nm == -INFINITY) continue;
        float add = 0.f;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          if (t0 + nt * 16 + l16 < cur_r[r]) add += __builtin_amdgcn_exp2f(acc[nt][r] - nm);
        sm[r] = sm[r] * __builtin_amdgcn_exp2f(mx[r] - nm) + add;  // 2^-inf = 0 on the first block
        mx[r] = nm;
      }
    });
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float m = mx[r], l = sm[r];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const float om = __shfl_xor(m, o, 64), ol = __shfl_xor(l, o, 64);
        const float nm = fmaxf(m, om);
        l = (l > 0.f ? l * __builtin_amdgcn_exp2f(m - nm) : 0.f) + (ol > 0.f ? ol * __builtin_amdgcn_exp2f(om - nm) : 0.f);
        m = nm;
      }
      lse[r] = l > 0.f ? m + __builtin_amdgcn_logf(l) : 0.f;  // cur = 0: no candidate uses it
    }

    // ---- pass 2: best two group scores of each lane's stripe, per token
    float top1[TPL], top2[TPL];
#pragma unroll
    for (int u = 0; u < TPL; ++u) top1[u] = top2[u] = -INFINITY;
    sweep(gm.n_init, t_end, [&](int t0, f32x4 (&acc)[4]) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int t = t0 + nt * 16 + l16;
#pragma unroll
        for (int u = 0; u < TPL; ++u) {
          const float sv = group(acc[nt], u);
          const float v = t < lo_t[u] ? sv : -INFINITY;
          const bool c1 = v > top1[u], c2 = v > top2[u];
          top2[u] = c1 ? top1[u] : (c2 ? v : top2[u]);
          top1[u] = c1 ? v : top1[u];
        }
      }
    });
    // ---- bar of each token: the largest stripe top v with at least k stripe tops >= v
    __syncthreads();
#pragma unroll
    for (int u = 0; u < TPL; ++u)
      if (lane_tok) {
        tops[(tok0 + u) * 32 + 2 * l16] = top1[u];
        tops[(tok0 + u) * 32 + 2 * l16 + 1] = top2[u];
      }
    wave_lds_sync();
#pragma unroll
    for (int u = 0; u < TPL; ++u) {
      const float4 *rowp = reinterpret_cast<const float4 *>(tops + (tok0 + u) * 32);
      int c1 = 0, c2 = 0;
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const float4 v = rowp[x];
        c1 += (v.x >= top1[u]) + (v.y >= top1[u]) + (v.z >= top1[u]) + (v.w >= top1[u]);
        c2 += (v.x >= top2[u]) + (v.y >= top2[u]) + (v.z >= top2[u]) + (v.w >= top2[u]);
      }
      float best = -INFINITY;
      if (c1 >= k) best = top1[u];
      if (c2 >= k) best = fmaxf(best, top2[u]);
      best = row_max16(best);
      if (lane_tok && l16 == 0) bar_s[tok0 + u] = best;
    }
    __syncthreads();
    float bar[TPL];
#pragma unroll
    for (int u = 0; u < TPL; ++u) bar[u] = bar_s[tok0 + u];

    // ---- pass 3: scores >= bar join their token's list
    const int own_tok = tid / LPT, own_str = tid % LPT;
    sweep(gm.n_init, t_end, [&](int t0, f32x4 (&acc)[4]) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int t = t0 + nt * 16 + l16;
#pragma unroll
        for (int u = 0; u < TPL; ++u) {
          const float sv = group(acc[nt], u);
          if (lane_tok && t < lo_t[u] && sv >= bar[u])
            cand[tok0 + u][atomicAdd(&ccnt[tok0 + u], 1)] = make_float2(sv, __int_as_float(t));
        }
      }
      __syncthreads();
      // a list that the next chunk could overflow keeps its k best (the staging
      // buffer is free until the next chunk is staged) and raises its bar
      const int n_own = ccnt[own_tok];
      const bool cut = n_own > CAP - CH;
      if (cut)
        for (int e = own_str; e < n_own; e += LPT) {
          const float2 me = cand[own_tok][e];
          int rk = 0;
          for (int f = 0; f < n_own; ++f) {
            const float2 o = cand[own_tok][f];
            rk += beats(o.x, __float_as_int(o.y), me.x, __float_as_int(me.y));
          }
          if (rk < k) {
            tops[own_tok * 2 * KMAX + 2 * rk] = me.x;
            tops[own_tok * 2 * KMAX + 2 * rk + 1] = me.y;
          }
        }
      __syncthreads();
      if (cut) {
        for (int r = own_str; r < k; r += LPT)
          cand[own_tok][r] = make_float2(tops[own_tok * 2 * KMAX + 2 * r], tops[own_tok * 2 * KMAX + 2 * r + 1]);
        if (own_str == 0) {
          ccnt[own_tok] = k;
          bar_s[own_tok] = tops[own_tok * 2 * KMAX + 2 * (k - 1)];
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < TPL; ++u) bar[u] = bar_s[tok0 + u];
    });
  }

  // ---- the k best of each token's list, then its row
  __syncthreads();
  {
    const int own_tok = tid / LPT, own_str = tid % LPT;
    const int n = ccnt[own_tok];
    for (int e = own_str; e < n; e += LPT) {
      const float2 me = cand[own_tok][e];
      int rk = 0;
      for (int f = 0; f < n; ++f) {
        const float2 o = cand[own_tok][f];
        rk += beats(o.x, __float_as_int(o.y), me.x, __float_as_int(me.y));
      }
      if (rk < k) picks[own_tok][rk] = __float_as_int(me.y);
    }
  }
  __syncthreads();
  if (tid >= NTOK) return;
  const int i = i0 + tid;
  if (i >= gm.Lq) return;
  const int cur = (gm.q_pos0 + i) / gm.m;
  emit_row(sel + ((int64_t)bg * gm.Lq + i) * gm.ksel, picks[tid], min(k, ccnt[tid]), cur, gm);
}

// bf16 inputs: scoring on the matrix cores, selection by a bar and a short exact rank.
//
// Scores.  The group's query heads are summed in float32
// (sum_h q_h . M = (sum_h q_h) . M), and both that sum and the float32
// representative M are split into bf16 hi + lo parts (M once per call, by
// select_split_kernel).  Three bf16 MFMA chains (hi.hi + hi.lo + lo.hi, float32
// accumulate) reproduce the float32 dot product to about 2^-17 relative, far
// inside the 1e-4 score gap the selection is compared at.  The selection is
// made on these sums before the (positive) softmax scale, which orders the
// blocks the same way.
//
// Tiling.  A workgroup of NW waves takes 32 NW query rows of one (b, g); wave
// w owns two 16-row tiles (rows 32w..32w+31), so every representative fragment
// read from LDS feeds two MFMAs, and one staged chunk of CH representatives
// serves all rows of the workgroup.  Chunks are copied from global memory
// straight into swizzled LDS tiles (global_load_lds); pass 1 keeps the next
// chunk(s) in flight, pass 2 one or two (hi, lo) pairs (DB).  With k <= 16
// the kernel runs with 4 waves and one pair: 80 KB of LDS, two workgroups per
// CU, whose phases then overlap.
// In the accumulator layout lane (q4, l16) holds, per tile, the scores of rows
// 4 q4 + r (r = 0..3) for blocks t0 + 16 nt + l16: the 16 lanes of a
// quarter-wave see every block of their rows, each lane a fixed residue of
// (t - n_init) mod 16 (its "stripe").
//
// Top-k in two passes over the candidate blocks:
//   pass 1: a single hi.hi chain gives approximate scores.  The dropped terms
//           obey |q_hi . M_lo + q_lo . M_hi| <= |q_hi| |M_lo| + |q_lo| |M_hi|
//           (Cauchy-Schwarz on each), and float32 accumulation of the chains
//           adds below 2^-15 |q_hi| |M_hi|.  With the largest |M_hi| and |M_lo|
//           over the (b, g)'s blocks (select_split_kernel stores every
//           block's), one margin per row bounds every block: s_exact >=
//           s_approx - margin.  Every lane keeps the best two of these lower
//           bounds in its stripe for each of its rows.  A row's 32
//           stripe tops belong to 32 distinct blocks, so the k-th largest of
//           them (the bar) lies below the row's k-th best exact score.
//   pass 2: the exact scores are computed and those >= bar are appended to a
//           list shared by the four rows that one accumulator register holds
//           across the quarter-waves (rows 4 q4 + r, q4 = 0..3), tagged with
//           the row's q4.  A ballot gives each passing lane its slot and the
//           list length grows by a scalar bit count, so an append costs a
//           compare, a lane count and one LDS store.  A row's entries arrive in
//           block order.  On random scores about k + 3 per row pass; a list
//           that could overflow with the next append is cut to each row's k
//           best (exact rank), whose k-th score becomes that row's bar.
//   final : each list is split by row (stable), and the k best of a row
//           (score descending, block ascending) are found by counting ranks
//           within its quarter-wave and written in block order between the
//           forced init and local blocks.

// float32 K_comp -> bf16 hi, lo (hi + lo = K_comp to about 2^-17 relative) and
// the Euclidean norms of every representative's hi and lo parts (float2).  D / 8
// consecutive threads hold one representative.
template <int D>
__global__ __launch_bounds__(256) void select_split_kernel(const float *__restrict__ Kc, bf16_t *__restrict__ Mh,
                                                           bf16_t *__restrict__ Ml, float2 *__restrict__ Mnorm,
                                                           int64_t n8) {
  constexpr int TPR = D / 8;
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  float v[8];
  if (x < n8) {
    const float4 a = reinterpret_cast<const float4 *>(Kc)[2 * x];
    const float4 c = reinterpret_cast<const float4 *>(Kc)[2 * x + 1];
    v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = c.x, v[5] = c.y, v[6] = c.z, v[7] = c.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = 0.f;
  }
  bf16_t hi[8], lo[8];
  float sh = 0.f, sl = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    hi[e] = f32_to_bf16(v[e]);
    const float h = bf16_to_f32(hi[e]);
    lo[e] = f32_to_bf16(v[e] - h);
    const float l = bf16_to_f32(lo[e]);
    sh = fmaf(h, h, sh);
    sl = fmaf(l, l, sl);
  }
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) {
    sh += __shfl_xor(sh, o, 64);
    sl += __shfl_xor(sl, o, 64);
  }
  if (x >= n8) return;
  reinterpret_cast<uint4 *>(Mh)[x] = *reinterpret_cast<const uint4 *>(hi);
  reinterpret_cast<uint4 *>(Ml)[x] = *reinterpret_cast<const uint4 *>(lo);
  if (x % TPR == 0) Mnorm[x / TPR] = make_float2(sqrtf(sh), sqrtf(sl));
}

// The value of lane (l16 + r) % 16 of this lane's 16-lane row (DPP row_ror:r).
template <int R>
__device__ __forceinline__ uint32_t row_ror32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x120 + R, 0xF, 0xF, true);
}
__device__ __forceinline__ uint64_t row_ror64(uint64_t v, int r) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  switch (r) {
#define PHSA_ROR_CASE(R) \
  case R: lo = row_ror32<R>(lo); hi = row_ror32<R>(hi); break;
    PHSA_ROR_CASE(1) PHSA_ROR_CASE(2) PHSA_ROR_CASE(3) PHSA_ROR_CASE(4) PHSA_ROR_CASE(5)
    PHSA_ROR_CASE(6) PHSA_ROR_CASE(7) PHSA_ROR_CASE(8) PHSA_ROR_CASE(9) PHSA_ROR_CASE(10)
    PHSA_ROR_CASE(11) PHSA_ROR_CASE(12) PHSA_ROR_CASE(13) PHSA_ROR_CASE(14) PHSA_ROR_CASE(15)
#undef PHSA_ROR_CASE
    default: break;
  }
  return ((uint64_t)hi << 32) | lo;
}

// A candidate list entry is (score, (q4 << 16) | (0xffff - block)): q4 names
// the entry's row among the four rows that share the list.  For ranking, an
// entry becomes a 64-bit key: the score's float32 bits mapped to an
// order-preserving unsigned integer in the high word (-0 counted as +0), the
// same low word.  For two entries of one row the key order is the selection's
// order (score descending, then block ascending), so a rank is one 64-bit
// compare.
__device__ __forceinline__ uint64_t cand_key(float2 e) {
  const uint32_t b = __float_as_uint(e.x + 0.f);
  const uint32_t hi = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)hi << 32) | __float_as_uint(e.y);
}
__device__ __forceinline__ float2 key_entry(uint64_t key) {
  const uint32_t hi = (uint32_t)(key >> 32);
  return make_float2(__uint_as_float((hi & 0x80000000u) ? (hi & 0x7fffffffu) : ~hi), __uint_as_float((uint32_t)key));
}
__device__ __forceinline__ int key_row(uint64_t key) { return ((uint32_t)key >> 16) & 3; }
__device__ __forceinline__ int key_block(uint64_t key) { return 0xffff - ((uint32_t)key & 0xffff); }

// Cuts a 4-row candidate list (n entries in LDS) to the k best entries of each
// row, keeping their order; ks[q] receives row q's k-th score (-inf for a row
// with fewer than k entries).  Returns the new length.  Called by a whole wave;
// rare, so kept out of line.
template <int C4>
__device__ __noinline__ int compact_list(float2 *lp, int n, int k, float *ks) {
  constexpr int U = (C4 + 63) / 64;
  const int lane = threadIdx.x & 63;
  const uint64_t below = (1ull << lane) - 1ull;
  uint64_t *kp = reinterpret_cast<uint64_t *>(lp);  // the same bytes, as keys
  if (lane < 4) ks[lane] = -INFINITY;
  uint64_t ent[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int e = lane + 64 * u;
    ent[u] = e < n ? cand_key(lp[e]) : 0ull;
  }
  wave_lds_sync();
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (lane + 64 * u < n) kp[lane + 64 * u] = ent[u];
  wave_lds_sync();
  bool keep[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int e = lane + 64 * u;
    int rk = 0;
    for (int f = 0; f < n; ++f) {
      const uint64_t o = kp[f];
      rk += (((uint32_t)(o ^ ent[u]) & 0x30000u) == 0) & (o > ent[u]);
    }
    keep[u] = e < n && rk < k;
    if (e < n && rk == k - 1) ks[key_row(ent[u])] = key_entry(ent[u]).x;
  }
  wave_lds_sync();
  int pos = 0;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const uint64_t m = __builtin_amdgcn_ballot_w64(keep[u]);
    if (keep[u]) lp[pos + __popcll(m & below)] = key_entry(ent[u]);
    pos += __popcll(m);
  }
  wave_lds_sync();
  return pos;
}

template <int D, int G, int KMAXK, int NW, bool DB, int CH>
__global__ __launch_bounds__(NW * 64) void select_mfma_kernel(const bf16_t *__restrict__ Q,
                                                              const bf16_t *__restrict__ Mh_g,
                                                              const bf16_t *__restrict__ Ml_g,
                                                              const float2 *__restrict__ Mnorm_g,
                                                              int32_t *__restrict__ sel, Geom gm) {
  constexpr int NT = CH / 16;             // 16-block columns per chunk of CH blocks
  constexpr int RT = 2;                   // 16-row tiles per wave (B fragments are reused across them)
  constexpr int ROWS = NW * 16 * RT;      // query rows per workgroup
  constexpr int NR = 4 * RT;              // rows per lane in the accumulator layout
  constexpr int MP = D + 8;               // LDS pitch of a staged representative (sizes the staging area)
  constexpr int KB = D / 32;
  constexpr int TILE = CH * MP;           // bf16 elements reserved per staged hi (or lo) chunk
  constexpr int TD = CH * D;              // bf16 elements of a chunk copied in (swizzled [CH][D], no padding)
  constexpr int NBUF = DB ? 2 : 1;        // pass 2 buffers (one: two barriers per chunk)
  constexpr int P1 = 2 * NBUF;            // pass 1 buffers (hi only): chunks in flight P1 - 1
  constexpr int VPR = D / 8, RPI = 64 / VPR, NI = CH / RPI / NW;  // 1 KB copies per wave per chunk
  constexpr int C4 = 4 * KMAXK + PHSA_SEL_SLACK;  // capacity of a 4-row list: 4 k survivors + one 64-entry append + slack
  constexpr int NGRP = NW * NR;           // lists per workgroup
  static_assert(NI >= 1 && NI * NW * RPI == CH && TD <= TILE, "chunk copies");
  static_assert(C4 >= 4 * KMAXK + 64, "list capacity");
  // staging: pass 1 uses P1 hi chunks, pass 2 NBUF (hi, lo) pairs; the same bytes
  __shared__ __attribute__((aligned(16))) bf16_t stg[NBUF * 2 * TILE];
  __shared__ __attribute__((aligned(16))) float2 lists[NGRP * C4];  // candidate entries; bar scratch first
  __shared__ float kth_s[NGRP * 4];
  __shared__ float2 nmax_s[NW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  const TileOrder wo;
  const int bg = wo.bg, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int i0 = wo.tile * ROWS;
  const int k = gm.top_k;
  const uint64_t grp_bits = 0xffffull << (16 * q4);
  const uint64_t below = (1ull << lane) - 1ull;
  // tile row of accumulator entry (j, r) held by this lane: 32 w + 16 j + 4 q4 + r
  auto crow = [&](int rr) { return wave * 16 * RT + (rr >> 2) * 16 + q4 * 4 + (rr & 3); };
  const bf16_t *mh_bg = Mh_g + (int64_t)bg * gm.T * D;
  const bf16_t *ml_bg = Ml_g + (int64_t)bg * gm.T * D;
  const float2 *mn_bg = Mnorm_g + (int64_t)bg * gm.T;

  // largest |M_hi| and |M_lo| over the (b, g)'s blocks, for the pass-1 margin
  {
    float2 mx = make_float2(0.f, 0.f);
    for (int t = tid; t < gm.T; t += NW * 64) {
      const float2 v = mn_bg[t];
      mx.x = fmaxf(mx.x, v.x);
      mx.y = fmaxf(mx.y, v.y);
    }
    mx.x = wave_max(mx.x);
    mx.y = wave_max(mx.y);
    if (lane == 0) nmax_s[wave] = mx;
  }

  // A operands: split query-head sums of rows 32w + 16j + l16, and the norms of their parts
  bf16x8 ah[RT][KB], al[RT][KB];
  float qnh[RT], qnl[RT];
#pragma unroll
  for (int j = 0; j < RT; ++j) {
    const int ia = i0 + wave * 16 * RT + j * 16 + l16;
    float ssh = 0.f, ssl = 0.f;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      // this feature slice summed over the G heads, HU heads' loads in flight at
      // a time (all of them at once would not fit in registers for G = 8)
      constexpr int HU = G < 4 ? G : 4;
      float qs[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) qs[e] = 0.f;
#pragma unroll 1
      for (int h0 = 0; h0 < G; h0 += HU) {
        u32x4 raw[HU];
#pragma unroll
        for (int hh = 0; hh < HU; ++hh)
          raw[hh] = ia < gm.Lq ? *reinterpret_cast<const u32x4 *>(
                                     Q + (((int64_t)b * gm.Lq + ia) * gm.Hq + g * G + h0 + hh) * D + kb * 32 + kq)
                               : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int hh = 0; hh < HU; ++hh) {
          const bf16_t *v = reinterpret_cast<const bf16_t *>(&raw[hh]);
#pragma unroll
          for (int e = 0; e < 8; ++e) qs[e] += bf16_to_f32(v[e]);
        }
      }
      bf16_t hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hi[e] = f32_to_bf16(qs[e]);
        const float h = bf16_to_f32(hi[e]);
        lo[e] = f32_to_bf16(qs[e] - h);
        const float l = bf16_to_f32(lo[e]);
        ssh = fmaf(h, h, ssh);
        ssl = fmaf(l, l, ssl);
      }
      ah[j][kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(hi));
      al[j][kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(lo));
    }
    ssh += __shfl_xor(ssh, 16, 64);
    ssh += __shfl_xor(ssh, 32, 64);
    ssl += __shfl_xor(ssl, 16, 64);
    ssl += __shfl_xor(ssl, 32, 64);
    qnh[j] = sqrtf(ssh);
    qnl[j] = sqrtf(ssl);
  }
  const int last_i = min(i0 + ROWS - 1, gm.Lq - 1);
  const int t_end = k > 0 ? max(0, (gm.q_pos0 + last_i) / gm.m - gm.window / gm.m) : 0;
  const int nch = t_end > gm.n_init ? (t_end - gm.n_init + CH - 1) / CH : 0;
  // chunks ending at or below the first row's first local block hold candidates of every row
  const int lo_first = max(0, (gm.q_pos0 + i0) / gm.m - gm.window / gm.m);

  // chunk c (blocks n_init + CH c ..) of src straight into LDS tile dst, in
  // the swizzled layout (element e of row r at swz<D>(r, e)): NI one-kilobyte
  // copies per wave, lane l of a copy landing at byte 16 l of it.  Rows past
  // the last block repeat it: such blocks are never candidates.  The copies
  // count in vmcnt; a chunk is read after its copies are waited for and a
  // barrier.
  auto dma_chunk = [&](const bf16_t *src, int c, bf16_t *dst) {
    const int t0 = gm.n_init + c * CH;
#pragma unroll
    for (int v = 0; v < NI; ++v) {
      const int blk = wave * NI + v, r = blk * RPI + lane / VPR, cc = (lane % VPR) ^ (r & (VPR - 1));
      __builtin_amdgcn_global_load_lds(src + (int64_t)min(t0 + r, gm.T - 1) * D + cc * 8,
                                       (lds_void_t *)(dst + blk * RPI * D), 16, 0, 0);
    }
  };
  // waits until at most n of this wave's copies are outstanding (n a multiple of NI, at most 2 NI)
  auto dma_wait_n = [&](int n) {
    if (n >= 2 * NI) __builtin_amdgcn_s_waitcnt(0x0f70 | (2 * NI));
    else if (n >= NI) __builtin_amdgcn_s_waitcnt(0x0f70 | NI);
    else __builtin_amdgcn_s_waitcnt(0x0f70);
  };
  static_assert(2 * NI < 16, "vmcnt immediate");
  // the B fragment of 16 representatives (rows n0 .. n0 + 15) for feature slice kb
  auto frag = [&](const bf16_t *tile, int n0, int kb) { return load_bf16x8(&tile[swz<D>(n0 + l16, kb * 32 + kq)]); };

  // ---- pass 1: best two approximate scores of each lane's stripe, per row
  int lo_r[NR];
  float top1[NR], top2[NR];
#pragma unroll
  for (int rr = 0; rr < NR; ++rr) {
    const int i = i0 + crow(rr);
    lo_r[rr] = i < gm.Lq ? max(0, (gm.q_pos0 + i) / gm.m - gm.window / gm.m) : 0;
    top1[rr] = top2[rr] = -INFINITY;
  }
  // P1 - 1 chunks in flight ahead of the one in use
  for (int j = 0; j < P1 - 1 && j < nch; ++j) dma_chunk(mh_bg, j, stg + j * TD);
  auto keep2 = [&](int rr, float v) {  // best two of the stripe (top1 >= top2)
    top2[rr] = __builtin_amdgcn_fmed3f(top1[rr], top2[rr], v);  // the middle of the three
    top1[rr] = fmaxf(top1[rr], v);
  };
  for (int c = 0; c < nch; ++c) {
    dma_wait_n(min(P1 - 2, nch - 1 - c) * NI);  // chunk c landed (later chunks may still be in flight)
    lds_barrier();
    // buffer (c + P1 - 1) % P1 held chunk c - 1, which every wave finished before this barrier
    if (c + P1 - 1 < nch) dma_chunk(mh_bg, c + P1 - 1, stg + ((c + P1 - 1) % P1) * TD);
    const bf16_t *hb = stg + (c % P1) * TD;
    const int t0 = gm.n_init + c * CH;
    f32x4 acc[RT][NT];
#pragma unroll
    for (int j = 0; j < RT; ++j)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[j][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      bf16x8 bh[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bh[nt] = frag(hb, nt * 16, kb);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int j = 0; j < RT; ++j) acc[j][nt] = mfma16x16x32(ah[j][kb], bh[nt], acc[j][nt]);
    }
    if (t0 + CH <= lo_first) {
#pragma unroll
      for (int rr = 0; rr < NR; ++rr)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) keep2(rr, acc[rr >> 2][nt][rr & 3]);
    } else {
#pragma unroll
      for (int rr = 0; rr < NR; ++rr)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          keep2(rr, t0 + nt * 16 + l16 < lo_r[rr] ? acc[rr >> 2][nt][rr & 3] : -INFINITY);
    }
  }
  lds_barrier();  // pass 2 copies into the same buffers

  // ---- bar of each row: the k-th largest of its 32 stripe lower bounds (the
  // largest v with at least k of them >= v), k distinct blocks whose exact
  // scores are at least that.  The margin: |s3 - s1| <= |q_hi| |M_lo| +
  // |q_lo| |M_hi| for the three-chain score s3 and the hi.hi score s1
  // (Cauchy-Schwarz on each dropped product), plus the float32 rounding of
  // both chains, below 2^-15 |q_hi| |M_hi|.  Rows past the end take nothing.
  float thr[NR];
  {
    float2 nm = nmax_s[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) {
      nm.x = fmaxf(nm.x, nmax_s[w].x);
      nm.y = fmaxf(nm.y, nmax_s[w].y);
    }
    // [ROWS][36]: the pitch puts the four rows a quarter-wave group reads
    // together (4 rows apart) in different banks
    constexpr int SP = 36;
    static_assert(ROWS * SP * sizeof(float) <= NGRP * C4 * sizeof(float2), "bar scratch");
    float *scr = reinterpret_cast<float *>(lists);  // free until pass 2
#pragma unroll
    for (int rr = 0; rr < NR; ++rr) {
      const float eh = __shfl(qnh[rr >> 2], q4 * 4 + (rr & 3), 64);
      const float el = __shfl(qnl[rr >> 2], q4 * 4 + (rr & 3), 64);
      const float mg = fmaf(eh, fmaf(nm.x, 0x1p-15f, nm.y), el * nm.x) * 1.0001f;
      top1[rr] -= mg;
      top2[rr] -= mg;
      *reinterpret_cast<float2 *>(&scr[crow(rr) * SP + 2 * l16]) = make_float2(top1[rr], top2[rr]);
    }
    wave_lds_sync();
#pragma unroll
    for (int rr = 0; rr < NR; ++rr) {
      const float4 *rowp = reinterpret_cast<const float4 *>(scr + crow(rr) * SP);
      int c1 = 0, c2 = 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float4 v = rowp[u];
        c1 += (v.x >= top1[rr]) + (v.y >= top1[rr]) + (v.z >= top1[rr]) + (v.w >= top1[rr]);
        c2 += (v.x >= top2[rr]) + (v.y >= top2[rr]) + (v.z >= top2[rr]) + (v.w >= top2[rr]);
      }
      float best = -INFINITY;
      if (c1 >= k) best = top1[rr];
      if (c2 >= k) best = fmaxf(best, top2[rr]);
      best = row_max16(best);
      thr[rr] = i0 + crow(rr) < gm.Lq ? best : INFINITY;
    }
    wave_lds_sync();
  }

  // ---- pass 2: exact scores >= bar join the 4-row lists
  float2 *mylists = lists + wave * NR * C4;  // list rr of this wave at mylists + rr * C4
  int cnt[NR];                                 // list lengths (wave-uniform)
#pragma unroll
  for (int rr = 0; rr < NR; ++rr) cnt[rr] = 0;
  const uint32_t low_lane = ((uint32_t)q4 << 16) | (uint32_t)(0xffff - l16);
  // cuts list rr to each row's k best, in order; each row's k-th score becomes its bar
  auto compact = [&](int rr) {
    float *ks = kth_s + (wave * NR + rr) * 4;
    cnt[rr] = __builtin_amdgcn_readfirstlane(compact_list<C4>(mylists + rr * C4, cnt[rr], k, ks));
    thr[rr] = fmaxf(thr[rr], ks[q4]);
  };
  // one chunk's exact scores (three chains over hi / lo staged chunks), appended
  auto pass2_chunk = [&](const bf16_t *hb, const bf16_t *lb, int c) {
    const int t0 = gm.n_init + c * CH;
    f32x4 acc[RT][NT];
#pragma unroll
    for (int j = 0; j < RT; ++j)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[j][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      bf16x8 bh[NT], bl[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        bh[nt] = frag(hb, nt * 16, kb);
        bl[nt] = frag(lb, nt * 16, kb);
      }
      // each chain over all RT x 4 accumulators in turn, so that consecutive
      // MFMAs are independent; every accumulator still takes hi.hi, hi.lo,
      // lo.hi of each kb in that order
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int j = 0; j < RT; ++j) acc[j][nt] = mfma16x16x32(ah[j][kb], bh[nt], acc[j][nt]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int j = 0; j < RT; ++j) acc[j][nt] = mfma16x16x32(ah[j][kb], bl[nt], acc[j][nt]);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int j = 0; j < RT; ++j) acc[j][nt] = mfma16x16x32(al[j][kb], bh[nt], acc[j][nt]);
    }
    float lowv[NT];                           // the entries' low words, per block column
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) lowv[nt] = __uint_as_float(low_lane - (uint32_t)(t0 + nt * 16));
    auto appends = [&](auto inner_c) {
      constexpr bool INNER = decltype(inner_c)::value;  // every block is a candidate of every row
#pragma unroll
      for (int rr = 0; rr < NR; ++rr) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          if (cnt[rr] > C4 - 64) compact(rr);
          const float sc = acc[rr >> 2][nt][rr & 3];
          // wave masks straight from the compares (FCMP_OGE = 3, ICMP_SLT = 40)
          uint64_t m = __builtin_amdgcn_fcmpf(sc, thr[rr], 3);
          if (!INNER) m &= __builtin_amdgcn_sicmp(t0 + nt * 16 + l16, lo_r[rr], 40);
          if (m) {
            if (__builtin_amdgcn_inverse_ballot_w64(m)) {  // the passing lanes, straight from the mask
              const int slot = (int)__builtin_amdgcn_mbcnt_hi(
                  (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, (uint32_t)cnt[rr]));
              float *ent = reinterpret_cast<float *>(mylists + rr * C4 + slot);
              ent[0] = sc;
              ent[1] = lowv[nt];
            }
            cnt[rr] = __builtin_amdgcn_readfirstlane(cnt[rr] + (int)__popcll(m));
          }
        }
      }
    };
    if (t0 + CH <= lo_first) appends(std::true_type{});
    else appends(std::false_type{});
  };
  if (DB) {  // chunk c + 1 is copied into the other (hi, lo) pair while chunk c is used
    if (nch > 0) {
      dma_chunk(mh_bg, 0, stg);
      dma_chunk(ml_bg, 0, stg + TD);
    }
    for (int c = 0; c < nch; ++c) {
      dma_wait_n(0);
      lds_barrier();  // chunk c landed; every wave finished chunk c - 1, whose pair is now free
      bf16_t *cur = stg + (c & 1) * 2 * TD, *nxt = stg + ((c + 1) & 1) * 2 * TD;
      if (c + 1 < nch) {
        dma_chunk(mh_bg, c + 1, nxt);
        dma_chunk(ml_bg, c + 1, nxt + TD);
      }
      pass2_chunk(cur, cur + TD, c);
    }
    lds_barrier();
  } else {
    for (int c = 0; c < nch; ++c) {
      lds_barrier();  // every wave finished chunk c - 1
      dma_chunk(mh_bg, c, stg);
      dma_chunk(ml_bg, c, stg + TD);
      dma_wait_n(0);
      lds_barrier();
      pass2_chunk(stg, stg + TD, c);
    }
    lds_barrier();
  }

  // ---- final: per list, split by row into the (now free) staging area, then
  // each quarter-wave ranks its row's entries and writes the row
  uint64_t *split = reinterpret_cast<uint64_t *>(stg) + wave * C4;  // this wave's scratch, as keys
  static_assert(NW * C4 * sizeof(uint64_t) <= NBUF * 2 * TILE * sizeof(bf16_t), "split scratch");
#pragma unroll 1
  for (int rr = 0; rr < NR; ++rr) {
    const float2 *lp = mylists + rr * C4;
    const int n = cnt[rr];
    // row counts, then a stable split into [row 0 | row 1 | row 2 | row 3]
    int nq[4] = {0, 0, 0, 0};
    for (int e0 = 0; e0 < n; e0 += 64) {
      const int e = e0 + lane;
      const int tg = e < n ? (int)(__float_as_uint(lp[e].y) >> 16) : 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) nq[q] += __popcll(__builtin_amdgcn_ballot_w64(tg == q));
    }
    int off[4] = {0, nq[0], nq[0] + nq[1], nq[0] + nq[1] + nq[2]};
    for (int e0 = 0; e0 < n; e0 += 64) {
      const int e = e0 + lane;
      const uint64_t ent = e < n ? cand_key(lp[e]) : 0ull;
      const int tg = e < n ? key_row(ent) : 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint64_t m = __builtin_amdgcn_ballot_w64(tg == q);
        if (tg == q) split[off[q] + __popcll(m & below)] = ent;
        off[q] += __popcll(m);
      }
    }
    wave_lds_sync();
    // this quarter-wave's row
    const int my_n = q4 == 0 ? nq[0] : q4 == 1 ? nq[1] : q4 == 2 ? nq[2] : nq[3];
    const int my_off = q4 == 0 ? 0 : q4 == 1 ? nq[0] : q4 == 2 ? nq[0] + nq[1] : nq[0] + nq[1] + nq[2];
    const int max_n = max(max(nq[0], nq[1]), max(nq[2], nq[3]));
    const uint64_t *rp = split + my_off;
    const int i = i0 + crow(rr);
    const bool live = i < gm.Lq;
    int32_t *out = sel + ((int64_t)bg * gm.Lq + (live ? i : 0)) * gm.ksel;
    const int cur = (gm.q_pos0 + i) / gm.m;
    const int ni = min(gm.n_init, cur + 1);
    const int npick = min(my_n, k);
    const bool cut = __builtin_amdgcn_ballot_w64(my_n > k) != 0;  // some row of the list has more than k
    int pos = 0;
    if (max_n <= 32) {
      // up to 32 entries per row: lane l16 holds entries l16 and 16 + l16 as keys
      // (0 for none, below every entry) and counts the keys above its own with
      // the 15 rotations of its 16-lane row (DPP, no LDS)
      const uint64_t k0 = l16 < my_n ? rp[l16] : 0ull, k1 = l16 + 16 < my_n ? rp[16 + l16] : 0ull;
      int r0 = k1 > k0, r1 = k0 > k1;
      if (cut && max_n <= 16) {  // one entry per lane
#pragma unroll
        for (int r = 1; r < 16; ++r) r0 += row_ror64(k0, r) > k0;
      } else if (cut) {
#pragma unroll
        for (int r = 1; r < 16; ++r) {
          const uint64_t o0 = row_ror64(k0, r), o1 = row_ror64(k1, r);
          r0 += (o0 > k0) + (o1 > k0);
          r1 += (o0 > k1) + (o1 > k1);
        }
      }
      const bool take0 = l16 < my_n && r0 < k, take1 = l16 + 16 < my_n && r1 < k;
      const uint64_t m0 = __builtin_amdgcn_ballot_w64(take0) & grp_bits;
      const uint64_t m1 = __builtin_amdgcn_ballot_w64(take1) & grp_bits;
      if (take0 && live) out[ni + __popcll(m0 & below)] = key_block(k0);
      if (take1 && live) out[ni + __popcll(m0) + __popcll(m1 & below)] = key_block(k1);
    } else {
      // longer lists (many equal scores): rank against every entry through LDS
      for (int j0 = 0; j0 < max_n; j0 += 16) {
        const int j = j0 + l16;
        const bool have = j < my_n;
        const uint64_t me = have ? rp[j] : 0ull;
        int rk = 0;
        for (int f = 0; f < max_n; ++f) rk += (f < my_n) & (rp[min(f, max(my_n - 1, 0))] > me);
        const bool take = have && rk < k;
        const uint64_t m = __builtin_amdgcn_ballot_w64(take) & grp_bits;
        if (take && live) out[ni + pos + __popcll(m & below)] = key_block(me);
        pos += __popcll(m);
      }
    }
    // forced init blocks, local blocks and padding around the picks
    if (live) {
      const int lo1 = max(max(0, cur - gm.window / gm.m), ni);
      for (int s = l16; s < gm.ksel; s += 16) {
        if (s >= ni && s < ni + npick) continue;
        const int x = s - ni - npick;
        out[s] = s < ni ? s : (lo1 + x <= cur ? lo1 + x : -1);
      }
    }
    wave_lds_sync();
  }
}

template <typename T, int D>
static hipError_t launch_select_t(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  dim3 grid((g.Lq + 63) / 64, g.B * g.Hkv);
  timing_begin("phsa_select", s);
  if (g.top_k <= 8)
    hipLaunchKernelGGL((select_kernel<T, D, 8>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  else if (g.top_k <= 16)
    hipLaunchKernelGGL((select_kernel<T, D, 16>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  else
    hipLaunchKernelGGL((select_kernel<T, D, 32>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  timing_end(s);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_select_softmax(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  dim3 grid((g.Lq + 64 / g.G - 1) / (64 / g.G), g.B * g.Hkv);
  timing_begin("phsa_select_softmax", s);
  if (g.top_k <= 8)
    hipLaunchKernelGGL((select_softmax_kernel<T, D, 8>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  else if (g.top_k <= 16)
    hipLaunchKernelGGL((select_softmax_kernel<T, D, 16>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  else
    hipLaunchKernelGGL((select_softmax_kernel<T, D, 32>), grid, dim3(256), 0, s, static_cast<const T *>(Q), Kc, sel, g);
  timing_end(s);
  return hipGetLastError();
}

template <int D, int G>
static hipError_t launch_select_mfma(const Geom &g, const void *Q, const float *Kc, int32_t *sel, char *ws,
                                     hipStream_t s) {
  const int64_t n = (int64_t)g.B * g.Hkv * g.T * D;
  bf16_t *mh = reinterpret_cast<bf16_t *>(ws), *ml = mh + n;
  float2 *mnorm = reinterpret_cast<float2 *>(ml + n);
  timing_begin("phsa_select_split", s);
  hipLaunchKernelGGL(select_split_kernel<D>, dim3((unsigned)((n / 8 + 255) / 256)), dim3(256), 0, s, Kc, mh, ml, mnorm,
                     n / 8);
  timing_end(s);
  timing_begin("phsa_select", s);
  if (g.top_k <= 16) {
    const dim3 grid((g.Lq + PHSA_SEL_NW * 32 - 1) / (PHSA_SEL_NW * 32), g.B * g.Hkv);
    hipLaunchKernelGGL((select_mfma_kernel<D, G, 16, PHSA_SEL_NW, PHSA_SEL_DB, PHSA_SEL_CH>), grid, dim3(PHSA_SEL_NW * 64), 0, s,
                       static_cast<const bf16_t *>(Q), mh, ml, mnorm, sel, g);
  } else {
    const dim3 grid((g.Lq + 255) / 256, g.B * g.Hkv);
    hipLaunchKernelGGL((select_mfma_kernel<D, G, 32, 8, false, 64>), grid, dim3(512), 0, s,
                       static_cast<const bf16_t *>(Q), mh, ml, mnorm, sel, g);
  }
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_select_mfma_d(const Geom &g, const void *Q, const float *Kc, int32_t *sel, char *split,
                                       hipStream_t s) {
  switch (g.G) {
    case 1: return launch_select_mfma<D, 1>(g, Q, Kc, sel, split, s);
    case 2: return launch_select_mfma<D, 2>(g, Q, Kc, sel, split, s);
    case 4: return launch_select_mfma<D, 4>(g, Q, Kc, sel, split, s);
    case 8: return launch_select_mfma<D, 8>(g, Q, Kc, sel, split, s);
    default: return launch_select_t<bf16_t, D>(g, Q, Kc, sel, s);
  }
}

template <int D, int G>
static hipError_t launch_select_softmax_mfma(const Geom &g, const void *Q, const float *Kc, int32_t *sel, char *ws,
                                             hipStream_t s) {
  const int64_t n = (int64_t)g.B * g.Hkv * g.T * D;
  bf16_t *mh = reinterpret_cast<bf16_t *>(ws), *ml = mh + n;
  float2 *mnorm = reinterpret_cast<float2 *>(ml + n);
  timing_begin("phsa_select_split", s);
  hipLaunchKernelGGL(select_split_kernel<D>, dim3((unsigned)((n / 8 + 255) / 256)), dim3(256), 0, s, Kc, mh, ml, mnorm,
                     n / 8);
  timing_end(s);
  constexpr int NTOK = 64 / G;
  const dim3 grid((g.Lq + NTOK - 1) / NTOK, g.B * g.Hkv);
  timing_begin("phsa_select_softmax", s);
  if (g.top_k <= 16)
    hipLaunchKernelGGL((select_softmax_mfma_kernel<D, G, 16>), grid, dim3(256), 0, s,
                       static_cast<const bf16_t *>(Q), mh, ml, sel, g);
  else
    hipLaunchKernelGGL((select_softmax_mfma_kernel<D, G, 32>), grid, dim3(256), 0, s,
                       static_cast<const bf16_t *>(Q), mh, ml, sel, g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_select_softmax_mfma_d(const Geom &g, const void *Q, const float *Kc, int32_t *sel,
                                               char *split, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_select_softmax_mfma<D, 1>(g, Q, Kc, sel, split, s);
    case 2: return launch_select_softmax_mfma<D, 2>(g, Q, Kc, sel, split, s);
    case 4: return launch_select_softmax_mfma<D, 4>(g, Q, Kc, sel, split, s);
    default: return launch_select_softmax_mfma<D, 8>(g, Q, Kc, sel, split, s);
  }
}

hipError_t launch_select(const Geom &g, const void *Q, const float *Kc, int32_t *sel, void *ws, hipStream_t s) {
  char *split = static_cast<char *>(ws);
  if (g.sel_mode == 1) {
    if (g.dtype == 0 && g.G <= 8)
      return g.d == 128 ? launch_select_softmax_mfma_d<128>(g, Q, Kc, sel, split, s)
                        : launch_select_softmax_mfma_d<64>(g, Q, Kc, sel, split, s);
    if (g.dtype == 0)
      return g.d == 128 ? launch_select_softmax<bf16_t, 128>(g, Q, Kc, sel, s)
                        : launch_select_softmax<bf16_t, 64>(g, Q, Kc, sel, s);
    return g.d == 128 ? launch_select_softmax<float, 128>(g, Q, Kc, sel, s)
                      : launch_select_softmax<float, 64>(g, Q, Kc, sel, s);
  }
  if (g.dtype == 0)
    return g.d == 128 ? launch_select_mfma_d<128>(g, Q, Kc, sel, split, s)
                      : launch_select_mfma_d<64>(g, Q, Kc, sel, split, s);
  return g.d == 128 ? launch_select_t<float, 128>(g, Q, Kc, sel, s) : launch_select_t<float, 64>(g, Q, Kc, sel, s);
}

}  // namespace phsa

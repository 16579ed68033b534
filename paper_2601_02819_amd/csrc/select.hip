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

#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool beats(float s1, int t1, float s2, int t2) {
  return s1 > s2 || (s1 == s2 && t1 < t2);
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
  const int bg = blockIdx.y, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int i = blockIdx.x * 64 + lane;
  const bool row_ok = i < gm.Lq;
  const int pos = gm.q_pos0 + (row_ok ? i : gm.Lq - 1);
  const int cur = pos / gm.m;
  const int lo = max(0, cur - gm.window / gm.m);       // first local block
  // candidate blocks of this row: n_init <= t < lo
  const int last_i = min(blockIdx.x * 64 + 63, gm.Lq - 1);
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

  // Merge the four wave lists.
  __syncthreads();
  float *list_s = reinterpret_cast<float *>(smem);
  int *list_t = reinterpret_cast<int *>(smem) + 4 * 64 * KMAX;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    list_s[(wave * 64 + lane) * KMAX + k] = ls[k];
    list_t[(wave * 64 + lane) * KMAX + k] = lt[k];
  }
  __syncthreads();
  if (wave != 0 || !row_ok) return;

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
  // ascending block order of the picks (insertion sort, at most KMAX items)
  for (int a = 1; a < npick; ++a) {
    const int x = picks[lane][a];
    int c = a - 1;
    while (c >= 0 && picks[lane][c] > x) {
      picks[lane][c + 1] = picks[lane][c];
      --c;
    }
    picks[lane][c + 1] = x;
  }
  int32_t *out = sel + ((int64_t)bg * gm.Lq + i) * gm.ksel;
  int n = 0;
  const int ni = min(gm.n_init, cur + 1);
  for (int t = 0; t < ni; ++t) out[n++] = t;
  for (int a = 0; a < npick; ++a) out[n++] = picks[lane][a];
  for (int t = max(lo, ni); t <= cur; ++t) out[n++] = t;
  for (; n < gm.ksel; ++n) out[n] = -1;
}

// bf16 inputs: scoring on the matrix cores.
//
// The group's query heads are summed in float32 (sum_h q_h . M = (sum_h q_h) . M),
// and both that sum and the float32 representative M are split into bf16
// hi + lo parts.  Three bf16 MFMA chains (hi.hi + hi.lo + lo.hi, float32
// accumulate) reproduce the float32 dot product to about 2^-17 relative, far
// inside the 1e-4 score gap the selection is compared at.  Wave w owns the
// 16 query rows 16w..16w+15 of the 64-row tile; representatives stream
// through LDS in chunks of 64 blocks, pre-split into hi/lo tiles.
//
// Top-k: four threads per row (one in each wave) keep private sorted lists
// of (score, block) in registers.  Each private list's k-th entry is a lower
// bound on the row's final k-th score, so the strongest of the four is the
// bar a new score must beat.  Scores that pass are appended to the row's LDS
// buffer, and the row's four threads insert every fourth of them into their
// lists (compare/select only, no memory traffic).  After the last chunk the
// four lists are merged.
template <int D, int G, int KMAX>
__global__ __launch_bounds__(256) void select_mfma_kernel(const bf16_t *__restrict__ Q, const float *__restrict__ Kc,
                                                          int32_t *__restrict__ sel, Geom gm) {
  constexpr int CH = 64;
  constexpr int MP = D + 8;
  constexpr int KB = D / 32;
  constexpr int TILE_BYTES = 2 * CH * MP * 2;
  constexpr int LIST_BYTES = 4 * 64 * KMAX * 8;
  constexpr int BUF = TILE_BYTES > LIST_BYTES ? TILE_BYTES : LIST_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[BUF];
  // candidate buffers, one row per query row; rows padded by one word so that the
  // merge threads (lane = row) do not all hit the same LDS bank
  __shared__ float nb_s[64][CH + 1];
  __shared__ int nb_t[64][CH + 1];
  __shared__ int nnew[64];
  __shared__ float bar_s[4][64];
  __shared__ int bar_t[4][64];
  bf16_t *Mh = reinterpret_cast<bf16_t *>(smem);
  bf16_t *Ml = Mh + CH * MP;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  const int bg = blockIdx.y, b = bg / gm.Hkv, g = bg % gm.Hkv;
  const int i0 = blockIdx.x * 64;

  // A operand: split query-head sums of row 16w + l16 (all loads issued together)
  bf16x8 ah[KB], al[KB];
  {
    const int ia = i0 + wave * 16 + l16;
    uint4 raw[G][KB];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        raw[hh][kb] = ia < gm.Lq ? *reinterpret_cast<const uint4 *>(
                                       Q + (((int64_t)b * gm.Lq + ia) * gm.Hq + g * G + hh) * D + kb * 32 + kq)
                                 : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      float qs[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) qs[e] = 0.f;
#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        const bf16_t *v = reinterpret_cast<const bf16_t *>(&raw[hh][kb]);
#pragma unroll
        for (int e = 0; e < 8; ++e) qs[e] += bf16_to_f32(v[e]);
      }
      bf16_t hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hi[e] = f32_to_bf16(qs[e]);
        lo[e] = f32_to_bf16(qs[e] - bf16_to_f32(hi[e]));
      }
      ah[kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(hi));
      al[kb] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(lo));
    }
  }
  // private list of thread (row = lane, part = wave)
  float ls[KMAX];
  int lt[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    ls[k] = -FLT_MAX;
    lt[k] = 0x7fffffff;
  }
  int nl = 0;
  nnew[lane] = 0;  // (every wave writes the same zero)
  bar_s[wave][lane] = -FLT_MAX;
  bar_t[wave][lane] = 0x7fffffff;
  // first local block of the 4 rows this lane holds in the C layout (no candidates past it)
  int lo_r[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + wave * 16 + q4 * 4 + r;
    lo_r[r] = i < gm.Lq ? max(0, (gm.q_pos0 + i) / gm.m - gm.window / gm.m) : 0;
  }
  const int last_i = min(i0 + 63, gm.Lq - 1);
  const int t_end = gm.top_k > 0 ? max(0, (gm.q_pos0 + last_i) / gm.m - gm.window / gm.m) : 0;
  const float *kc_bg = Kc + (int64_t)bg * gm.T * D;

  // representative chunks: the next chunk's float32 rows are fetched into
  // registers while the current chunk is scored
  constexpr int NM = CH * D / (256 * 4);
  float4 mreg[NM];
  auto fetch_chunk = [&](int t0) {
    const int nblk = min(CH, gm.T - t0);
#pragma unroll
    for (int k = 0; k < NM; ++k) {
      const int e = (tid + 256 * k) * 4, row = e / D, c = e % D;
      mreg[k] = row < nblk ? *reinterpret_cast<const float4 *>(kc_bg + (int64_t)(t0 + row) * D + c)
                           : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  if (gm.n_init < t_end) fetch_chunk(gm.n_init);

  for (int t0 = gm.n_init; t0 < t_end; t0 += CH) {
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NM; ++k) {
      const int e = (tid + 256 * k) * 4, row = e / D, c = e % D;
      const float mv[4] = {mreg[k].x, mreg[k].y, mreg[k].z, mreg[k].w};
      bf16_t hi[4], lo[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        hi[x] = f32_to_bf16(mv[x]);
        lo[x] = f32_to_bf16(mv[x] - bf16_to_f32(hi[x]));
      }
      *reinterpret_cast<uint2 *>(&Mh[row * MP + c]) = *reinterpret_cast<const uint2 *>(hi);
      *reinterpret_cast<uint2 *>(&Ml[row * MP + c]) = *reinterpret_cast<const uint2 *>(lo);
    }
    __syncthreads();
    if (t0 + CH < t_end) fetch_chunk(t0 + CH);

    f32x4 acc[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const bf16x8 bh = load_bf16x8(&Mh[(nt * 16 + l16) * MP + kb * 32 + kq]);
        const bf16x8 bl = load_bf16x8(&Ml[(nt * 16 + l16) * MP + kb * 32 + kq]);
        acc[nt] = mfma16x16x32(ah[kb], bh, acc[nt]);
        acc[nt] = mfma16x16x32(ah[kb], bl, acc[nt]);
        acc[nt] = mfma16x16x32(al[kb], bh, acc[nt]);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = wave * 16 + q4 * 4 + r;
      float bs = bar_s[0][row];
      int bt = bar_t[0][row];
#pragma unroll
      for (int p = 1; p < 4; ++p) {
        const float s2 = bar_s[p][row];
        const int t2 = bar_t[p][row];
        if (beats(s2, t2, bs, bt)) {
          bs = s2;
          bt = t2;
        }
      }
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int t = t0 + nt * 16 + l16;
        const float s = acc[nt][r] * gm.scale;
        if (t < lo_r[r] && beats(s, t, bs, bt)) {
          const int slot = atomicAdd(&nnew[row], 1);
          nb_s[row][slot] = s;
          nb_t[row][slot] = t;
        }
      }
    }
    __syncthreads();
    const int nn = nnew[lane];
    for (int e = wave; e < nn; e += 4) {
      float s = nb_s[lane][e];
      int ct = nb_t[lane][e];
      if (!beats(s, ct, ls[KMAX - 1], lt[KMAX - 1])) continue;
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
      ++nl;
    }
    if (nl >= gm.top_k) {  // list holds top_k real entries: its k-th is a valid bar
      float ks = ls[0];
      int kt = lt[0];
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k == gm.top_k - 1) {
          ks = ls[k];
          kt = lt[k];
        }
      bar_s[wave][lane] = ks;
      bar_t[wave][lane] = kt;
    }
    __syncthreads();
    if (wave == 0) nnew[lane] = 0;
  }

  // merge the four private lists of every row
  __syncthreads();
  float *list_s = reinterpret_cast<float *>(smem);
  int *list_t = reinterpret_cast<int *>(smem) + 4 * 64 * KMAX;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    list_s[(wave * 64 + lane) * KMAX + k] = ls[k];
    list_t[(wave * 64 + lane) * KMAX + k] = lt[k];
  }
  __syncthreads();
  const int i = i0 + lane;
  if (wave != 0 || i >= gm.Lq) return;
  int head[4] = {0, 0, 0, 0};
  int picks[KMAX];
  int npick = 0;
#pragma unroll 1
  for (int p = 0; p < gm.top_k; ++p) {
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
    // insert bt into the ascending picks (the elements above bt form a suffix)
    int pos = npick;
#pragma unroll
    for (int k = KMAX - 2; k >= 0; --k)
      if (k < npick && picks[k] > bt) {
        picks[k + 1] = picks[k];
        pos = k;
      }
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (k == pos) picks[k] = bt;
    ++npick;
  }
  const int cur = (gm.q_pos0 + i) / gm.m;
  const int lo = max(0, cur - gm.window / gm.m);
  int32_t *out = sel + ((int64_t)bg * gm.Lq + i) * gm.ksel;
  int n = 0;
  const int ni = min(gm.n_init, cur + 1);
  for (int t = 0; t < ni; ++t) out[n++] = t;
#pragma unroll
  for (int k = 0; k < KMAX; ++k)
    if (k < npick) out[n + k] = picks[k];
  n += npick;
  for (int t = max(lo, ni); t <= cur; ++t) out[n++] = t;
  for (; n < gm.ksel; ++n) out[n] = -1;
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

template <int D, int G>
static hipError_t launch_select_mfma(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  dim3 grid((g.Lq + 63) / 64, g.B * g.Hkv);
  const bf16_t *q = static_cast<const bf16_t *>(Q);
  timing_begin("phsa_select", s);
  if (g.top_k <= 8)
    hipLaunchKernelGGL((select_mfma_kernel<D, G, 8>), grid, dim3(256), 0, s, q, Kc, sel, g);
  else if (g.top_k <= 16)
    hipLaunchKernelGGL((select_mfma_kernel<D, G, 16>), grid, dim3(256), 0, s, q, Kc, sel, g);
  else
    hipLaunchKernelGGL((select_mfma_kernel<D, G, 32>), grid, dim3(256), 0, s, q, Kc, sel, g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_select_mfma_d(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_select_mfma<D, 1>(g, Q, Kc, sel, s);
    case 2: return launch_select_mfma<D, 2>(g, Q, Kc, sel, s);
    case 4: return launch_select_mfma<D, 4>(g, Q, Kc, sel, s);
    case 8: return launch_select_mfma<D, 8>(g, Q, Kc, sel, s);
    default: return launch_select_t<bf16_t, D>(g, Q, Kc, sel, s);
  }
}

hipError_t launch_select(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  if (g.dtype == 0)
    return g.d == 128 ? launch_select_mfma_d<128>(g, Q, Kc, sel, s) : launch_select_mfma_d<64>(g, Q, Kc, sel, s);
  return g.d == 128 ? launch_select_t<float, 128>(g, Q, Kc, sel, s) : launch_select_t<float, 64>(g, Q, Kc, sel, s);
}

}  // namespace phsa

// Relevance scoring + block selection (Eq. 8 logits; Algorithm 1 block
// selection with forced init / local blocks, causal block mask, top-k and
// Unique).
//
// One workgroup per (64-query tile, b*Hkv + g).  Lane r of every wave owns
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

hipError_t launch_select(const Geom &g, const void *Q, const float *Kc, int32_t *sel, hipStream_t s) {
  if (g.dtype == 0)
    return g.d == 128 ? launch_select_t<bf16_t, 128>(g, Q, Kc, sel, s) : launch_select_t<bf16_t, 64>(g, Q, Kc, sel, s);
  return g.d == 128 ? launch_select_t<float, 128>(g, Q, Kc, sel, s) : launch_select_t<float, 64>(g, Q, Kc, sel, s);
}

}  // namespace phsa

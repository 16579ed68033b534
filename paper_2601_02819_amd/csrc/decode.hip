// One decode step with a block KV cache: each of B sequences has one new
// query at position Lk - 1 (its key/value are already in the cache), scores
// the cache's T block representatives, selects, and attends over the chosen
// blocks (Eq. 8, Algorithm 1 selection, Eq. 10-11).  All three kernels are
// memory-bound: the representatives and the selected K/V blocks are each
// read once.
//
//   decode_select : one workgroup of 8 waves per (b, g).  Lanes read K_comp
//                   rows as float4 (D / 4 lanes per row, 8 loads in flight
//                   each) and reduce a row's dot product by shuffles; the
//                   top-k (score desc, block asc) comes from per-wave bitonic
//                   sorts of 64-candidate chunks merged pairwise in LDS.
//   decode_attn   : one workgroup per (b, g) streams its selected K/V blocks
//                   with coalesced 16-byte loads, keeps a running softmax per
//                   wave and merges the waves in LDS: O and LSE directly.
// With per-sequence cache lengths (phsa_decode_varlen) sequence b's query sits
// at position len[b] - 1; its own block may be partly written, and keys past
// the query are masked without reading their values.  cache_append adds one
// token per sequence and maintains the block representatives.
#include <float.h>
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {

__device__ __forceinline__ bool beats_d(float s1, int t1, float s2, int t2) {
  return s1 > s2 || (s1 == s2 && t1 < t2);
}

// One (score, block) pair per lane, sorted across the wave best first
// (higher score, then lower block) by a bitonic network over shuffles.
__device__ __forceinline__ void wave_sort_best_first(float &s, int &t, int lane) {
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const float os = __shfl_xor(s, stride, 64);
      const int ot = __shfl_xor(t, stride, 64);
      const bool want_better = ((lane & size) == 0) == ((lane & stride) == 0);
      if (beats_d(os, ot, s, t) == want_better && !(os == s && ot == t)) {
        s = os;
        t = ot;
      }
    }
}

// r := the best 64 of r and v, best first (both best-first sorted across the wave).
__device__ __forceinline__ void wave_merge_best_first(float &rs, int &rt, float vs, int vt, int lane) {
  const float ws = __shfl(vs, 63 - lane, 64);
  const int wt = __shfl(vt, 63 - lane, 64);
  if (beats_d(ws, wt, rs, rt)) {
    rs = ws;
    rt = wt;
  }
  // r is now bitonic; finish with the merge stages of a best-first sort
#pragma unroll
  for (int stride = 32; stride > 0; stride >>= 1) {
    const float os = __shfl_xor(rs, stride, 64);
    const int ot = __shfl_xor(rt, stride, 64);
    const bool want_better = (lane & stride) == 0;
    if (beats_d(os, ot, rs, rt) == want_better && !(os == rs && ot == rt)) {
      rs = os;
      rt = ot;
    }
  }
}

// Cache length of sequence b: clen[b] clamped to [1, capacity], or the
// uniform Lk when no length array is given.
__device__ __forceinline__ int seq_len(const int32_t *clen, int b, const Geom &gm) {
  return clen ? min(max(clen[b], 1), gm.Lk) : gm.Lk;
}

// Sum over the CPR consecutive lanes that share a key row (CPR = 8, 16 or 32),
// every lane getting the total.  Within a 16-lane row DPP moves do it: lane ^ 1
// and lane ^ 2 (quad permutations), then the mirrored half row and the
// mirrored row, which pair the quad sums as lane ^ 4 and lane ^ 8 would (the
// same additions, so the same result as a shuffle butterfly).  Rows are paired
// by a shuffle.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float a) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), CTRL, 0xF, 0xF, true));
}
template <int CPR>
__device__ __forceinline__ float key_row_sum(float a) {
  static_assert(CPR == 8 || CPR == 16 || CPR == 32, "key rows span 8, 16 or 32 lanes");
  a += dpp_move<0xB1>(a);   // quad_perm [1, 0, 3, 2]
  a += dpp_move<0x4E>(a);   // quad_perm [2, 3, 0, 1]
  a += dpp_move<0x141>(a);  // row_half_mirror
  if constexpr (CPR >= 16) a += dpp_move<0x140>(a);  // row_mirror
  if constexpr (CPR >= 32) a += __shfl_xor(a, 16, 64);
  return a;
}

// MODE 0 ranks on the summed logits of the group's heads.  MODE 1
// (PHSA_FLAG_SELECT_SOFTMAX_SUM) keeps every head's log2 logits of the
// complete blocks 0..cur-1 in LDS, reduces each head's log2 normaliser over
// the workgroup, and scores a candidate by log2 sum_h 2^(x_h - lse_h).
template <typename T, int D, int MODE>
__global__ __launch_bounds__(512) void decode_select_kernel(const T *__restrict__ Q, const float *__restrict__ Kc,
                                                            const int32_t *__restrict__ clen,
                                                            int32_t *__restrict__ sel, Geom gm) {
  constexpr int LPR = D / 4;      // lanes per representative row (one float4 each)
  constexpr int RPW = 64 / LPR;   // rows per wave load instruction
  constexpr int U = 8;            // load instructions in flight per lane
  constexpr int GM = MODE == 1 ? 8 : 1;   // heads kept apart (the group size is at most 8)
  extern __shared__ float sc[];   // MODE 0: [T] scores; MODE 1: [G][T] head logits, then scores in row 0
  __shared__ float mbuf_s[4][64];
  __shared__ int mbuf_t[4][64];
  __shared__ float red_m[8][8], red_l[8][8];
  const int bg = blockIdx.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane / LPR, c4 = (lane % LPR) * 4;
  const int NH = MODE == 1 ? gm.G : 1;
  float q[GM][4];
#pragma unroll
  for (int h = 0; h < GM; ++h)
#pragma unroll
    for (int e = 0; e < 4; ++e) q[h][e] = 0.f;
  for (int hh = 0; hh < gm.G; ++hh) {
    const T *src = Q + ((int64_t)b * gm.Hq + g * gm.G + hh) * D + c4;
#pragma unroll
    for (int h = 0; h < GM; ++h)
      if (MODE == 0 || h == hh) {
#pragma unroll
        for (int e = 0; e < 4; ++e) q[h][e] += to_f32<T>(src[e]) * (MODE == 1 ? gm.scale * kLog2e : 1.f);
      }
  }
  const int cur = (seq_len(clen, b, gm) - 1) / gm.m;  // the query's own block
  const int lo = max(0, cur - gm.window / gm.m);
  // MODE 0 scores the candidates n_init <= t < lo; MODE 1 every complete block t < cur
  const int s0 = MODE == 1 ? 0 : gm.n_init, s1 = MODE == 1 ? cur : lo;
  const float *kc = Kc + (int64_t)bg * gm.T * D;
  for (int t0 = s0 + wave * RPW * U; t0 < s1; t0 += 8 * RPW * U) {
    float4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * RPW + sub;
      v[u] = t < s1 ? *reinterpret_cast<const float4 *>(kc + (int64_t)t * D + c4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * RPW + sub;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h >= NH) break;
        float a = fmaf(q[h][0], v[u].x, fmaf(q[h][1], v[u].y, fmaf(q[h][2], v[u].z, q[h][3] * v[u].w)));
        a = key_row_sum<LPR>(a);
        if (lane % LPR == 0 && t < s1) sc[h * gm.T + t] = MODE == 1 ? a : a * gm.scale;
      }
    }
  }
  __syncthreads();
  if (MODE == 1) {
    // per-head log2 normaliser over t < cur: thread-local running (max, sum),
    // merged across the wave by shuffles and across the waves through LDS
    float lse[GM];
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (h >= NH) break;
      float mx = -INFINITY, sm = 0.f;
      for (int t = tid; t < cur; t += 512) {
        const float x = sc[h * gm.T + t];
        if (x > mx) {
          sm = sm * exp2f(mx - x) + 1.f;
          mx = x;
        } else {
          sm += exp2f(x - mx);
        }
      }
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const float om = __shfl_xor(mx, o, 64), os = __shfl_xor(sm, o, 64);
        const float nm = fmaxf(mx, om);
        sm = (sm > 0.f ? sm * exp2f(mx - nm) : 0.f) + (os > 0.f ? os * exp2f(om - nm) : 0.f);
        mx = nm;
      }
      if (lane == 0) {
        red_m[wave][h] = mx;
        red_l[wave][h] = sm;
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (h >= NH) break;
      float M = -INFINITY, L = 0.f;
#pragma unroll
      for (int w = 0; w < 8; ++w) M = fmaxf(M, red_m[w][h]);
#pragma unroll
      for (int w = 0; w < 8; ++w)
        if (red_l[w][h] > 0.f) L += red_l[w][h] * exp2f(red_m[w][h] - M);
      lse[h] = L > 0.f ? M + log2f(L) : 0.f;  // cur = 0 leaves no candidate
    }
    // candidates: the group score replaces head 0's logit in place (one thread per block)
    for (int t = gm.n_init + tid; t < lo; t += 512) {
      float y[GM], ym = -INFINITY;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h >= NH) break;
        y[h] = sc[h * gm.T + t] - lse[h];
        ym = fmaxf(ym, y[h]);
      }
      float e = 0.f;
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        if (h >= NH) break;
        e += exp2f(y[h] - ym);
      }
      sc[t] = ym + log2f(e);
    }
    __syncthreads();
  }

  // Top-k: every wave sorts its 64-candidate chunks best-first across its
  // lanes (bitonic network over shuffles) and keeps the best 64 seen; the
  // eight sorted lists are then merged pairwise through LDS.
  const int nc = max(0, lo - gm.n_init);
  float rs = -INFINITY;
  int rt = 0x7fffffff;
  for (int c0 = wave * 64; c0 < nc; c0 += 8 * 64) {
    float vs = c0 + lane < nc ? sc[gm.n_init + c0 + lane] : -INFINITY;
    int vt = c0 + lane < nc ? gm.n_init + c0 + lane : 0x7fffffff;
    wave_sort_best_first(vs, vt, lane);
    wave_merge_best_first(rs, rt, vs, vt, lane);
  }
  for (int half = 4; half >= 1; half >>= 1) {
    if (wave >= half && wave < 2 * half) {
      mbuf_s[wave - half][lane] = rs;
      mbuf_t[wave - half][lane] = rt;
    }
    __syncthreads();
    if (wave < half) wave_merge_best_first(rs, rt, mbuf_s[wave][lane], mbuf_t[wave][lane], lane);
    __syncthreads();
  }
  if (wave != 0) return;
  const int npick = min(gm.top_k, nc);
  const int mine = rt;  // lanes 0..npick-1 hold the picks, best first
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

// Attention of one decode query over its selected blocks, one workgroup per
// (b, g); wave w takes slots w, w + 4, ....  A block's K and V rows arrive
// with coalesced 16-byte loads, NI per lane (lane = one 16-byte chunk of a key
// row, KPI key rows per load); the CPR lanes of a row reduce its dot products
// (key_row_sum).  Each wave keeps a running (m, l, o) per head (log2 units);
// the four are merged through LDS and O, LSE written directly.
template <typename T, int D, int G>
__global__ __launch_bounds__(256, G >= 8 ? 1 : 2) void decode_attn_kernel(const T *__restrict__ Q, const T *__restrict__ K,
                                                          const T *__restrict__ V, const int32_t *__restrict__ clen,
                                                          const int32_t *__restrict__ sel, T *__restrict__ O,
                                                          float *__restrict__ LSE, Geom gm) {
  constexpr int VEC = 16 / sizeof(T);   // elements per 16-byte chunk
  constexpr int CPR = D / VEC;          // chunks (lanes) per key row
  constexpr int KPI = 64 / CPR;         // key rows per load instruction
  constexpr int NI = (8 * KPI > 64 ? 64 : 8 * KPI) / KPI;    // loads per tensor per key group
  constexpr int KG = NI * KPI;          // keys per group
  __shared__ float wm[4][G], wl[4][G];
  __shared__ float wo[4][G][D];
  const int bg = blockIdx.x, b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ch = lane % CPR, sub = lane / CPR;
  const float sl2 = gm.scale * kLog2e;
  float qv[G][VEC];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const uint4 raw = *reinterpret_cast<const uint4 *>(Q + ((int64_t)b * gm.Hq + g * G + h) * D + ch * VEC);
    const T *pv = reinterpret_cast<const T *>(&raw);
#pragma unroll
    for (int e = 0; e < VEC; ++e) qv[h][e] = to_f32<T>(pv[e]) * sl2;
  }
  float mrun[G], lrun[G], o[G][VEC];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    mrun[h] = -INFINITY;
    lrun[h] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[h][e] = 0.f;
  }
  const int pos = seq_len(clen, b, gm) - 1, cur = pos / gm.m;
  // this wave's slots w, w + 4, ...: lane j holds slot w + 4j (Ksel <= 64), and
  // the valid ones are taken in slot order from a wave-uniform bit mask
  const int sj = wave + 4 * lane;
  const int tl = sj < gm.ksel ? sel[(int64_t)bg * gm.ksel + sj] : -1;
  uint64_t todo = __ballot(tl >= 0 && tl <= cur && tl < gm.T);
  auto load_group = [&](int t, int k0, u32x4 (&kr)[NI], u32x4 (&vr)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int key = min(k0 + i * KPI + sub, gm.m - 1);  // rows past a short block are masked below
      const int64_t src = (((int64_t)b * gm.Lk + (int64_t)t * gm.m + key) * gm.Hkv + g) * D + ch * VEC;
      kr[i] = *reinterpret_cast<const u32x4 *>(K + src);
      vr[i] = *reinterpret_cast<const u32x4 *>(V + src);
    }
  };
  auto attend = [&](int t, int k0, const u32x4 (&kr)[NI], const u32x4 (&vr)[NI]) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float sc[NI];
      float bm = -INFINITY;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const T *pk = reinterpret_cast<const T *>(&kr[i]);
        float a = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) a = fmaf(qv[h][e], to_f32<T>(pk[e]), a);
        a = key_row_sum<CPR>(a);
        const int kb = k0 + i * KPI + sub;
        sc[i] = kb < gm.m && t * gm.m + kb <= pos ? a : -INFINITY;
        bm = fmaxf(bm, sc[i]);
      }
#pragma unroll
      for (int x = CPR; x < 64; x <<= 1) bm = fmaxf(bm, __shfl_xor(bm, x, 64));
      const float mn = fmaxf(mrun[h], bm);
      // mn stays -inf only while every key so far was past the query (a partly
      // written own block): nothing has been accumulated yet
      const float f = mn == -INFINITY ? 1.f : exp2f(mrun[h] - mn);
      float ls = 0.f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[h][e] *= f;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        // keys past the query (the unwritten tail of its own block) add nothing,
        // whatever their V slots hold
        const int kb = k0 + i * KPI + sub;
        const bool valid = kb < gm.m && t * gm.m + kb <= pos;
        const float p = valid ? exp2f(sc[i] - mn) : 0.f;
        ls += p;
        const T *pv = reinterpret_cast<const T *>(&vr[i]);
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[h][e] = valid ? fmaf(p, to_f32<T>(pv[e]), o[h][e]) : o[h][e];
      }
      // ls counts this lane's keys; the CPR lanes of a key row hold the same keys
      lrun[h] = lrun[h] * f + ls;
      mrun[h] = mn;
    }
  };
  for (; todo; todo &= todo - 1) {
    const int t = __builtin_amdgcn_readlane(tl, __builtin_ctzll(todo));
    for (int k0 = 0; k0 < gm.m; k0 += KG) {
      u32x4 kr[NI], vr[NI];  // native vectors: uint4 arrays here would live in scratch
      load_group(t, k0, kr, vr);
      attend(t, k0, kr, vr);
    }
  }
  // reduce over the key-row groups of the wave (lanes with the same chunk)
#pragma unroll
  for (int h = 0; h < G; ++h) {
#pragma unroll
    for (int x = CPR; x < 64; x <<= 1) {
      lrun[h] += __shfl_xor(lrun[h], x, 64);
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[h][e] += __shfl_xor(o[h][e], x, 64);
    }
    if (lane == 0) {
      wm[wave][h] = mrun[h];
      wl[wave][h] = lrun[h];
    }
    if (sub == 0) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) wo[wave][h][ch * VEC + e] = o[h][e];
    }
  }
  __syncthreads();
  for (int x = tid; x < G * D; x += 256) {
    const int h = x / D, c = x - h * D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w][h]);
    float L = 0.f, acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = wm[w][h] == -INFINITY ? 0.f : exp2f(wm[w][h] - M);
      L = fmaf(f, wl[w][h], L);
      acc = fmaf(f, wo[w][h][c], acc);
    }
    O[((int64_t)b * gm.Hq + g * G + h) * D + c] = from_f32<T>(L > 0.f ? acc / L : 0.f);
    if (c == 0) LSE[(int64_t)b * gm.Hq + g * G + h] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  }
}

template <typename T, int D, int G>
static hipError_t launch_decode_g(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc,
                                  const int32_t *clen, int32_t *sel, void *O, float *LSE, hipStream_t s) {
  timing_begin("phsa_decode_select", s);
  if (g.sel_mode == 1)
    hipLaunchKernelGGL((decode_select_kernel<T, D, 1>), dim3(g.B * g.Hkv), dim3(512),
                       (size_t)g.G * g.T * sizeof(float), s, static_cast<const T *>(Q), Kc, clen, sel, g);
  else
    hipLaunchKernelGGL((decode_select_kernel<T, D, 0>), dim3(g.B * g.Hkv), dim3(512), (size_t)g.T * sizeof(float), s,
                       static_cast<const T *>(Q), Kc, clen, sel, g);
  timing_end(s);
  timing_begin("phsa_decode_attn", s);
  hipLaunchKernelGGL((decode_attn_kernel<T, D, G>), dim3(g.B * g.Hkv), dim3(256), 0, s, static_cast<const T *>(Q),
                     static_cast<const T *>(K), static_cast<const T *>(V), clen, sel, static_cast<T *>(O), LSE, g);
  timing_end(s);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_decode_t(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc,
                                  const int32_t *clen, int32_t *sel, void *O, float *LSE, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_decode_g<T, D, 1>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
    case 2: return launch_decode_g<T, D, 2>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
    case 4: return launch_decode_g<T, D, 4>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
    default: return launch_decode_g<T, D, 8>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
  }
}

// ---------------------------------------------------------------- cache append
// One token per sequence joins the cache at position len[b]; the length grows
// by one.  When the token completes block t, that block's representative is
// computed from the cache (Eq. 6-8, the same pooling as phsa_compress) and
// written to K_comp[b, :, t].  One workgroup per sequence; a sequence whose
// cache is full is left unchanged.  Rows move in 16-byte chunks; for the
// pooling, the Hkv*d elements are split into 16-byte chunks and the block's m
// keys into 256 / #chunks slices, whose partial sums meet in LDS.
template <typename T, int D>
__global__ __launch_bounds__(256) void cache_append_kernel(const T *__restrict__ Kn, const T *__restrict__ Vn,
                                                           const uint8_t *__restrict__ pn, T *__restrict__ Kcache,
                                                           T *__restrict__ Vcache, uint8_t *__restrict__ pcache,
                                                           int32_t *__restrict__ clen, float *__restrict__ Kc,
                                                           Geom gm) {
  constexpr int VEC = 16 / sizeof(T);
  __shared__ float red[2][256][VEC];
  __shared__ int npun;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int pos = clen[b];
  if (pos < 0 || pos >= gm.Lk) return;  // full (or invalid): nothing changes
  const int HD = gm.Hkv * D, NCH = HD / VEC;
  for (int x = tid; x < NCH; x += 256) {
    const int64_t dst = ((int64_t)b * gm.Lk + pos) * HD + x * VEC;
    *reinterpret_cast<uint4 *>(Kcache + dst) = *reinterpret_cast<const uint4 *>(Kn + (int64_t)b * HD + x * VEC);
    *reinterpret_cast<uint4 *>(Vcache + dst) = *reinterpret_cast<const uint4 *>(Vn + (int64_t)b * HD + x * VEC);
  }
  if (tid == 0) pcache[(int64_t)b * gm.Lk + pos] = pn[b];
  if ((pos + 1) % gm.m == 0) {
    // the block is complete: pool its m keys (the newest one from the input,
    // the others from the cache, which this launch does not write)
    const int t = pos / gm.m, j0 = t * gm.m;
    if (tid == 0) {
      int c = 0;
      for (int j = j0; j < j0 + gm.m; ++j) c += (j == pos ? pn[b] : pcache[(int64_t)b * gm.Lk + j]) != 0;
      npun = c;
    }
    for (int x0 = 0; x0 < NCH; x0 += 256) {
      const int nch = min(256, NCH - x0);       // chunks handled in this pass
      const int slices = 256 / nch;             // key slices
      const int ch = tid % nch, sl = tid / nch;
      float sum[VEC], psum[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) sum[e] = psum[e] = 0.f;
      if (sl < slices) {
        for (int j = j0 + sl; j < j0 + gm.m; j += slices) {
          const bool newest = j == pos;
          const uint4 raw = newest ? *reinterpret_cast<const uint4 *>(Kn + (int64_t)b * HD + (x0 + ch) * VEC)
                                   : *reinterpret_cast<const uint4 *>(Kcache + ((int64_t)b * gm.Lk + j) * HD +
                                                                      (x0 + ch) * VEC);
          const bool pj = (newest ? pn[b] : pcache[(int64_t)b * gm.Lk + j]) != 0;
          const T *pv = reinterpret_cast<const T *>(&raw);
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const float k = to_f32<T>(pv[e]);
            sum[e] += k;
            psum[e] += pj ? k : 0.f;
          }
        }
      }
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        red[0][tid][e] = sum[e];
        red[1][tid][e] = psum[e];
      }
      __syncthreads();
      if (tid < nch) {
        const int np = npun;
        float rep[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          float s0 = 0.f, s1 = 0.f;
          for (int q = 0; q < slices; ++q) {
            s0 += red[0][q * nch + tid][e];
            s1 += red[1][q * nch + tid][e];
          }
          const float m0 = s0 / (float)gm.m;
          rep[e] = np > 0 ? gm.lambda * m0 + (1.f - gm.lambda) * (s1 / (float)np) : m0;
        }
        const int x = (x0 + tid) * VEC, g = x / D, c = x - g * D;
        float *dst = Kc + (((int64_t)b * gm.Hkv + g) * gm.T + t) * D + c;
#pragma unroll
        for (int e = 0; e < VEC; e += 4) *reinterpret_cast<float4 *>(dst + e) = make_float4(rep[e], rep[e + 1], rep[e + 2], rep[e + 3]);
      }
      __syncthreads();
    }
  }
  __syncthreads();
  if (tid == 0) clen[b] = pos + 1;
}

template <typename T, int D>
static hipError_t launch_cache_append_t(const Geom &g, const void *Kn, const void *Vn, const uint8_t *pn, void *Kcache,
                                        void *Vcache, uint8_t *pcache, int32_t *clen, float *Kc, hipStream_t s) {
  timing_begin("phsa_cache_append", s);
  hipLaunchKernelGGL((cache_append_kernel<T, D>), dim3(g.B), dim3(256), 0, s, static_cast<const T *>(Kn),
                     static_cast<const T *>(Vn), pn, static_cast<T *>(Kcache), static_cast<T *>(Vcache), pcache, clen,
                     Kc, g);
  timing_end(s);
  return hipGetLastError();
}

hipError_t launch_cache_append(const Geom &g, const void *Kn, const void *Vn, const uint8_t *pn, void *Kcache,
                               void *Vcache, uint8_t *pcache, int32_t *clen, float *Kc, hipStream_t s) {
  if (g.dtype == 0)
    return g.d == 128 ? launch_cache_append_t<bf16_t, 128>(g, Kn, Vn, pn, Kcache, Vcache, pcache, clen, Kc, s)
                      : launch_cache_append_t<bf16_t, 64>(g, Kn, Vn, pn, Kcache, Vcache, pcache, clen, Kc, s);
  return g.d == 128 ? launch_cache_append_t<float, 128>(g, Kn, Vn, pn, Kcache, Vcache, pcache, clen, Kc, s)
                    : launch_cache_append_t<float, 64>(g, Kn, Vn, pn, Kcache, Vcache, pcache, clen, Kc, s);
}

hipError_t launch_decode(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc,
                         const int32_t *clen, int32_t *sel, void *O, float *LSE, hipStream_t s) {
  if (g.dtype == 0)
    return g.d == 128 ? launch_decode_t<bf16_t, 128>(g, Q, K, V, Kc, clen, sel, O, LSE, s)
                      : launch_decode_t<bf16_t, 64>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
  return g.d == 128 ? launch_decode_t<float, 128>(g, Q, K, V, Kc, clen, sel, O, LSE, s)
                    : launch_decode_t<float, 64>(g, Q, K, V, Kc, clen, sel, O, LSE, s);
}

}  // namespace phsa

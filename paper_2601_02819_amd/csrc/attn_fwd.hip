// Sparse attention forward, bf16 (Eq. 10-11; Algorithm 1 attention step).
//
// Work is key-block-major.  Every query row selects its own blocks, so the
// only operand that many rows share is a key/value block.  A workgroup takes
// one work unit = one (b, g, t) block plus up to unit_tokens entries of the
// list of rows that selected it and keeps K_t and V_t in LDS.  Each wave then
// works through the unit on its own, in wave chunks of 16 MFMA rows (16 / G
// tokens x the G heads of the group), chunks w, w + 4, ...:
//
//   S^T = K_t Q^T                      (64 keys x 16 rows, 16x16x32 bf16 MFMA)
//   m = rowmax, P = 2^(S - m), l = rowsum(P)      (token-level causal mask)
//   O^T = V_t^T P^T                    (d x 16 rows)
//
// The gathered query rows go straight from global memory into registers in
// the B-operand layout of S^T (lane (q, j) holds features 32kb + 8q .. +7 of
// row j), so there is no shared query tile and no barrier after the K/V
// load; each wave fetches its next chunk's rows while it computes the current
// one, with the list entries read one chunk further ahead.  The S^T
// accumulator layout (lane (q, j) holds keys 4q + r of row j) is used directly
// as the P^T operand of the second product, pairing key tiles {4q..4q+3} and
// {16+4q..16+4q+3}; V_t^T is read with transposing LDS loads over the same
// key set, so P never goes through LDS.  O^T leaves each lane with 4
// consecutive features of one row; a wave stages its 16 rows in LDS and
// stores them as full 16-byte lanes, with non-temporal stores (only the merge
// reads them, so they should not displace the rows and tiles the kernel reuses).
//
// Blocks of 16 or 32 tokens run on the same 64-key tiles: each list entry
// carries the mask of the 16-key quarters its row selected, and keys of the
// other quarters get zero weight (key tile kt of S^T is quarter kt).
//
// Output per list entry (row, slot), stored in list order so that a unit
// writes one contiguous run: the unnormalised partial O (bf16) and (m, l) in
// log2 units.  A second kernel merges the at most Ksel partials of each row:
//   M = max_s m_s,  w_s = 2^(m_s - M),  O = sum_s w_s O_s / sum_s w_s l_s,
//   LSE = (M + log2 sum_s w_s l_s) ln 2
// (computed with a running maximum in slot order).
#include <math.h>

#include "common.h"
#include "launch.h"

namespace phsa {

template <int D, int G>
__global__ __launch_bounds__(256, 3) void attn_fwd_sparse_kernel(const bf16_t *__restrict__ Q,
                                                              const bf16_t *__restrict__ K,
                                                              const bf16_t *__restrict__ V, Geom gm, IndexWs ix,
                                                              bf16_t *__restrict__ opart, float2 *__restrict__ ml) {
  constexpr int TW = 16 / G;         // query tokens per wave chunk
  constexpr int KP = D + 16;         // K pitch: 16-byte row reads of 16 rows are conflict-free at D + 16
  constexpr int VPR = D / 8;         // 16-byte vectors per row
  constexpr int KB = D / 32;
  constexpr int NT = D / 16;
  constexpr int SP = D + 8;          // pitch of the per-wave output staging rows
  __shared__ __attribute__((aligned(16))) bf16_t Ks[64 * KP];
  // V is read by transposing reads only; it is stored without padding in the
  // swizzled layout of swz() (with D + 8 padding those reads conflict, and D + 16
  // would not leave three workgroups per CU)
  __shared__ __attribute__((aligned(16))) bf16_t Vs[64 * D];
  __shared__ __attribute__((aligned(16))) bf16_t Os[4][16 * SP];  // per-wave partial rows

  const int u = blockIdx.x;
  if (u >= ix.totals[1]) return;
  const int2 unit = ix.units[u];
  const int bgt = unit.x, e0 = unit.y;
  const int n_ent = min(ix.cnt[bgt] - e0, ix.unit_tokens);
  const int bg = bgt / gm.T, t = bgt - bg * gm.T;
  const int b = bg / gm.Hkv, g = bg - b * gm.Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4, kq = q4 * 8;
  // list position of the unit's first entry, read once (a load inside the chunk loop
  // would make the wait for it also wait for the prefetched rows)
  const int64_t list0 = (int64_t)ix.off[bgt] + e0;
  const int32_t *list = ix.tok + list0;

  for (int x = tid; x < 64 * VPR; x += 256) {
    const int kk = x / VPR, c = (x % VPR) * 8;
    const int64_t grow = ((int64_t)b * gm.Lk + (int64_t)t * 64 + kk) * gm.Hkv + g;
    *reinterpret_cast<uint4 *>(&Ks[kk * KP + c]) = *reinterpret_cast<const uint4 *>(K + grow * D + c);
    *reinterpret_cast<uint4 *>(&Vs[swz<D>(kk, c)]) = *reinterpret_cast<const uint4 *>(V + grow * D + c);
  }
  __syncthreads();

  // lane (q, j) works on row j = l16 of the wave chunk: token j / G, head j % G
  const int hh = l16 % G;
  const int nch = (n_ent + TW - 1) / TW;
  // Loads are issued unconditionally (rows past the list read its last entry,
  // or query row 0): their results are masked, and a fixed number of loads per
  // chunk lets the compiler wait for exactly the ones a chunk needs.
  auto entry = [&](int c) {
    const int tk = c * TW + l16 / G;
    const int v = list[min(tk, n_ent - 1)];
    return tk < n_ent ? v : -1;
  };
  auto fetch = [&](int e, bf16x8 (&qf)[KB]) {
    const int64_t row = e >= 0 ? (e >> 10) : 0;  // an empty chunk row is masked to zero weight
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      qf[kb] = load_bf16x8(Q + (((int64_t)b * gm.Lq + row) * gm.Hq + g * G + hh) * D + kb * 32 + kq);
  };

  const float sl2 = gm.scale * kLog2e;
  const int key0 = t * 64;
  // rows of discarded stores (past a chunk's end): one spare partial row
  const int64_t discard = ix.discard;

  // one wave chunk: rows of list entry e (-1: none) with query fragments q
  auto chunk = [&](int c, int e, const bf16x8 (&q)[KB]) {
    f32x4 st[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
        st[kt] = mfma16x16x32(load_bf16x8(&Ks[(kt * 16 + l16) * KP + kb * 32 + kq]), q[kb], st[kt]);
    // key tile kt is quarter kt of the block: allowed if the row selected it
    const int pos = e >= 0 ? gm.q_pos0 + (e >> 10) : -1;
    const int qm = e >= 0 ? (e >> 6) & 15 : 0;
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool ok = ((qm >> kt) & 1) && (key0 + kt * 16 + q4 * 4 + r) <= pos;
        const float v = ok ? st[kt][r] * sl2 : -INFINITY;
        st[kt][r] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (mx == -INFINITY) mx = 0.f;
    float l = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = __builtin_amdgcn_exp2f(st[kt][r] - mx);
        st[kt][r] = p;
        l += p;
      }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    const bf16x8 pb0 = pack_bf16x8(st[0], st[1]);  // keys {4q..4q+3} and {16+4q..16+4q+3}
    const bf16x8 pb1 = pack_bf16x8(st[2], st[3]);  // keys 32 + the same

    f32x4 ot[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      ot[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      ot[nt] = mfma16x16x32(lds_col8_sw<D>(Vs, q4 * 4, 16 + q4 * 4, nt * 16, l16), pb0, ot[nt]);
      ot[nt] = mfma16x16x32(lds_col8_sw<D>(Vs, 32 + q4 * 4, 48 + q4 * 4, nt * 16, l16), pb1, ot[nt]);
    }
    // The chunk's 16 partial rows are one contiguous run of the list-ordered
    // partial buffer (entries c*TW.., heads inner): stage them in LDS and write
    // full 16-byte lanes.  Every lane stores (unused lanes to the discard row),
    // so a chunk issues a fixed number of stores and the waits for the
    // prefetched rows need not wait for them.
    const int64_t run0 = list0 + c * TW;  // list position of the chunk's first entry
    st_stream_f2(&ml[e >= 0 && q4 == 0 ? (run0 + l16 / G) * G + hh : discard], mx, l);
    bf16_t *os = Os[wave];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16_t o4[4] = {f32_to_bf16(ot[nt][0]), f32_to_bf16(ot[nt][1]), f32_to_bf16(ot[nt][2]),
                            f32_to_bf16(ot[nt][3])};
      *reinterpret_cast<uint2 *>(&os[l16 * SP + nt * 16 + q4 * 4]) = *reinterpret_cast<const uint2 *>(o4);
    }
    wave_lds_sync();
    const int nrows = min(TW, n_ent - c * TW) * G;  // valid rows of this chunk
#pragma unroll
    for (int k = 0; k < 16 * D / 8 / 64; ++k) {
      const int v = lane + 64 * k, r = v / (D / 8), cc = (v % (D / 8)) * 8;
      const int64_t row = r < nrows ? run0 * G + r : discard;
      st_stream16(opart + row * D + cc, &os[r * SP + cc]);
    }
    wave_lds_sync();
  };

  // Two register sets alternate: while one chunk computes, the next one's rows
  // are in flight in the other set and the entries of the one after that too.
  int e_a = entry(wave), e_b = entry(wave + 4);
  bf16x8 qa[KB], qb[KB];
  fetch(e_a, qa);
  for (int c = wave; c < nch; c += 8) {
    int e_n = entry(c + 8);
    fetch(e_b, qb);
    chunk(c, e_a, qa);
    if (c + 4 >= nch) break;
    e_a = e_n;
    e_n = entry(c + 12);
    fetch(e_a, qa);
    chunk(c + 4, e_b, qb);
    e_b = e_n;
  }
}

// Merge of a row's per-slot partials.  Half a wave per (b, g, query row), 8
// features per lane (16-byte loads).  The row's list positions come in one
// load spread over the lanes (RowSlots); the partials and their (m, l) of up
// to 16 slots are then loaded together and folded in slot order with a
// running maximum, so a row costs two dependent global loads.
template <int D, int G>
__global__ __launch_bounds__(256) void attn_fwd_combine_kernel(const int32_t *__restrict__ pmap,
                                                               const bf16_t *__restrict__ opart,
                                                               const float2 *__restrict__ ml, bf16_t *__restrict__ O,
                                                               float *__restrict__ LSE, Geom gm) {
  constexpr int U = 16;  // slots whose partials are in flight together
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int64_t x = ((int64_t)blockIdx.x * 4 + wave) * 2 + half;  // bg * Lq + i
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
    // online merge in slot order: running max M (log2 units), sum L, sum a
    float M = -INFINITY, L = 0.f, a[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) a[k] = 0.f;
    for (int s0 = 0; s0 < ns; s0 += U) {
      float2 q[U];
      uint4 raw[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int s = s0 + k;
        const int p = s < ns ? rs.pos(s, half) : -1;
        const bool ok = act && p >= 0;
        q[k] = ok ? ml[(int64_t)p * G + hh] : make_float2(-INFINITY, 0.f);
        raw[k] = ok ? ld_stream16(opart + ((int64_t)p * G + hh) * D + c) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if (q[k].x == -INFINITY) continue;
        const float mn = fmaxf(M, q[k].x);
        const float sc = __builtin_amdgcn_exp2f(M - mn), w = __builtin_amdgcn_exp2f(q[k].x - mn);
        L = fmaf(w, q[k].y, L * sc);
        const bf16_t *pv = reinterpret_cast<const bf16_t *>(&raw[k]);
#pragma unroll
        for (int j = 0; j < 8; ++j) a[j] = fmaf(w, bf16_to_f32(pv[j]), a[j] * sc);
        M = mn;
      }
    }
    if (!row_ok || !act) continue;
    const float inv = L > 0.f ? 1.f / L : 0.f;
    bf16_t outv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) outv[k] = f32_to_bf16(a[k] * inv);
    *reinterpret_cast<uint4 *>(O + (((int64_t)b * gm.Lq + i) * gm.Hq + g * G + hh) * D + c) =
        *reinterpret_cast<const uint4 *>(outv);
    if (c == 0) LSE[((int64_t)b * gm.Hq + g * G + hh) * gm.Lq + i] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
  }
}

template <int D, int G>
static hipError_t launch_fwd_t(const Geom &g, const void *Q, const void *K, const void *V, void *O, float *LSE,
                               const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  timing_begin("phsa_attn_fwd_sparse", s);
  hipLaunchKernelGGL((attn_fwd_sparse_kernel<D, G>), dim3((unsigned)ix.units_max), dim3(256), 0, s,
                     static_cast<const bf16_t *>(Q), static_cast<const bf16_t *>(K), static_cast<const bf16_t *>(V),
                     g, ix, static_cast<bf16_t *>(opart), ml);
  timing_end(s);
  if (g.band) {  // the band kernel runs after the sparse one and merges every row itself
    const hipError_t e = launch_fwd_band(g, Q, K, V, ix, opart, ml, O, LSE, s);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  const int64_t rows = (int64_t)g.B * g.Hkv * g.Lq;
  timing_begin("phsa_attn_fwd_combine", s);
  hipLaunchKernelGGL((attn_fwd_combine_kernel<D, G>), dim3((unsigned)((rows + 7) / 8)), dim3(256), 0, s, ix.pmap,
                     static_cast<const bf16_t *>(opart), ml, static_cast<bf16_t *>(O), LSE, g);
  timing_end(s);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_fwd_d(const Geom &g, const void *Q, const void *K, const void *V, void *O, float *LSE,
                               const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  switch (g.G) {
    case 1: return launch_fwd_t<D, 1>(g, Q, K, V, O, LSE, ix, opart, ml, s);
    case 2: return launch_fwd_t<D, 2>(g, Q, K, V, O, LSE, ix, opart, ml, s);
    case 4: return launch_fwd_t<D, 4>(g, Q, K, V, O, LSE, ix, opart, ml, s);
    default: return launch_fwd_t<D, 8>(g, Q, K, V, O, LSE, ix, opart, ml, s);
  }
}

hipError_t launch_attn_fwd(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel, void *O,
                           float *LSE, const IndexWs &ix, void *opart, float2 *ml, hipStream_t s) {
  hipError_t e = launch_build_index(g, sel, ix, s);
  if (e != hipSuccess) return e;
  return g.d == 128 ? launch_fwd_d<128>(g, Q, K, V, O, LSE, ix, opart, ml, s)
                    : launch_fwd_d<64>(g, Q, K, V, O, LSE, ix, opart, ml, s);
}

}  // namespace phsa

// Internal launchers: one per kernel family.  The C ABI (api.hip) validates
// every argument before calling any of these; launchers only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "phsa.h"

namespace phsa {

// Geometry resolved once by the ABI layer.
struct Geom {
  int B, Lq, Lk, Hq, Hkv, G, d, m, T;
  int top_k, n_init, window, ksel;
  int q_pos0;         // position of query row 0 = Lk - Lq
  float lambda;
  float scale;        // softmax scale
  int dtype;          // 0 bf16, 1 fp32
  int sel_mode;       // group aggregation of block scores: 0 summed logits, 1 summed per-head softmax
  int sm;             // block size of the selection (m of a tile geometry is 64; n_init, window keep sm units)
  int band;           // 1: the local window of every row holding it whole is attended by the band kernels
};

// Index (inverted selection) workspace, carved out of the caller's buffer.
struct IndexWs {
  int W;              // query tiles of kIndexTile rows
  int unit_tokens;    // list entries per attention work unit
  int64_t units_max;  // upper bound on the number of work units
  int64_t nnz_max;    // upper bound on list entries
  int32_t *cntw;      // [B*Hkv, W, T]  per-tile counts, then per-tile list offsets
  int32_t *cnt;       // [B*Hkv*T]      list length per (b, g, t)
  int32_t *off;       // [B*Hkv*T + 1]  list start per (b, g, t)
  int32_t *uoff;      // [B*Hkv*T + 1]  first work unit per (b, g, t)
  int32_t *totals;    // [4]            nnz, n_units, blocks in fin
  int4 *wsum;         // [ceil(B*Hkv*T / 256)] per 256 (b, g, t): sums of list lengths, units and
                      //                 finalize flags, then their exclusive offsets
  int32_t *fin;       // [B*Hkv*T]      the (b, g, t) whose dK/dV the finalize writes (not one work unit)
  int32_t *tok;       // [nnz_max]      (query row << 10) | (quarter mask << 6) | slot, ascending row per list
  int32_t *pmap;      // [B*Hkv*Lq*Ksel] list position of each valid (row, slot); partials are
                      //                 stored in list order and the merges gather through this map
  int2 *units;        // [units_max]    (b*Hkv*T + g*T + t, first list entry)
  int64_t band_base;  // list position of the band partial of row (b, g, i): band_base + (b*Hkv + g)*Lq + i
  int64_t discard;    // partial row that absorbs stores past a chunk's end (after the list and band rows)
  uint8_t *bflag;     // [B*Hkv*Lq] 1: the row's forced blocks are in the band (NULL: no band)
};

constexpr int kIndexTile = 256;  // query rows per index-building workgroup

// Host validation of the C ABI's parameters for an operation (api.hip); fills
// the resolved geometry when out is not NULL.
phsa_status validate(const phsa_params *p, int op, Geom *out);

// Hooks around every kernel launch, given the kernel's profiling name.  The
// library defines them empty (api.hip); the profiling build links definitions
// that bracket the launch with HIP events on its stream (prof/kernel_timing.hip).
void timing_begin(const char *name, hipStream_t s);
void timing_end(hipStream_t s);

hipError_t launch_punct_mask(const int32_t *ids, int64_t n, const int32_t *pset, int n_punct, uint8_t *mask,
                             hipStream_t s);
hipError_t launch_compress(const Geom &g, const void *K, const uint8_t *punct, float *Kc, hipStream_t s);
// ws: select_split_bytes(g) bytes (bf16 hi/lo copies of K_comp), unused for float32
size_t select_split_bytes(const Geom &g);
hipError_t launch_select(const Geom &g, const void *Q, const float *Kc, int32_t *sel, void *ws, hipStream_t s);
// g: the index's geometry (the tile geometry of m-token blocks); sel is the
// selection as phsa_select writes it (its own block size and Ksel)
hipError_t launch_build_index(const Geom &g, const int32_t *sel, const IndexWs &ix, hipStream_t s);
hipError_t launch_attn_fwd(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel, void *O,
                           float *LSE, const IndexWs &ix, void *opart, float2 *ml, hipStream_t s);
// bkv: with g.band, float32 [B*Hkv*T][2][64][d] for the band's dK, dV per 64-key tile;
// seg_sums: the init tiles' per-segment sums, in the sparse dK/dV partial buffer (dead until the sparse kernel)
hipError_t launch_attn_bwd(const Geom &g, const void *Q, const void *K, const void *V, const void *O,
                           const void *dO, const float *LSE, const int32_t *sel, void *dQ,
                           void *dK, void *dV, const IndexWs &ix, float *Dvec, void *dqpart, float *dkvpart,
                           float *bkv, bool reuse_index, hipStream_t s);
// band kernels (attn_band.hip): local windows as dense query-major / key-major attention
// the forward band kernel runs after the sparse forward and merges every row
// (the sparse partials, then its own band partial) into O and LSE
hipError_t launch_fwd_band(const Geom &g, const void *Q, const void *K, const void *V, const IndexWs &ix,
                           const void *opart, const float2 *ml, void *O, float *LSE, hipStream_t s);
// the band's dK/dV tiles (before the sparse backward, whose epilogue adds them)
hipError_t launch_bwd_band_dkv(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                               const float *LSE, const float *Dvec, const IndexWs &ix, float *bkv, float *seg_sums,
                               hipStream_t s);
// the band's dQ (after the sparse backward): merges every row's sparse dQ
// partials and its band dQ into dQ
hipError_t launch_bwd_band_dq(const Geom &g, const void *Q, const void *K, const void *V, const void *dO,
                              const float *LSE, const float *Dvec, const IndexWs &ix, const void *dqpart, void *dQ,
                              hipStream_t s);
hipError_t launch_bwd_pre(const Geom &g, const void *O, const void *dO, float *Dvec, hipStream_t s);
hipError_t launch_attn_fwd_fp32(const Geom &g, const float *Q, const float *K, const float *V,
                                const int32_t *sel, float *O, float *LSE, hipStream_t s);
hipError_t launch_attn_bwd_fp32(const Geom &g, const float *Q, const float *K, const float *V,
                                const float *O, const float *dO, const float *LSE, const int32_t *sel,
                                float *dQ, float *dK, float *dV, float *Dvec, hipStream_t s);
hipError_t launch_decode(const Geom &g, const void *Q, const void *K, const void *V, const float *Kc,
                         const int32_t *clen, int32_t *sel, void *O, float *LSE, hipStream_t s);
hipError_t launch_cache_append(const Geom &g, const void *Kn, const void *Vn, const uint8_t *pn, void *Kcache,
                               void *Vcache, uint8_t *pcache, int32_t *clen, float *Kc, hipStream_t s);

}  // namespace phsa

// C ABI of libphsa: host-side validation, workspace layout and dispatch.
// Nothing here allocates device memory; every kernel goes on the caller's stream.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <exception>

#include "phsa.h"
#include "launch.h"

namespace phsa {

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Carves the inverted-index workspace starting at `base` (NULL = size only).
size_t index_layout(const Geom &g, char *base, IndexWs *ix) {
  IndexWs w{};
  const int64_t R = (int64_t)g.B * g.Hkv;
  const int64_t nbgt = R * g.T;
  w.W = (g.Lq + kIndexTile - 1) / kIndexTile;
  w.unit_tokens = 64 * (64 / g.G);  // 64 chunks of 64 MFMA rows
  w.nnz_max = R * g.Lq * (g.ksel - g.band);  // a band geometry keeps one slot per row for the band partial
  w.band_base = w.nnz_max;
  w.discard = (w.nnz_max + (g.band ? R * g.Lq : 0)) * g.G;
  w.units_max = nbgt + (w.nnz_max + w.unit_tokens - 1) / w.unit_tokens;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char *p = base ? base + off : nullptr;
    off += align_up(bytes);
    return p;
  };
  w.cntw = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * R * w.W * g.T));
  w.cnt = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * nbgt));
  w.off = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (nbgt + 1)));
  w.uoff = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (nbgt + 1)));
  w.totals = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * 4));
  w.wsum = reinterpret_cast<int4 *>(take(sizeof(int4) * ((nbgt + 255) / 256)));
  w.fin = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * nbgt));
  w.tok = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * w.nnz_max));
  w.pmap = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * R * g.Lq * g.ksel));  // every slot, band slot too
  w.units = reinterpret_cast<int2 *>(take(sizeof(int2) * w.units_max));
  if (ix) *ix = w;
  return off;
}

// bf16 attention with a local window of at least one 64-key tile attends to
// every row's forced blocks (init blocks and local window, Algorithm 1) with
// the band kernels (dense, query-major for O and dQ, key-major for dK/dV) and
// to its other selected blocks with the sparse ones.  Without a window a row
// has two forced tiles (block 0 and its own), too few for the band kernels'
// per-workgroup cost: at 4 x 32k with 64-token blocks the band took the step
// from 11.47 to 12.02 ms, so those forced blocks stay in the sparse kernels.
bool band_on(const Geom &g) {
  return g.dtype == PHSA_BF16 && g.window >= 64 && g.Lk % 64 == 0 && std::min(g.ksel, g.Lk / 64) <= 63;
}

// bf16 attention with blocks of m = 16 or 32 tokens, or with the band, runs
// on a regrouped selection: 64-key tiles with a mask of their 16-key quarters.
bool tiles_coarsened(const Geom &g) { return g.dtype == PHSA_BF16 && (g.m != 64 || band_on(g)); }

// Tile geometry: m = 64, T = Lk / 64, and ksel = the most distinct tiles a
// row can hold, min(Ksel, T), plus the band slot.  (A selection made by
// phsa_select needs fewer: ceil(n_init m / 64) init tiles, at most
// ceil(w / 64) + 1 local ones and one per pick, 27 against Ksel = 57 in the
// paper's geometry; but sel may be any ascending causal block list.)  n_init
// and window stay in units of the selection's blocks (sm).
Geom tile_geom(const Geom &g) {
  if (!tiles_coarsened(g)) return g;
  Geom t = g;
  t.band = band_on(g) ? 1 : 0;
  t.m = 64;
  t.T = g.Lk / 64;
  t.ksel = std::min(g.ksel, t.T) + t.band;
  return t;
}

struct Coarse {
  Geom gc;            // tile geometry (== g when not coarsened)
  uint8_t *bflag;     // [B, Hkv, Lq] rows whose local window is in the band (band geometry only)
};

// The band flags sit at the start of the forward and backward workspaces,
// followed by the index, so a backward that reuses the forward's index finds
// them at the same place.  The index builder regroups sel into tiles as it
// reads it; no regrouped copy is stored.
size_t coarse_layout(const Geom &g, char *base, Coarse *c) {
  Coarse w{tile_geom(g), nullptr};
  size_t off = 0;
  if (w.gc.band) {
    w.bflag = base ? reinterpret_cast<uint8_t *>(base) : nullptr;
    off += align_up((size_t)g.B * g.Hkv * g.Lq);
  }
  if (c) *c = w;
  return off;
}

struct FwdWs {
  Coarse co;
  IndexWs ix;
  void *opart;
  float2 *ml;
};
struct BwdWs {
  Coarse co;
  IndexWs ix;
  float *Dvec;
  void *dqpart;
  float *dkvpart;
  float *bkv;         // band geometry: the band's dK/dV per 64-key tile, float32 [B*Hkv*T][2][64][d]
};

size_t elem_bytes(const Geom &g) { return g.dtype == PHSA_BF16 ? 2 : 4; }

size_t fwd_layout(const Geom &g0, char *base, FwdWs *ws) {
  if (g0.dtype == PHSA_FP32) return 0;
  FwdWs w{};
  size_t off = coarse_layout(g0, base, &w.co);
  const Geom &g = w.co.gc;
  off += index_layout(g, base ? base + off : nullptr, &w.ix);
  w.ix.bflag = w.co.bflag;
  // partials in list order, one per (entry, head), then the band partials (a
  // band geometry), then one discard row that absorbs the stores of rows past
  // the end of a chunk
  const int64_t slots = w.ix.discard + 1;
  w.opart = base ? base + off : nullptr;
  off += align_up(slots * g.d * elem_bytes(g));
  w.ml = base ? reinterpret_cast<float2 *>(base + off) : nullptr;
  off += align_up(slots * sizeof(float2));
  if (ws) *ws = w;
  return off;
}

size_t bwd_layout(const Geom &g0, char *base, BwdWs *ws) {
  BwdWs w{};
  w.co = Coarse{tile_geom(g0), nullptr};
  const Geom g = w.co.gc;
  size_t off = 0;
  if (g.dtype == PHSA_BF16) {
    off = coarse_layout(g0, base, &w.co);
    off += index_layout(g, base ? base + off : nullptr, &w.ix);
    w.ix.bflag = w.co.bflag;
  }
  w.Dvec = base ? reinterpret_cast<float *>(base + off) : nullptr;
  off += align_up(sizeof(float) * (size_t)g.B * g.Hq * g.Lq);
  if (g.dtype == PHSA_BF16) {
    const int64_t slots = w.ix.discard + 1;  // list and band partials + the discard row
    w.dqpart = base ? base + off : nullptr;
    off += align_up(slots * g.d * elem_bytes(g));
    w.dkvpart = base ? reinterpret_cast<float *>(base + off) : nullptr;
    off += align_up(sizeof(float) * (size_t)w.ix.units_max * 2 * 64 * g.d);
    if (g.band) {
      w.bkv = base ? reinterpret_cast<float *>(base + off) : nullptr;
      off += align_up(sizeof(float) * (size_t)g.B * g.Hkv * g.T * 2 * 64 * g.d);
    }
  }
  if (ws) *ws = w;
  return off;
}

size_t decode_layout(const Geom &) { return 0; }  // the decode kernels need no scratch

}  // namespace

// bf16 selection scratch, as launch_select carves it: K_comp split into bf16 hi
// and lo [B, Hkv, T, d] each, then the norms of both parts per block (float2).
size_t select_split_bytes(const Geom &g) {
  const size_t nblk = (size_t)g.B * g.Hkv * g.T;
  return g.dtype == PHSA_BF16 ? nblk * (2 * g.d * sizeof(uint16_t) + 2 * sizeof(float)) : 0;
}

namespace {

bool is_attention_op(int op) {
  return op == PHSA_OP_ATTN_FWD || op == PHSA_OP_ATTN_BWD || op == PHSA_OP_FORWARD || op == PHSA_OP_DECODE;
}

}  // namespace

// Host validation of p for op (shared with the scratch-free entry point).
phsa_status validate(const phsa_params *p, int op, Geom *out) {
  if (!p) return PHSA_ERR_NULL;
  if (op < PHSA_OP_COMPRESS || op > PHSA_OP_DECODE) return PHSA_ERR_INVALID_ARG;
  if (p->dtype != PHSA_BF16 && p->dtype != PHSA_FP32) return PHSA_ERR_DTYPE;
  if (p->batch < 1 || p->seqlen_q < 1 || p->seqlen_k < 1 || p->n_heads_q < 1 || p->n_heads_kv < 1 ||
      p->head_dim < 1 || p->block_size < 1)
    return PHSA_ERR_SHAPE;
  if (p->n_heads_q % p->n_heads_kv != 0) return PHSA_ERR_SHAPE;
  if (p->seqlen_k % p->block_size != 0) return PHSA_ERR_SHAPE;
  if (p->seqlen_q > p->seqlen_k) return PHSA_ERR_SHAPE;
  if (op == PHSA_OP_DECODE && p->seqlen_q != 1) return PHSA_ERR_SHAPE;
  if (p->top_k < 0 || p->n_init_blocks < 0 || p->window < 0 || p->window % p->block_size != 0)
    return PHSA_ERR_INVALID_ARG;
  if ((p->flags & ~(PHSA_FLAG_REUSE_INDEX | PHSA_FLAG_SELECT_SOFTMAX_SUM)) != 0) return PHSA_ERR_INVALID_ARG;
  if (!(p->lambda >= 0.f && p->lambda <= 1.f)) return PHSA_ERR_INVALID_ARG;
  if (!isfinite(p->softmax_scale)) return PHSA_ERR_INVALID_ARG;
  // What the kernels implement.
  if (p->head_dim != 64 && p->head_dim != 128) return PHSA_ERR_UNSUPPORTED;
  const int64_t T = p->seqlen_k / p->block_size;
  const int64_t ksel = (int64_t)p->n_init_blocks + p->window / p->block_size + 1 + p->top_k;
  const int G = p->n_heads_q / p->n_heads_kv;
  if (ksel > 64 || p->top_k > 32) return PHSA_ERR_UNSUPPORTED;
  if (T > 2048 || p->seqlen_q >= (1 << 25)) return PHSA_ERR_UNSUPPORTED;
  // bf16 attention on blocks below 64 tokens runs on 64-key tiles (quarter masks)
  const bool coarse = p->dtype == PHSA_BF16 && p->block_size != 64;
  const int64_t ksel_tiles = coarse ? std::min<int64_t>(ksel, p->seqlen_k / 64) : ksel;
  if (p->batch > 65535 || p->n_heads_q > 65535 || (int64_t)p->batch * p->n_heads_kv > 65535)
    return PHSA_ERR_UNSUPPORTED;  // grid y/z extents
  // the softmax-sum kernels give each lane one (row, head) pair, at most 8 heads in decode
  if ((p->flags & PHSA_FLAG_SELECT_SOFTMAX_SUM) && (G > 64 || 64 % G != 0)) return PHSA_ERR_UNSUPPORTED;
  if (is_attention_op(op)) {
    if (p->block_size != 64 && p->block_size != 32 && p->block_size != 16) return PHSA_ERR_UNSUPPORTED;
    if (G != 1 && G != 2 && G != 4 && G != 8) return PHSA_ERR_UNSUPPORTED;
    if (p->seqlen_q >= (1 << 21)) return PHSA_ERR_UNSUPPORTED;  // index entries hold the row in 21 bits
    // the 64-key tiles of m-token blocks must not run past the keys
    if (coarse && op != PHSA_OP_DECODE && p->seqlen_k % 64 != 0) return PHSA_ERR_UNSUPPORTED;
    const int64_t nnz = (int64_t)p->batch * p->n_heads_kv * p->seqlen_q * ksel_tiles;
    if (nnz >= ((int64_t)1 << 31) / 2) return PHSA_ERR_UNSUPPORTED;
  }
  if (out) {
    Geom g{};
    g.B = p->batch;
    g.Lq = p->seqlen_q;
    g.Lk = p->seqlen_k;
    g.Hq = p->n_heads_q;
    g.Hkv = p->n_heads_kv;
    g.G = G;
    g.d = p->head_dim;
    g.m = p->block_size;
    g.T = (int)T;
    g.top_k = p->top_k;
    g.n_init = p->n_init_blocks;
    g.window = p->window;
    g.ksel = (int)ksel;
    g.q_pos0 = p->seqlen_k - p->seqlen_q;
    g.lambda = p->lambda;
    g.scale = p->softmax_scale > 0.f ? p->softmax_scale : 1.f / sqrtf((float)p->head_dim);
    g.dtype = p->dtype;
    g.sel_mode = (p->flags & PHSA_FLAG_SELECT_SOFTMAX_SUM) ? 1 : 0;
    g.sm = g.m;
    g.band = 0;
    *out = g;
  }
  return PHSA_OK;
}

namespace {

size_t workspace_bytes(const Geom &g, int op) {
  switch (op) {
    case PHSA_OP_SELECT: return align_up(select_split_bytes(g));
    case PHSA_OP_ATTN_FWD: return fwd_layout(g, nullptr, nullptr);
    // the selection scratch is dead before the attention step reuses the same bytes
    case PHSA_OP_FORWARD: return std::max(fwd_layout(g, nullptr, nullptr), align_up(select_split_bytes(g)));
    case PHSA_OP_ATTN_BWD: return bwd_layout(g, nullptr, nullptr);
    case PHSA_OP_DECODE: return decode_layout(g);
    default: return 0;
  }
}

phsa_status check_ws(const Geom &g, int op, const void *ws, size_t ws_bytes) {
  const size_t need = workspace_bytes(g, op);
  if (need == 0) return PHSA_OK;
  if (!ws || ws_bytes < need) return PHSA_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return PHSA_ERR_WORKSPACE;
  return PHSA_OK;
}

phsa_status from_hip(hipError_t e) { return e == hipSuccess ? PHSA_OK : PHSA_ERR_HIP; }

// bf16 forward attention over sel: index (on 64-key tiles when m < 64 or with
// the band), sparse kernel, band kernel and merge.
hipError_t attn_fwd_bf16(const Geom &g, const void *Q, const void *K, const void *V, const int32_t *sel, void *O,
                         float *LSE, void *ws, hipStream_t s) {
  FwdWs w;
  fwd_layout(g, static_cast<char *>(ws), &w);
  return launch_attn_fwd(w.co.gc, Q, K, V, sel, O, LSE, w.ix, w.opart, w.ml, s);
}

}  // namespace

// Launch hooks around every kernel (launch.h).  This library defines them
// empty and keeps no state; the profiling build (libphsa_prof.so, see
// include/phsa_prof.h) links definitions that record HIP events instead.
__attribute__((weak, noinline)) void timing_begin(const char *, hipStream_t) {}
__attribute__((weak, noinline)) void timing_end(hipStream_t) {}

}  // namespace phsa

using namespace phsa;

#define PHSA_GUARD(body)            \
  try {                             \
    body                            \
  } catch (const std::exception &) { \
    return PHSA_ERR_HIP;            \
  } catch (...) {                   \
    return PHSA_ERR_HIP;            \
  }

extern "C" {

int32_t phsa_ksel(const phsa_params *p) {
  if (!p || p->block_size < 1 || p->n_init_blocks < 0 || p->window < 0 || p->top_k < 0) return 0;
  const int64_t k = (int64_t)p->n_init_blocks + p->window / p->block_size + 1 + p->top_k;
  return k > INT32_MAX ? 0 : (int32_t)k;
}

phsa_status phsa_validate(const phsa_params *p, int32_t op) { return validate(p, op, nullptr); }

size_t phsa_workspace_size(const phsa_params *p, int32_t op) {
  Geom g;
  if (validate(p, op, &g) != PHSA_OK) return 0;
  return workspace_bytes(g, op);
}

const char *phsa_status_string(phsa_status s) {
  // a C caller may pass any int: read the bits as one, not as the enum
  int v;
  memcpy(&v, &s, sizeof v);
  switch (v) {
    case PHSA_OK: return "ok";
    case PHSA_ERR_INVALID_ARG: return "invalid argument";
    case PHSA_ERR_SHAPE: return "inconsistent shape";
    case PHSA_ERR_DTYPE: return "unknown dtype";
    case PHSA_ERR_NULL: return "null pointer";
    case PHSA_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case PHSA_ERR_UNSUPPORTED: return "configuration not implemented by the kernels";
    case PHSA_ERR_HIP: return "HIP launch failure";
    case PHSA_ERR_SCRATCH_LIMIT: return "problem larger than the fixed scratch of the scratch-free entry point";
  }
  return "unknown status";
}

phsa_status phsa_compress(const phsa_params *p, const void *K, const uint8_t *punct, float *K_comp, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_COMPRESS, &g);
    if (st != PHSA_OK) return st;
    if (!K || !punct || !K_comp) return PHSA_ERR_NULL;
    return from_hip(launch_compress(g, K, punct, K_comp, static_cast<hipStream_t>(stream)));
  })
}

phsa_status phsa_punct_mask(const int32_t *ids, int64_t n_tokens, const int32_t *punct_ids, int32_t n_punct,
                            uint8_t *mask, void *stream) {
  PHSA_GUARD({
    if (n_tokens < 0 || n_punct < 0) return PHSA_ERR_INVALID_ARG;
    if (n_punct > PHSA_MAX_PUNCT_IDS) return PHSA_ERR_UNSUPPORTED;
    if (n_tokens > 0 && (!ids || !mask)) return PHSA_ERR_NULL;
    if (n_punct > 0 && !punct_ids) return PHSA_ERR_NULL;
    if (n_tokens == 0) return PHSA_OK;  // nothing to do, nothing launched
    return from_hip(launch_punct_mask(ids, n_tokens, punct_ids, n_punct, mask, static_cast<hipStream_t>(stream)));
  })
}

phsa_status phsa_select(const phsa_params *p, const void *Q, const float *K_comp, int32_t *sel, void *ws,
                        size_t ws_bytes, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_SELECT, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K_comp || !sel) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_SELECT, ws, ws_bytes)) != PHSA_OK) return st;
    return from_hip(launch_select(g, Q, K_comp, sel, ws, static_cast<hipStream_t>(stream)));
  })
}

phsa_status phsa_attn_fwd(const phsa_params *p, const void *Q, const void *K, const void *V, const int32_t *sel,
                          void *O, float *LSE, void *ws, size_t ws_bytes, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_ATTN_FWD, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K || !V || !sel || !O || !LSE) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_ATTN_FWD, ws, ws_bytes)) != PHSA_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (g.dtype == PHSA_FP32)
      return from_hip(launch_attn_fwd_fp32(g, static_cast<const float *>(Q), static_cast<const float *>(K),
                                           static_cast<const float *>(V), sel, static_cast<float *>(O), LSE, s));
    return from_hip(attn_fwd_bf16(g, Q, K, V, sel, O, LSE, ws, s));
  })
}

phsa_status phsa_attn_bwd(const phsa_params *p, const void *Q, const void *K, const void *V, const void *O,
                          const void *dO, const float *LSE, const int32_t *sel, void *dQ, void *dK, void *dV, void *ws,
                          size_t ws_bytes, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_ATTN_BWD, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K || !V || !O || !dO || !LSE || !sel || !dQ || !dK || !dV) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_ATTN_BWD, ws, ws_bytes)) != PHSA_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    BwdWs w;
    bwd_layout(g, static_cast<char *>(ws), &w);
    if (g.dtype == PHSA_FP32)
      return from_hip(launch_attn_bwd_fp32(g, static_cast<const float *>(Q), static_cast<const float *>(K),
                                           static_cast<const float *>(V), static_cast<const float *>(O),
                                           static_cast<const float *>(dO), LSE, sel, static_cast<float *>(dQ),
                                           static_cast<float *>(dK), static_cast<float *>(dV), w.Dvec, s));
    const bool reuse = (p->flags & PHSA_FLAG_REUSE_INDEX) != 0;
    return from_hip(launch_attn_bwd(w.co.gc, Q, K, V, O, dO, LSE, sel, dQ, dK, dV, w.ix, w.Dvec, w.dqpart, w.dkvpart,
                                    w.bkv, reuse, s));
  })
}

phsa_status phsa_forward(const phsa_params *p, const void *Q, const void *K, const void *V, const uint8_t *punct,
                         float *K_comp, int32_t *sel, void *O, float *LSE, void *ws, size_t ws_bytes, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_FORWARD, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K || !V || !punct || !K_comp || !sel || !O || !LSE) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_FORWARD, ws, ws_bytes)) != PHSA_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = launch_compress(g, K, punct, K_comp, s);
    if (e == hipSuccess) e = launch_select(g, Q, K_comp, sel, ws, s);
    if (e != hipSuccess) return PHSA_ERR_HIP;
    if (g.dtype == PHSA_FP32)
      return from_hip(launch_attn_fwd_fp32(g, static_cast<const float *>(Q), static_cast<const float *>(K),
                                           static_cast<const float *>(V), sel, static_cast<float *>(O), LSE, s));
    return from_hip(attn_fwd_bf16(g, Q, K, V, sel, O, LSE, ws, s));
  })
}

phsa_status phsa_decode(const phsa_params *p, const void *Q, const void *K_cache, const void *V_cache,
                        const float *K_comp, int32_t *sel, void *O, float *LSE, void *ws, size_t ws_bytes,
                        void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_DECODE, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K_cache || !V_cache || !K_comp || !sel || !O || !LSE) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_DECODE, ws, ws_bytes)) != PHSA_OK) return st;
    return from_hip(
        launch_decode(g, Q, K_cache, V_cache, K_comp, nullptr, sel, O, LSE, static_cast<hipStream_t>(stream)));
  })
}

phsa_status phsa_decode_varlen(const phsa_params *p, const void *Q, const void *K_cache, const void *V_cache,
                               const float *K_comp, const int32_t *cache_len, int32_t *sel, void *O, float *LSE,
                               void *ws, size_t ws_bytes, void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_DECODE, &g);
    if (st != PHSA_OK) return st;
    if (!Q || !K_cache || !V_cache || !K_comp || !cache_len || !sel || !O || !LSE) return PHSA_ERR_NULL;
    if ((st = check_ws(g, PHSA_OP_DECODE, ws, ws_bytes)) != PHSA_OK) return st;
    return from_hip(
        launch_decode(g, Q, K_cache, V_cache, K_comp, cache_len, sel, O, LSE, static_cast<hipStream_t>(stream)));
  })
}

phsa_status phsa_cache_append(const phsa_params *p, const void *K_new, const void *V_new, const uint8_t *punct_new,
                              void *K_cache, void *V_cache, uint8_t *punct_cache, int32_t *cache_len, float *K_comp,
                              void *stream) {
  PHSA_GUARD({
    Geom g;
    phsa_status st = validate(p, PHSA_OP_DECODE, &g);
    if (st != PHSA_OK) return st;
    if (!K_new || !V_new || !punct_new || !K_cache || !V_cache || !punct_cache || !cache_len || !K_comp)
      return PHSA_ERR_NULL;
    return from_hip(launch_cache_append(g, K_new, V_new, punct_new, K_cache, V_cache, punct_cache, cache_len, K_comp,
                                        static_cast<hipStream_t>(stream)));
  })
}

}  // extern "C"

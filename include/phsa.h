/*
 * phsa.h - C ABI of libphsa, the MI355X (gfx950) implementation of PHSA,
 * Punctuation-aware Hybrid Sparse Attention (arXiv 2601.02819).
 *
 * The method (the paper's Section 3.2 and Algorithm 1):
 *   1. cut the keys into T = Lk / m blocks of m tokens (Eq. 3);
 *   2. give every block a representative key M = lambda*M0 + (1-lambda)*Mp,
 *      where M0 is the mean of the block's keys (Eq. 6) and Mp the mean of
 *      the keys at punctuation tokens (Eq. 7), M = M0 when the block has no
 *      punctuation (Eq. 8 and the fallback under Eq. 7);
 *   3. score every causal block against each query, q.M / sqrt(d) (Eq. 8),
 *      keep the forced init blocks and the local window, and add the top-k
 *      remaining blocks (Algorithm 1, block selection);
 *   4. run exact softmax attention over only the selected blocks (Eq. 10-11).
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE pointers; the caller owns every buffer,
 *     including the workspace.  The library never allocates device memory and
 *     never synchronises; all work is enqueued on `stream` (a hipStream_t, or
 *     NULL for the default stream) and the call returns immediately.
 *   - Layouts are contiguous row-major:
 *       Q, O, dO, dQ     [B, Lq, Hq, d]       (dtype)
 *       K, V, dK, dV     [B, Lk, Hkv, d]      (dtype)
 *       punct            [B, Lk]              uint8, 1 = punctuation token
 *       K_comp           [B, Hkv, T, d]       float32, T = Lk / m
 *       sel              [B, Hkv, Lq, Ksel]   int32, ascending block ids,
 *                                             padded at the end with -1
 *       LSE              [B, Hq, Lq]          float32, natural log of
 *                                             sum_j exp(scale * q.k_j)
 *     with Ksel = n_init_blocks + window / block_size + 1 + top_k.
 *   - Query row i sits at sequence position (Lk - Lq) + i: prefill has
 *     Lq = Lk, a decode step has Lq = 1 at position Lk - 1.
 *   - Query head h reads key/value head h / (Hq / Hkv) (grouped-query
 *     attention).  Selection is shared by the Hq / Hkv heads of a group: a
 *     block's group score is the sum over those heads of q_h.M / sqrt(d).
 *   - Ties in the top-k are broken towards the lower block index.
 *   - Validation runs on the host before anything is enqueued.  On an error
 *     nothing is launched and no output is written.  PHSA_ERR_HIP reports a
 *     failed launch; faults inside kernels surface at the caller's next
 *     synchronisation of the stream.
 *   - No C++ exception crosses this interface.
 *   - The library keeps no mutable global state: calls are reentrant, and
 *     calls on different streams with separate workspaces are independent.
 */
#ifndef PHSA_H
#define PHSA_H

#include <stddef.h>
#include <stdint.h>

/* Symbols of the C ABI; the library exports nothing else. */
#ifndef PHSA_API
#define PHSA_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PHSA_OK = 0,
  PHSA_ERR_INVALID_ARG = 1, /* a scalar parameter is out of range (lambda, top_k, ...) */
  PHSA_ERR_SHAPE = 2,       /* inconsistent sizes (Lk % m, Hq % Hkv, Lq > Lk, ...) */
  PHSA_ERR_DTYPE = 3,       /* dtype is not PHSA_BF16 / PHSA_FP32 */
  PHSA_ERR_NULL = 4,        /* a required pointer is NULL */
  PHSA_ERR_WORKSPACE = 5,   /* ws_bytes < phsa_workspace_size(params, op) or ws is NULL */
  PHSA_ERR_UNSUPPORTED = 6, /* valid for the method but outside what the kernels implement */
  PHSA_ERR_HIP = 7,         /* a HIP launch failed */
  PHSA_ERR_SCRATCH_LIMIT = 8 /* needs more than the fixed scratch of a scratch-free entry point */
} phsa_status;

typedef enum { PHSA_BF16 = 0, PHSA_FP32 = 1 } phsa_dtype;

/* Operation ids for phsa_workspace_size / phsa_validate. */
typedef enum {
  PHSA_OP_COMPRESS = 0,
  PHSA_OP_SELECT = 1,
  PHSA_OP_ATTN_FWD = 2,
  PHSA_OP_ATTN_BWD = 3,
  PHSA_OP_FORWARD = 4,
  PHSA_OP_DECODE = 5
} phsa_op;

/* Problem description (Algorithm 1's inputs plus the tensor geometry). */
typedef struct {
  int32_t batch;         /* B  >= 1 */
  int32_t seqlen_q;      /* Lq >= 1, Lq <= Lk */
  int32_t seqlen_k;      /* Lk, a multiple of block_size (Eq. 3 with no tail) */
  int32_t n_heads_q;     /* Hq, a multiple of n_heads_kv */
  int32_t n_heads_kv;    /* Hkv >= 1 */
  int32_t head_dim;      /* d; the kernels implement 64 and 128 */
  int32_t block_size;    /* m, tokens per key block (Eq. 3).  compress/select take any m;
                            attention takes 16, 32 and 64 (bf16 forward/backward with
                            m < 64 also need seqlen_k to be a multiple of 64) */
  int32_t top_k;         /* k, free picks after the forced blocks are excluded */
  int32_t n_init_blocks; /* n_init, blocks 0..n_init-1 always kept (clipped to causal) */
  int32_t window;        /* w, local window in tokens, a multiple of block_size;
                            blocks max(0, cur - w/m) .. cur are always kept */
  float lambda;          /* gate of Eq. 8, in [0, 1] */
  float softmax_scale;   /* <= 0 selects 1 / sqrt(head_dim) (Eq. 2, 8, 11) */
  int32_t dtype;         /* phsa_dtype of Q, K, V, O, dO, dQ, dK, dV */
  int32_t flags;         /* bitwise OR of phsa_flag values, 0 for none */
} phsa_params;

/* phsa_params.flags */
typedef enum {
  /* phsa_attn_bwd only: `ws` is the workspace a preceding phsa_attn_fwd or
   * phsa_forward call used with the same params and the same sel, and it has
   * not been modified since.  The inverted selection index that call built
   * (the first part of the workspace) is reused instead of rebuilt; the rest of
   * the workspace is overwritten.  ws_bytes must still cover
   * phsa_workspace_size(p, PHSA_OP_ATTN_BWD). */
  PHSA_FLAG_REUSE_INDEX = 1,
  /* phsa_select, phsa_forward, phsa_decode, phsa_decode_varlen: rank blocks
   * by Eq. 8's softmax taken per query head and summed over the heads that
   * share a KV head (the grouped-query aggregation of NSA) instead of by the
   * summed logits.  Each head's softmax runs over the complete blocks before
   * the query's own block (0 .. cur-1): the own block holds keys past the
   * query in prefill and is still filling in generation.  For one head per
   * group both modes select the same blocks.  Forced blocks are unchanged. */
  PHSA_FLAG_SELECT_SOFTMAX_SUM = 2
} phsa_flag;

/* Number of index slots per (query row, KV head): n_init + w/m + 1 + top_k;
 * 0 when p is NULL, block_size < 1, a count is negative or the sum exceeds
 * INT32_MAX. */
PHSA_API int32_t phsa_ksel(const phsa_params *p);

/* Host-only validation of `p` for operation `op` (no GPU access). */
PHSA_API phsa_status phsa_validate(const phsa_params *p, int32_t op);

/* Workspace bytes `op` needs for `p` (0 if none, or if `p` is invalid). */
PHSA_API size_t phsa_workspace_size(const phsa_params *p, int32_t op);

/* Static, human-readable name of a status code. */
PHSA_API const char *phsa_status_string(phsa_status s);

/* Punctuation mask from token ids: mask[i] = 1 if ids[i] is one of the
 * punctuation ids, else 0 (the indicator I(x_i in P) of Eq. 7, Section 3.2
 * "Punctuation Token Selection").  ids and mask hold n_tokens entries of any
 * shape (e.g. [B, Lk], the layout phsa_compress reads); punct_ids holds the
 * set P and must be sorted ascending (duplicates are allowed).  All device
 * pointers.  n_punct may be 0 (no token is punctuation) and at most
 * PHSA_MAX_PUNCT_IDS (PHSA_ERR_UNSUPPORTED beyond).  Building P from a
 * tokenizer's vocabulary is the caller's part. */
#define PHSA_MAX_PUNCT_IDS 16384
PHSA_API phsa_status phsa_punct_mask(const int32_t *ids, int64_t n_tokens, const int32_t *punct_ids, int32_t n_punct,
                            uint8_t *mask, void *stream);

/* Block representatives (Eq. 6-8, Algorithm 1 representative-token step).
 * Reads K [B, Lk, Hkv, d] and punct [B, Lk]; writes K_comp [B, Hkv, T, d]
 * (float32, sums accumulated in float32).  Uses seqlen_k, not seqlen_q. */
PHSA_API phsa_status phsa_compress(const phsa_params *p, const void *K, const uint8_t *punct, float *K_comp,
                          void *stream);

/* Relevance scoring and block selection (Eq. 8, Algorithm 1 scoring and
 * selection).  Reads Q and K_comp; writes sel [B, Hkv, Lq, Ksel].  Scores
 * are computed in float32 from float32 K_comp.  The bf16 path needs
 * phsa_workspace_size(p, PHSA_OP_SELECT) bytes of workspace (split copies of
 * K_comp); the float32 path needs none (ws may then be NULL). */
PHSA_API phsa_status phsa_select(const phsa_params *p, const void *Q, const float *K_comp, int32_t *sel,
                        void *ws, size_t ws_bytes, void *stream);

/* Sparse attention forward (Eq. 10-11, Algorithm 1 attention step) over the
 * blocks listed in sel, with the token-level causal mask j <= position(i).
 * Writes O [B, Lq, Hq, d] (dtype) and LSE [B, Hq, Lq].  sel rows must be
 * ascending, duplicate-free, within 0..cur of their row, and -1 padded. */
PHSA_API phsa_status phsa_attn_fwd(const phsa_params *p, const void *Q, const void *K, const void *V,
                          const int32_t *sel, void *O, float *LSE, void *ws, size_t ws_bytes,
                          void *stream);

/* Sparse attention backward with sel held fixed (the top-k is piecewise
 * constant, so K_comp, lambda and the mask receive no gradient).  Reads the
 * forward tensors, dO and LSE; writes dQ [B, Lq, Hq, d] and dK, dV
 * [B, Lk, Hkv, d] (dtype; float32 accumulation).  dK/dV sum over the heads
 * of each group; keys that no query selected get zero gradient. */
PHSA_API phsa_status phsa_attn_bwd(const phsa_params *p, const void *Q, const void *K, const void *V,
                          const void *O, const void *dO, const float *LSE, const int32_t *sel,
                          void *dQ, void *dK, void *dV, void *ws, size_t ws_bytes, void *stream);

/* Whole forward: phsa_compress, phsa_select, phsa_attn_fwd in one call.
 * Writes K_comp, sel, O and LSE. */
PHSA_API phsa_status phsa_forward(const phsa_params *p, const void *Q, const void *K, const void *V,
                         const uint8_t *punct, float *K_comp, int32_t *sel, void *O, float *LSE,
                         void *ws, size_t ws_bytes, void *stream);

/* One decode step (generation with a block KV cache): Lq must be 1, the
 * query sits at position Lk - 1.  K_comp [B, Hkv, T, d] holds the cache's
 * block representatives (from phsa_compress).  Writes sel [B, Hkv, 1, Ksel],
 * O [B, 1, Hq, d] and LSE [B, Hq, 1]. */
PHSA_API phsa_status phsa_decode(const phsa_params *p, const void *Q, const void *K_cache,
                        const void *V_cache, const float *K_comp, int32_t *sel, void *O,
                        float *LSE, void *ws, size_t ws_bytes, void *stream);

/* Generation with per-sequence cache lengths.  The caches have capacity
 * Lk = p->seqlen_k tokens (a multiple of block_size): K_cache, V_cache
 * [B, Lk, Hkv, d], punct_cache [B, Lk], K_comp [B, Hkv, Lk / m, d];
 * cache_len [B] (device int32) holds the number of valid tokens of each
 * sequence.  Validation is that of phsa_decode (seqlen_q must be 1).
 *
 * phsa_cache_append: one new token per sequence, K_new and V_new [B, Hkv, d],
 * punct_new [B], is written at position cache_len[b], and cache_len[b] grows
 * by one.  When the token completes block t = cache_len[b] / m (old length),
 * the block's representative (Eq. 6-8, as phsa_compress computes it) is
 * written to K_comp[b, :, t]; no other block is touched ("block-level
 * key-value caching", Section 3.2 "Block Segmentation").  A sequence whose
 * cache is full (cache_len[b] >= Lk) is left unchanged.
 *
 * phsa_decode_varlen: as phsa_decode, but sequence b's query sits at position
 * cache_len[b] - 1 (lengths are clamped to [1, Lk]).  Its own block may be
 * partly written: it is always selected (forced), and keys past the query are
 * masked without their values being read.  Only complete blocks are scored,
 * so K_comp must hold the representatives of every complete block below the
 * query's own (phsa_compress on the prefilled prefix, then phsa_cache_append). */
PHSA_API phsa_status phsa_decode_varlen(const phsa_params *p, const void *Q, const void *K_cache,
                               const void *V_cache, const float *K_comp, const int32_t *cache_len,
                               int32_t *sel, void *O, float *LSE, void *ws, size_t ws_bytes,
                               void *stream);
PHSA_API phsa_status phsa_cache_append(const phsa_params *p, const void *K_new, const void *V_new,
                              const uint8_t *punct_new, void *K_cache, void *V_cache,
                              uint8_t *punct_cache, int32_t *cache_len, float *K_comp, void *stream);

/* Scratch-free selection, for callers that cannot allocate device memory:
 * code under HIP graph capture, allocation-free serving loops, harnesses that
 * forbid hipMalloc.  It is phsa_select without a workspace: the bf16 path's
 * scratch (the bf16 hi/lo split of K_comp and the block norms,
 * phsa_workspace_size(p, PHSA_OP_SELECT) bytes) lives in a static device array
 * of PHSA_NOALLOC_SCRATCH_BYTES inside the library.  Each GPU the library runs
 * on holds its own copy until the process ends; its address is looked up once
 * per GPU, on the first call there.  The call allocates nothing.
 *   - A problem whose scratch exceeds the array (B * Hkv * (Lk / m) blocks at
 *     2 * 2 * d + 4 bytes each) returns PHSA_ERR_SCRATCH_LIMIT; nothing is
 *     launched.
 *   - `stream` must belong to the current device (PHSA_ERR_INVALID_ARG
 *     otherwise).
 *   - All calls on one GPU share its array and leave their contents in it:
 *     calls that overlap in time on one GPU (different streams or host
 *     threads) race, and the caller must order them.
 * Results are those of phsa_select with the same arguments. */
#define PHSA_NOALLOC_SCRATCH_BYTES (64u << 20)
PHSA_API phsa_status phsa_select_noalloc(const phsa_params *p, const void *Q, const float *K_comp, int32_t *sel,
                                         void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PHSA_H */

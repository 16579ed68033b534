// Host-side exercise of the C ABI layer (validation, workspace sizing and
// layout, dispatch up to the launchers) for a build under AddressSanitizer and
// UndefinedBehaviorSanitizer.  The launchers are stand-ins that fail, so no GPU
// is needed.  Exits 0 when every check holds; any sanitizer report aborts.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "phsa.h"

static int g_fail = 0;
static long g_checks = 0;

#define CHECK(c)                                                        \
  do {                                                                  \
    ++g_checks;                                                         \
    if (!(c)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);   \
      ++g_fail;                                                         \
    }                                                                   \
  } while (0)

// a small deterministic generator (64-bit LCG, high bits)
static unsigned long long g_state = 0x9e3779b97f4a7c15ull;
static unsigned rnd() {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return (unsigned)(g_state >> 33);
}
static int pick(const int *v, int n) { return v[rnd() % n]; }

static phsa_params base() {
  phsa_params p;
  memset(&p, 0, sizeof(p));
  p.batch = 1;
  p.seqlen_q = 1024;
  p.seqlen_k = 1024;
  p.n_heads_q = 2;
  p.n_heads_kv = 1;
  p.head_dim = 64;
  p.block_size = 64;
  p.top_k = 2;
  p.n_init_blocks = 1;
  p.window = 0;
  p.lambda = 0.5f;
  p.softmax_scale = 0.f;
  p.dtype = PHSA_BF16;
  p.flags = 0;
  return p;
}

static phsa_params random_params() {
  static const int sizes[] = {-1, 0, 1, 2, 3, 16, 63, 64, 65, 100, 128, 192, 1000, 1024, 4096, 32768, 65536,
                              1 << 20, 1 << 25, 0x7fffffff};
  static const int small[] = {-1, 0, 1, 2, 3, 4, 6, 8, 12, 16, 17, 31, 32, 33, 63, 64, 65, 1000, 0x7fffffff};
  static const int dims[] = {0, 1, 32, 64, 96, 128, 256};
  static const int blocks[] = {0, 1, 8, 16, 32, 48, 64, 128, 0x7fffffff};
  phsa_params p = base();
  p.batch = pick(small, 19);
  p.seqlen_k = pick(sizes, 20);
  p.seqlen_q = (rnd() & 1) ? p.seqlen_k : pick(sizes, 20);
  p.n_heads_kv = pick(small, 19);
  const long long hq = (long long)p.n_heads_kv * (1 + (rnd() % 8));
  p.n_heads_q = (rnd() & 1) && hq <= 0x7fffffff ? (int)hq : pick(small, 19);
  p.head_dim = pick(dims, 7);
  p.block_size = pick(blocks, 9);
  p.top_k = pick(small, 19);
  p.n_init_blocks = pick(small, 19);
  const long long w = (long long)p.block_size * (rnd() % 40);
  p.window = (rnd() & 1) && w <= 0x7fffffff ? (int)w : pick(sizes, 20);
  const float lams[] = {0.f, 0.5f, 1.f, -0.1f, 1.5f, __builtin_nanf("")};
  p.lambda = lams[rnd() % 6];
  const float scales[] = {0.f, -1.f, 0.125f, __builtin_inff()};
  p.softmax_scale = scales[rnd() % 4];
  p.dtype = (int)(rnd() % 3);
  p.flags = (int)(rnd() % 5);
  return p;
}

// Entry points on host memory: returns the status of a call whose pointers are
// never dereferenced on the host (the launchers are stand-ins).
static void call_all(const phsa_params &p) {
  static float dummy[64];
  void *d = dummy;
  const size_t need = phsa_workspace_size(&p, PHSA_OP_ATTN_BWD) + phsa_workspace_size(&p, PHSA_OP_FORWARD) +
                      phsa_workspace_size(&p, PHSA_OP_SELECT);
  if (need > ((size_t)64 << 20)) return;
  // 256-byte aligned host workspace; the layout code only computes addresses in it
  std::vector<unsigned char> mem(need + 512);
  unsigned char *ws = mem.data() + (256 - ((uintptr_t)mem.data() & 255));
  const size_t ws_bytes = need;
  const phsa_status v_c = phsa_validate(&p, PHSA_OP_COMPRESS);
  const phsa_status r_c = phsa_compress(&p, d, (const uint8_t *)d, (float *)d, NULL);
  CHECK(r_c == (v_c == PHSA_OK ? PHSA_ERR_HIP : v_c));
  const phsa_status v_s = phsa_validate(&p, PHSA_OP_SELECT);
  const phsa_status r_s = phsa_select(&p, d, (const float *)d, (int32_t *)d, ws, ws_bytes, NULL);
  CHECK(r_s == (v_s == PHSA_OK ? PHSA_ERR_HIP : v_s));
  const phsa_status v_f = phsa_validate(&p, PHSA_OP_ATTN_FWD);
  const phsa_status r_f = phsa_attn_fwd(&p, d, d, d, (const int32_t *)d, d, (float *)d, ws, ws_bytes, NULL);
  CHECK(r_f == (v_f == PHSA_OK ? PHSA_ERR_HIP : v_f));
  const phsa_status v_b = phsa_validate(&p, PHSA_OP_ATTN_BWD);
  const phsa_status r_b =
      phsa_attn_bwd(&p, d, d, d, d, d, (const float *)d, (const int32_t *)d, d, d, d, ws, ws_bytes, NULL);
  CHECK(r_b == (v_b == PHSA_OK ? PHSA_ERR_HIP : v_b));
  const phsa_status v_w = phsa_validate(&p, PHSA_OP_FORWARD);
  const phsa_status r_w =
      phsa_forward(&p, d, d, d, (const uint8_t *)d, (float *)d, (int32_t *)d, d, (float *)d, ws, ws_bytes, NULL);
  CHECK(r_w == (v_w == PHSA_OK ? PHSA_ERR_HIP : v_w));
  const phsa_status v_d = phsa_validate(&p, PHSA_OP_DECODE);
  const phsa_status r_d = phsa_decode(&p, d, d, d, (const float *)d, (int32_t *)d, d, (float *)d, ws, ws_bytes, NULL);
  CHECK(r_d == (v_d == PHSA_OK ? PHSA_ERR_HIP : v_d));
  const phsa_status r_v = phsa_decode_varlen(&p, d, d, d, (const float *)d, (const int32_t *)d, (int32_t *)d, d,
                                             (float *)d, ws, ws_bytes, NULL);
  CHECK(r_v == (v_d == PHSA_OK ? PHSA_ERR_HIP : v_d));
  const phsa_status r_a = phsa_cache_append(&p, d, d, (const uint8_t *)d, d, d, (uint8_t *)d, (int32_t *)d,
                                            (float *)d, NULL);
  CHECK(r_a == (v_d == PHSA_OK ? PHSA_ERR_HIP : v_d));
  // a workspace one byte short is refused before anything is launched
  const size_t wf = phsa_workspace_size(&p, PHSA_OP_ATTN_FWD);
  if (v_f == PHSA_OK && wf > 0)
    CHECK(phsa_attn_fwd(&p, d, d, d, (const int32_t *)d, d, (float *)d, ws, wf - 1, NULL) == PHSA_ERR_WORKSPACE);
}

int main() {
  // NULL arguments
  CHECK(phsa_validate(NULL, PHSA_OP_SELECT) == PHSA_ERR_NULL);
  CHECK(phsa_workspace_size(NULL, PHSA_OP_ATTN_FWD) == 0);
  CHECK(phsa_ksel(NULL) == 0);
  phsa_params p = base();
  CHECK(phsa_compress(&p, NULL, NULL, NULL, NULL) == PHSA_ERR_NULL);
  CHECK(phsa_punct_mask(NULL, 0, NULL, 0, NULL, NULL) == PHSA_OK);
  CHECK(phsa_punct_mask(NULL, 5, NULL, 0, NULL, NULL) == PHSA_ERR_NULL);
  CHECK(phsa_punct_mask(NULL, -5, NULL, 0, NULL, NULL) == PHSA_ERR_INVALID_ARG);
  for (int s = -3; s < 12; ++s) CHECK(phsa_status_string((phsa_status)s) != NULL);
  for (int op = -2; op < 8; ++op) (void)phsa_workspace_size(&p, op);

  // the workloads' configurations, bf16 and fp32
  const int shapes[][10] = {
      // B, L, Hq, Hkv, d, m, top_k, n_init, window, dtype
      {1, 1024, 2, 1, 64, 64, 2, 1, 0, PHSA_FP32},
      {1, 8192, 16, 8, 128, 64, 14, 1, 0, PHSA_BF16},
      {1, 32768, 16, 8, 128, 64, 12, 1, 0, PHSA_BF16},
      {4, 32768, 16, 8, 128, 16, 16, 8, 512, PHSA_BF16},
      {64, 32768, 16, 8, 128, 64, 12, 1, 0, PHSA_BF16},
      {2, 320, 8, 2, 128, 32, 5, 2, 64, PHSA_BF16},
  };
  for (const auto &c : shapes) {
    phsa_params q = base();
    q.batch = c[0];
    q.seqlen_q = q.seqlen_k = c[1];
    q.n_heads_q = c[2];
    q.n_heads_kv = c[3];
    q.head_dim = c[4];
    q.block_size = c[5];
    q.top_k = c[6];
    q.n_init_blocks = c[7];
    q.window = c[8];
    q.dtype = c[9];
    CHECK(phsa_validate(&q, PHSA_OP_ATTN_BWD) == PHSA_OK);
    CHECK(phsa_workspace_size(&q, PHSA_OP_FORWARD) >= phsa_workspace_size(&q, PHSA_OP_SELECT));
    call_all(q);
    q.seqlen_q = 1;
    call_all(q);
  }

  // random and extreme parameters: validation, sizing and layout must stay
  // free of overflow and out-of-range arithmetic
  for (int it = 0; it < 20000; ++it) {
    phsa_params q = random_params();
    for (int op = 0; op <= PHSA_OP_DECODE; ++op) {
      const phsa_status v = phsa_validate(&q, op);
      const size_t w = phsa_workspace_size(&q, op);
      if (v != PHSA_OK) CHECK(w == 0);
    }
    (void)phsa_ksel(&q);
    call_all(q);
  }
  printf("%ld checks, %d failed\n", g_checks, g_fail);
  return g_fail == 0 ? 0 : 1;
}

/*
 * PHSA oracle: a plain, slow, obviously-correct CPU implementation of
 * Punctuation-aware Hybrid Sparse Attention (arXiv 2601.02819).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference the GPU library is
 * checked against.  Only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark may load it; the product path never does.  It shares no
 * code, header, table or helper with the HIP library.
 *
 * Arithmetic is IEEE double throughout.  Inputs arrive as float32 arrays,
 * which hold bf16 and fp32 values exactly, and are widened to double on use.
 * Loops follow the paper's definitions directly; OpenMP only distributes
 * independent rows/blocks over host cores.
 *
 * Layouts (row-major, contiguous):
 *   Q   [B, Lq, Hq,  d]      K, V [B, Lk, Hkv, d]      punct [B, Lk] (0/1)
 *   Kc  [B, Hkv, T, d]       T = Lk / m
 *   sel [B, Hkv, Lq, Ksel]   ascending block ids, padded with -1
 * Query row i sits at sequence position q_pos0 + i (q_pos0 = Lk - Lq: prefill
 * has q_pos0 = 0, a one-token decode step has q_pos0 = Lk - 1).
 * Query head h reads key/value head g = h / (Hq / Hkv).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Number of threads the oracle's parallel loops run on (as timed by the
 * benchmark's CPU baseline). */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
  return n;
}

#define IDX4(a, b, c, d_, B_, C_, D_) ((((int64_t)(a) * (B_) + (b)) * (C_) + (c)) * (D_) + (d_))

/* ------------------------------------------------------------------------ */
/* Punctuation indicator of Eq. 7 (Section 3.2, Punctuation Token Selection):
 * mask[i] = I(x_i in P), the token id x_i compared with every id of the set
 * P in turn.  ids [n], punct_ids [n_punct] in any order.                    */
void oracle_punct_mask(int64_t n, const int32_t *ids, int32_t n_punct, const int32_t *punct_ids,
                       uint8_t *mask) {
  for (int64_t i = 0; i < n; ++i) {
    uint8_t hit = 0;
    for (int32_t j = 0; j < n_punct; ++j)
      if (ids[i] == punct_ids[j]) hit = 1;
    mask[i] = hit;
  }
}

/* ------------------------------------------------------------------------ */
/* Block representatives: global mean (Eq. 6), punctuation mean (Eq. 7),
 * gated fusion (Eq. 8), with the no-punctuation fallback M = M0 of Eq. 7 and
 * the "else" branch of Algorithm 1's representative-token step.            */
void oracle_compress(int B, int Lk, int Hkv, int d, int m, double lambda,
                     const float *K, const uint8_t *punct, double *Kc) {
  const int T = Lk / m; /* Eq. 3: T = floor(L / m) blocks of m tokens */
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < Hkv; ++g)
      for (int t = 0; t < T; ++t) {
        double *out = Kc + IDX4(b, g, t, 0, Hkv, T, d);
        int npunct = 0;
        for (int i = t * m; i < (t + 1) * m; ++i) npunct += punct[(int64_t)b * Lk + i] ? 1 : 0;
        for (int c = 0; c < d; ++c) {
          double sum_all = 0.0, sum_p = 0.0;
          for (int i = t * m; i < (t + 1) * m; ++i) {
            double k = (double)K[IDX4(b, i, g, c, Lk, Hkv, d)];
            sum_all += k;
            if (punct[(int64_t)b * Lk + i]) sum_p += k;
          }
          double M0 = sum_all / (double)m; /* Eq. 6 */
          if (npunct > 0) {
            double Mp = sum_p / (double)npunct;        /* Eq. 7 */
            out[c] = lambda * M0 + (1.0 - lambda) * Mp; /* Eq. 8 */
          } else {
            out[c] = M0; /* fallback stated under Eq. 7 */
          }
        }
      }
}

/* ------------------------------------------------------------------------ */
/* Relevance of block t for query row i and KV group g: the scaled logit
 * q^T M(B_t) / sqrt(d_k) of Eq. 8 / Algorithm 1 (relevance scoring), summed
 * over the query heads that share KV head g.  Softmax is monotone per row,
 * so ranking on these logits ranks the Eq. 8 weights identically.          */
static double group_score(const float *Q, const double *Kc, int b, int i, int g, int t,
                          int Lq, int Hq, int Hkv, int T, int d, double scale) {
  const int G = Hq / Hkv;
  double s = 0.0;
  for (int hh = 0; hh < G; ++hh) {
    const int h = g * G + hh;
    double dot = 0.0;
    for (int c = 0; c < d; ++c)
      dot += (double)Q[IDX4(b, i, h, c, Lq, Hq, d)] * Kc[IDX4(b, g, t, c, Hkv, T, d)];
    s += scale * dot;
  }
  return s;
}

/* Scaled logit q_h^T M(B_t) / sqrt(d_k) of one query head h (Eq. 8). */
static double head_logit(const float *Q, const double *Kc, int b, int i, int h, int g, int t,
                         int Lq, int Hq, int Hkv, int T, int d, double scale) {
  double dot = 0.0;
  for (int c = 0; c < d; ++c) dot += (double)Q[IDX4(b, i, h, c, Lq, Hq, d)] * Kc[IDX4(b, g, t, c, Hkv, T, d)];
  return scale * dot;
}

/* Selection mode SOFTMAX_SUM: Eq. 8 taken literally per query head, i.e. the
 * softmax of the head's block logits, and the group's heads combined by
 * adding their probabilities.  The softmax runs over the complete blocks in
 * the query's causal past, 0 .. cur-1: the query's own block is left out
 * because it holds keys past the query (in prefill) or is still being filled
 * (in generation).  lse[hh] = log sum_{t < cur} exp(logit_h(t)) for the G
 * heads of group g; -inf when cur = 0.                                      */
static void head_log_normalisers(const float *Q, const double *Kc, int b, int i, int g, int cur,
                                 int Lq, int Hq, int Hkv, int T, int d, double scale, double *lse) {
  const int G = Hq / Hkv;
  for (int hh = 0; hh < G; ++hh) {
    const int h = g * G + hh;
    double mx = -INFINITY;
    for (int t = 0; t < cur; ++t) {
      const double x = head_logit(Q, Kc, b, i, h, g, t, Lq, Hq, Hkv, T, d, scale);
      if (x > mx) mx = x;
    }
    double sum = 0.0;
    for (int t = 0; t < cur; ++t) sum += exp(head_logit(Q, Kc, b, i, h, g, t, Lq, Hq, Hkv, T, d, scale) - mx);
    lse[hh] = cur > 0 ? mx + log(sum) : -INFINITY;
  }
}

/* Group score of block t in mode SOFTMAX_SUM, in log units:
 * log sum_h softmax_h(t), which ranks blocks exactly as the summed
 * probabilities do.                                                         */
static double group_softmax_score(const float *Q, const double *Kc, int b, int i, int g, int t,
                                  int Lq, int Hq, int Hkv, int T, int d, double scale, const double *lse) {
  const int G = Hq / Hkv;
  double p = 0.0;
  for (int hh = 0; hh < G; ++hh)
    p += exp(head_logit(Q, Kc, b, i, g * G + hh, g, t, Lq, Hq, Hkv, T, d, scale) - lse[hh]);
  return log(p);
}

/* Scores of every block for one (b, i, g) in the given mode (0 = summed
 * logits, 1 = summed per-head softmax); query row i sits at q_pos0 + i.
 * In mode 1 blocks outside 0 .. cur-1 get -inf.                              */
void oracle_score_row(int B, int Lq, int Lk, int Hq, int Hkv, int d, int m, double scale,
                      const float *Q, const double *Kc, int b, int i, int g, int q_pos0, int mode,
                      double *scores_T) {
  (void)B;
  const int T = Lk / m;
  if (mode == 1) {
    const int cur = (q_pos0 + i) / m;
    double lse[64];
    head_log_normalisers(Q, Kc, b, i, g, cur, Lq, Hq, Hkv, T, d, scale, lse);
    for (int t = 0; t < T; ++t)
      scores_T[t] = t < cur ? group_softmax_score(Q, Kc, b, i, g, t, Lq, Hq, Hkv, T, d, scale, lse) : -INFINITY;
    return;
  }
  for (int t = 0; t < T; ++t)
    scores_T[t] = group_score(Q, Kc, b, i, g, t, Lq, Hq, Hkv, T, d, scale);
}

typedef struct {
  double s;
  int t;
} cand_t;

/* score descending, then lower block index first */
static int cand_cmp(const void *a, const void *b) {
  const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->t < y->t) ? -1 : (x->t > y->t);
}

static int int_cmp(const void *a, const void *b) {
  int x = *(const int *)a, y = *(const int *)b;
  return (x > y) - (x < y);
}

/* Block selection of Algorithm 1: forced init blocks {0..n_init-1} and local
 * window {max(0, cur - w/m) .. cur}; causal mask of future blocks; forced
 * blocks excluded from the ranking; top-k of the rest; Unique of the union.
 * Rows: list of b*Lq + i (NULL = all rows, in order).  Outputs are compact:
 *   sel_out [n_rows, Hkv, Ksel], kth_out/gap_out [n_rows, Hkv].
 * kth_out = score of the k-th pick (NaN if no pick), gap_out = k-th minus
 * (k+1)-th score (+inf when there is no (k+1)-th candidate).
 * mode 0 ranks on the group's summed logits, mode 1 on log sum_h softmax_h
 * (SOFTMAX_SUM above); kth/gap are in the mode's own units.                */
void oracle_select(int B, int Lq, int Lk, int Hq, int Hkv, int d, int m, int top_k, int n_init,
                   int window, int q_pos0, int mode, double scale, const float *Q, const double *Kc,
                   int64_t n_rows, const int64_t *rows, int32_t *sel_out, double *kth_out,
                   double *gap_out) {
  (void)B;
  const int T = Lk / m;
  const int Ksel = n_init + window / m + 1 + top_k;
#pragma omp parallel
  {
    cand_t *cand = (cand_t *)malloc(sizeof(cand_t) * (size_t)(T > 0 ? T : 1));
    int *final_set = (int *)malloc(sizeof(int) * (size_t)(T + Ksel + 1));
    char *forced = (char *)malloc((size_t)(T > 0 ? T : 1));
#pragma omp for collapse(2) schedule(dynamic, 16)
    for (int64_t r = 0; r < n_rows; ++r)
      for (int g = 0; g < Hkv; ++g) {
        const int64_t row = rows ? rows[r] : r;
        const int b = (int)(row / Lq), i = (int)(row % Lq);
        const int pos = q_pos0 + i;
        const int cur = pos / m;
        memset(forced, 0, (size_t)T);
        for (int t = 0; t < n_init && t <= cur; ++t) forced[t] = 1; /* init, clipped to <= cur */
        int lo = cur - window / m;
        if (lo < 0) lo = 0;
        for (int t = lo; t <= cur; ++t) forced[t] = 1; /* local window incl. own block */
        double lse[64];
        if (mode == 1) head_log_normalisers(Q, Kc, b, i, g, cur, Lq, Hq, Hkv, T, d, scale, lse);
        int nc = 0;
        for (int t = 0; t <= cur; ++t) /* causal: only blocks <= cur */
          if (!forced[t]) {
            cand[nc].t = t;
            cand[nc].s = mode == 1 ? group_softmax_score(Q, Kc, b, i, g, t, Lq, Hq, Hkv, T, d, scale, lse)
                                   : group_score(Q, Kc, b, i, g, t, Lq, Hq, Hkv, T, d, scale);
            ++nc;
          }
        qsort(cand, (size_t)nc, sizeof(cand_t), cand_cmp);
        const int npick = nc < top_k ? nc : top_k;
        int nf = 0;
        for (int t = 0; t <= cur; ++t)
          if (forced[t]) final_set[nf++] = t;
        for (int p = 0; p < npick; ++p) final_set[nf++] = cand[p].t;
        qsort(final_set, (size_t)nf, sizeof(int), int_cmp);
        int32_t *o = sel_out + (r * Hkv + g) * Ksel;
        for (int p = 0; p < Ksel; ++p) o[p] = p < nf ? final_set[p] : -1;
        if (kth_out) kth_out[r * Hkv + g] = npick > 0 ? cand[npick - 1].s : NAN;
        if (gap_out)
          gap_out[r * Hkv + g] = (npick > 0 && nc > npick) ? cand[npick - 1].s - cand[npick].s : INFINITY;
      }
    free(cand);
    free(final_set);
    free(forced);
  }
}

/* ------------------------------------------------------------------------ */
/* Sparse attention of Eq. 10-11 / Algorithm 1 (attention step): the query at
 * position pos attends to the keys j <= pos of its selected blocks, with
 * weights softmax(q.k_j / sqrt(d_k)).  Also returns the natural-log
 * normaliser LSE = log sum_j exp(s_j).                                      */
typedef struct {
  int B, Lq, Lk, Hq, Hkv, d, m, Ksel, q_pos0;
  double scale;
} dims_t;

/* Collect the key indices a (row, group) attends to, in ascending order. */
static int row_keys(const dims_t *D, const int32_t *sel, int b, int i, int g, int *keys) {
  const int pos = D->q_pos0 + i;
  const int32_t *s = sel + IDX4(b, g, i, 0, D->Hkv, D->Lq, D->Ksel);
  int n = 0;
  for (int p = 0; p < D->Ksel; ++p) {
    const int t = s[p];
    if (t < 0) continue;
    for (int j = t * D->m; j < (t + 1) * D->m; ++j)
      if (j <= pos) keys[n++] = j;
  }
  return n;
}

/* Forward for one (b, i, h): fills probs[n] = exp(s_j - LSE), out[d], returns LSE. */
static double row_forward(const dims_t *D, const float *Q, const float *K, const float *V, int b,
                          int i, int h, const int *keys, int n, double *probs, double *out) {
  const int g = h / (D->Hq / D->Hkv);
  double mx = -INFINITY;
  for (int a = 0; a < n; ++a) {
    double dot = 0.0;
    for (int c = 0; c < D->d; ++c)
      dot += (double)Q[IDX4(b, i, h, c, D->Lq, D->Hq, D->d)] *
             (double)K[IDX4(b, keys[a], g, c, D->Lk, D->Hkv, D->d)];
    probs[a] = D->scale * dot;
    if (probs[a] > mx) mx = probs[a];
  }
  double sum = 0.0;
  for (int a = 0; a < n; ++a) sum += exp(probs[a] - mx);
  const double lse = mx + log(sum);
  for (int a = 0; a < n; ++a) probs[a] = exp(probs[a] - lse);
  for (int c = 0; c < D->d; ++c) {
    double acc = 0.0;
    for (int a = 0; a < n; ++a) acc += probs[a] * (double)V[IDX4(b, keys[a], g, c, D->Lk, D->Hkv, D->d)];
    out[c] = acc;
  }
  return lse;
}

/* Rows: list of b*Lq + i (NULL = all).  O_out [n_rows, Hq, d], LSE_out [n_rows, Hq]. */
void oracle_attn_fwd(int B, int Lq, int Lk, int Hq, int Hkv, int d, int m, int Ksel, int q_pos0,
                     double scale, const float *Q, const float *K, const float *V,
                     const int32_t *sel, int64_t n_rows, const int64_t *rows, double *O_out,
                     double *LSE_out) {
  const dims_t D = {B, Lq, Lk, Hq, Hkv, d, m, Ksel, q_pos0, scale};
  const int G = Hq / Hkv;
#pragma omp parallel
  {
    int *keys = (int *)malloc(sizeof(int) * (size_t)Ksel * (size_t)m + 1);
    double *probs = (double *)malloc(sizeof(double) * (size_t)Ksel * (size_t)m + 8);
#pragma omp for collapse(2) schedule(dynamic, 16)
    for (int64_t r = 0; r < n_rows; ++r)
      for (int h = 0; h < Hq; ++h) {
        const int64_t row = rows ? rows[r] : r;
        const int b = (int)(row / Lq), i = (int)(row % Lq);
        const int n = row_keys(&D, sel, b, i, h / G, keys);
        LSE_out[r * Hq + h] =
            row_forward(&D, Q, K, V, b, i, h, keys, n, probs, O_out + (r * Hq + h) * d);
      }
    free(keys);
    free(probs);
  }
}

/* ------------------------------------------------------------------------ */
/* Backward of the sparse attention with the selection held fixed (the top-k
 * is piecewise constant, so no gradient reaches Kc, lambda or the mask).
 * With P_j = exp(s_j - LSE), D = dO . o:
 *   dV_j += P_j dO,  dS_j = P_j (dO . v_j - D),
 *   dQ   += scale sum_j dS_j k_j,  dK_j += scale dS_j q.
 * dQ is produced for the listed rows (NULL = all), compact [n_rows, Hq, d].
 * dK/dV are produced for the listed key blocks (entries b*Hkv*T + g*T + t,
 * NULL = all), compact [n_blocks, m, d]; the all-blocks order is (b, g, t). */
void oracle_attn_bwd(int B, int Lq, int Lk, int Hq, int Hkv, int d, int m, int Ksel, int q_pos0,
                     double scale, const float *Q, const float *K, const float *V,
                     const float *dO, const int32_t *sel, int64_t n_rows, const int64_t *rows,
                     double *dQ_out, int64_t n_blocks, const int64_t *blocks, double *dK_out,
                     double *dV_out) {
  const dims_t D = {B, Lq, Lk, Hq, Hkv, d, m, Ksel, q_pos0, scale};
  const int G = Hq / Hkv;
  const int T = Lk / m;
  const size_t nkeys = (size_t)Ksel * (size_t)m + 1;

  /* dQ: each row depends only on its own forward. */
  if (n_rows > 0 && dQ_out) {
#pragma omp parallel
    {
      int *keys = (int *)malloc(sizeof(int) * nkeys);
      double *probs = (double *)malloc(sizeof(double) * nkeys);
      double *o = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for collapse(2) schedule(dynamic, 16)
      for (int64_t r = 0; r < n_rows; ++r)
        for (int h = 0; h < Hq; ++h) {
          const int64_t row = rows ? rows[r] : r;
          const int b = (int)(row / Lq), i = (int)(row % Lq), g = h / G;
          const int n = row_keys(&D, sel, b, i, g, keys);
          row_forward(&D, Q, K, V, b, i, h, keys, n, probs, o);
          const float *dorow = dO + IDX4(b, i, h, 0, Lq, Hq, d);
          double Dd = 0.0;
          for (int c = 0; c < d; ++c) Dd += (double)dorow[c] * o[c];
          double *dq = dQ_out + (r * Hq + h) * d;
          for (int c = 0; c < d; ++c) dq[c] = 0.0;
          for (int a = 0; a < n; ++a) {
            double dp = 0.0;
            for (int c = 0; c < d; ++c) dp += (double)dorow[c] * (double)V[IDX4(b, keys[a], g, c, Lk, Hkv, d)];
            const double ds = probs[a] * (dp - Dd);
            for (int c = 0; c < d; ++c) dq[c] += scale * ds * (double)K[IDX4(b, keys[a], g, c, Lk, Hkv, d)];
          }
        }
      free(keys);
      free(probs);
      free(o);
    }
  }

  /* dK, dV: block slot in the compact output, -1 if not requested. */
  if (n_blocks > 0 && dK_out && dV_out) {
    const int64_t nall = (int64_t)B * Hkv * T;
    int64_t *slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)nall);
    for (int64_t x = 0; x < nall; ++x) slot[x] = blocks ? -1 : x;
    if (blocks)
      for (int64_t x = 0; x < n_blocks; ++x) slot[blocks[x]] = x;
    memset(dK_out, 0, sizeof(double) * (size_t)n_blocks * m * d);
    memset(dV_out, 0, sizeof(double) * (size_t)n_blocks * m * d);
    /* (b, g) pairs own disjoint dK/dV blocks, so they run in parallel. */
#pragma omp parallel
    {
      int *keys = (int *)malloc(sizeof(int) * nkeys);
      double *probs = (double *)malloc(sizeof(double) * nkeys);
      double *o = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for collapse(2) schedule(dynamic, 1)
      for (int b = 0; b < B; ++b)
        for (int g = 0; g < Hkv; ++g)
          for (int i = 0; i < Lq; ++i) {
            const int32_t *s = sel + IDX4(b, g, i, 0, Hkv, Lq, Ksel);
            int any = 0;
            for (int p = 0; p < Ksel; ++p)
              if (s[p] >= 0 && slot[((int64_t)b * Hkv + g) * T + s[p]] >= 0) any = 1;
            if (!any) continue;
            const int n = row_keys(&D, sel, b, i, g, keys);
            for (int hh = 0; hh < G; ++hh) {
              const int h = g * G + hh;
              row_forward(&D, Q, K, V, b, i, h, keys, n, probs, o);
              const float *dorow = dO + IDX4(b, i, h, 0, Lq, Hq, d);
              const float *qrow = Q + IDX4(b, i, h, 0, Lq, Hq, d);
              double Dd = 0.0;
              for (int c = 0; c < d; ++c) Dd += (double)dorow[c] * o[c];
              for (int a = 0; a < n; ++a) {
                const int j = keys[a], t = j / m;
                const int64_t sl = slot[((int64_t)b * Hkv + g) * T + t];
                if (sl < 0) continue;
                double dp = 0.0;
                for (int c = 0; c < d; ++c) dp += (double)dorow[c] * (double)V[IDX4(b, j, g, c, Lk, Hkv, d)];
                const double ds = probs[a] * (dp - Dd);
                double *dk = dK_out + (sl * m + (j - t * m)) * d;
                double *dv = dV_out + (sl * m + (j - t * m)) * d;
                for (int c = 0; c < d; ++c) {
                  dv[c] += probs[a] * (double)dorow[c];
                  dk[c] += scale * ds * (double)qrow[c];
                }
              }
            }
          }
      free(keys);
      free(probs);
      free(o);
    }
    free(slot);
  }
}

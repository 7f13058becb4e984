/*
 * ckv_oracle.c -- plain fp64 CPU oracle of CompressKV's prefill-end token selection.
 *
 * TEST INFRASTRUCTURE ONLY. This library is the parity reference for the HIP
 * library. Only the test suite, the smoke check and the benchmark's CPU-baseline
 * leg may load it; the product path never does. It shares no source, header,
 * table or helper with the HIP library.
 *
 * What it computes follows CompressKV (Lin et al., arXiv 2508.02401):
 *   - Token selection, paper Sec. 3.3 ("Token Selection Driven by Semantic
 *     Retrieval Heads"): the attention-score matrices of the chosen heads over
 *     the observation window are summed over the window, pooled along the
 *     token axis, averaged over the chosen heads, and the top-N tokens keep
 *     their K/V pairs.
 *   - Attention scores are the row softmax of Q K^T (Eq. 2), here with the
 *     usual 1/sqrt(d) factor passed in as `scale`.
 *   - Hyper-parameters (window, pooling kernel, average pooling) from the
 *     appendix "More Implementation Details".
 *   - Layer budgets: Algorithm 1 (error-aware layer-adaptive allocation), fed
 *     by the compression error of every layer (Eq. 6-8: decode attention
 *     with the full and the compressed cache, projected by W_O) normalised
 *     over profiling sets (Eq. 10-12).
 *
 * Readings of points the paper leaves open (each is listed in the design notes):
 *   R1 scale = 1/sqrt(d) unless given (Eq. 2 omits it).
 *   R2 window row i (absolute position L-w+i) sees keys 0..L-w+i (causal).
 *   R3 softmax over all visible keys; only the prefix [0, L-w) is ranked.
 *   R4 the window reduction is a sum.
 *   R5 pooling: stride 1, half-width r = kp/2, window clipped to [0, L-w);
 *      average divides by kp (zero padding), max ignores padding.
 *   R6 pool each head, then average the pooled vectors over the heads.
 *   R8 two head scopes: per KV group (each group's chosen heads pick that
 *      group's tokens), or the paper's layer-shared form (the chosen heads of
 *      the whole layer pick one index set for every head; the mean runs over
 *      all chosen heads, each scored against its own group's keys).
 *   R9 the budget B counts the w window tokens, which are always kept; the
 *      other B-w come from the prefix; B >= L keeps every token. With the
 *      keep-window flag off (the *_all functions) the window tokens are not
 *      kept by rule: every column of [0, L) is scored (window columns by the
 *      rows that see them, R2), pooled over [0, L) with R5's padding, and the
 *      best B of all L tokens are kept (B >= 1).
 *   R10 equal scores: the lower token index wins.
 *   R11 retained indices are returned in ascending order.
 *   R13 query head h belongs to KV group h / (H / n_kv).
 *   R14 Algorithm 1's round() is round-half-to-even; R15 its argmax/argmin
 *      ties go to the lowest layer index.
 *   R17 the attention of Eq. 6-7 is decode attention with the scale of R1
 *      and the GQA map of R13, the heads' outputs concatenated head-major;
 *      R18 a one-token output's Frobenius norm is its 2-norm; R19 the decode
 *      queries attend to the prompt's cache only (tokens generated while
 *      profiling are not appended).
 *
 * Everything is fp64 with plain loops; no blocking, fusion or reordering.
 * OpenMP only runs independent KV groups on separate threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define CKVO_OK 0
#define CKVO_EINVAL -1
#define CKVO_EBUDGET -3
#define CKVO_EMASK -4
#define CKVO_ENOMEM -7

#define CKVO_POOL_AVG 0
#define CKVO_POOL_MAX 1

/* One row of attention scores (Eq. 2): softmax over keys 0..n_visible-1 of
 * scale * <q, k_j>.  p[j] = exp(s_j - max s) / sum_j' exp(s_j' - max s). */
int ckvo_attention_row(const double *q, const double *k, int64_t n_visible,
                       int32_t d, double scale, double *p) {
  if (!q || !k || !p || n_visible < 1 || d < 1) return CKVO_EINVAL;
  double m = -INFINITY;
  for (int64_t j = 0; j < n_visible; ++j) {
    double dot = 0.0;
    for (int32_t c = 0; c < d; ++c) dot += q[c] * k[j * (int64_t)d + c];
    p[j] = scale * dot;
    if (p[j] > m) m = p[j];
  }
  double z = 0.0;
  for (int64_t j = 0; j < n_visible; ++j) {
    p[j] = exp(p[j] - m);
    z += p[j];
  }
  for (int64_t j = 0; j < n_visible; ++j) p[j] /= z;
  return CKVO_OK;
}

/* Window sums of one KV group (Sec. 3.3: the attention scores are added up
 * across the window's rows): for each of the n_sel chosen heads, S[h][j] = sum over the w window
 * rows of that head's attention scores on key j, over the full range j in
 * [0, L).  q_sel is [n_sel][w][d], k is [L][d], S is [n_sel][L]. */
int ckvo_window_sums(const double *q_sel, int32_t n_sel, const double *k,
                     int64_t L, int32_t d, int32_t w, double scale, double *S) {
  if (!q_sel || !k || !S || n_sel < 1 || w < 1 || L <= w || d < 1)
    return CKVO_EINVAL;
  double *row = (double *)malloc(sizeof(double) * (size_t)L);
  if (!row) return CKVO_ENOMEM;
  for (int32_t h = 0; h < n_sel; ++h) {
    double *Sh = S + (int64_t)h * L;
    for (int64_t j = 0; j < L; ++j) Sh[j] = 0.0;
    for (int32_t i = 0; i < w; ++i) {
      int64_t n_visible = L - w + i + 1; /* R2: causal inside the window */
      const double *qi = q_sel + ((int64_t)h * w + i) * d;
      ckvo_attention_row(qi, k, n_visible, d, scale, row);
      for (int64_t j = 0; j < n_visible; ++j) Sh[j] += row[j];
    }
  }
  free(row);
  return CKVO_OK;
}

/* The softmax normaliser of every window row (Eq. 2), as its natural log:
 * lse[h][i] = log sum_{j <= L-w+i} exp(scale * <q_i, k_j>), the quantity a
 * causal prefill attention kernel keeps per query row. Computed max-shifted:
 * m + log sum exp(s_j - m). q_sel [n_sel][w][d], k [L][d], lse [n_sel][w]. */
int ckvo_window_lse(const double *q_sel, int32_t n_sel, const double *k, int64_t L, int32_t d,
                    int32_t w, double scale, double *lse) {
  if (!q_sel || !k || !lse || n_sel < 1 || w < 1 || L <= w || d < 1) return CKVO_EINVAL;
  double *row = (double *)malloc(sizeof(double) * (size_t)L);
  if (!row) return CKVO_ENOMEM;
  for (int32_t h = 0; h < n_sel; ++h)
    for (int32_t i = 0; i < w; ++i) {
      const int64_t n_visible = L - w + i + 1; /* R2: causal inside the window */
      const double *qi = q_sel + ((int64_t)h * w + i) * d;
      double m = -INFINITY;
      for (int64_t j = 0; j < n_visible; ++j) {
        double dot = 0.0;
        for (int32_t c = 0; c < d; ++c) dot += qi[c] * k[j * (int64_t)d + c];
        row[j] = scale * dot;
        if (row[j] > m) m = row[j];
      }
      double z = 0.0;
      for (int64_t j = 0; j < n_visible; ++j) z += exp(row[j] - m);
      lse[(int64_t)h * w + i] = m + log(z);
    }
  free(row);
  return CKVO_OK;
}

/* 1-D pooling along the token axis (Sec. 3.3; kernel size and average pooling
 * from the appendix). Stride 1, odd kernel kp, half-width r = kp/2; the
 * neighbourhood of j is [j-r, j+r] clipped to [0, n). */
int ckvo_pool(const double *x, int64_t n, int32_t kp, int32_t mode, double *y) {
  if (!x || !y || n < 1 || kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (mode != CKVO_POOL_AVG && mode != CKVO_POOL_MAX) return CKVO_EINVAL;
  int64_t r = kp / 2;
  for (int64_t j = 0; j < n; ++j) {
    int64_t lo = j - r < 0 ? 0 : j - r;
    int64_t hi = j + r > n - 1 ? n - 1 : j + r;
    if (mode == CKVO_POOL_AVG) {
      double s = 0.0;
      for (int64_t t = lo; t <= hi; ++t) s += x[t];
      y[j] = s / (double)kp; /* zero padding counts toward the kernel */
    } else {
      double m = -INFINITY;
      for (int64_t t = lo; t <= hi; ++t)
        if (x[t] > m) m = x[t];
      y[j] = m;
    }
  }
  return CKVO_OK;
}

typedef struct {
  double score;
  int64_t index;
} ckvo_ranked;

/* Higher score first; equal scores: lower index first (R10). */
static int ckvo_rank_cmp(const void *a, const void *b) {
  const ckvo_ranked *x = (const ckvo_ranked *)a, *y = (const ckvo_ranked *)b;
  if (x->score > y->score) return -1;
  if (x->score < y->score) return 1;
  return (x->index < y->index) ? -1 : (x->index > y->index);
}

static int ckvo_index_cmp(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* Top-N selection (Sec. 3.3: the N tokens with the largest scores are
 * kept), under reading R9: the w window tokens are always
 * kept and count toward the budget, the remaining budget-w tokens are the best
 * of the prefix [0, L-w) by score a[]. Returns the number of retained indices
 * (min(budget, L)) written to idx in ascending order, or a negative code. */
int64_t ckvo_select_tokens(const double *a, int64_t L, int32_t w,
                           int64_t budget, int32_t *idx) {
  if (!a || !idx || w < 1 || L <= w) return CKVO_EINVAL;
  if (budget < w) return CKVO_EBUDGET;
  if (budget >= L) {
    for (int64_t j = 0; j < L; ++j) idx[j] = (int32_t)j;
    return L;
  }
  int64_t Ls = L - w, n_keep = budget - w;
  ckvo_ranked *r = (ckvo_ranked *)malloc(sizeof(ckvo_ranked) * (size_t)Ls);
  if (!r) return CKVO_ENOMEM;
  for (int64_t j = 0; j < Ls; ++j) {
    r[j].score = a[j];
    r[j].index = j;
  }
  qsort(r, (size_t)Ls, sizeof(ckvo_ranked), ckvo_rank_cmp);
  for (int64_t t = 0; t < n_keep; ++t) idx[t] = (int32_t)r[t].index;
  free(r);
  qsort(idx, (size_t)n_keep, sizeof(int32_t), ckvo_index_cmp);
  for (int32_t i = 0; i < w; ++i) idx[n_keep + i] = (int32_t)(Ls + i);
  return budget;
}

/* Retain/evict (Sec. 3.3): the kept tokens' rows, copied byte for byte.
 * src is [L][row_bytes], dst is [n][row_bytes]. */
int ckvo_gather_rows(const void *src, int64_t row_bytes, const int32_t *idx,
                     int64_t n, void *dst) {
  if ((!src || !idx || !dst) && n > 0) return CKVO_EINVAL;
  for (int64_t t = 0; t < n; ++t)
    memcpy((char *)dst + t * row_bytes, (const char *)src + idx[t] * row_bytes,
           (size_t)row_bytes);
  return CKVO_OK;
}

/* The whole selection for one KV group: window sums of the chosen heads,
 * pooling of each head over the prefix (R6), mean over the heads (Sec. 3.3
 * averages the pooled vectors of the chosen heads), then top-N. scores is [L-w]; idx gets
 * min(budget, L) entries. pooled (optional) receives [n_sel][L-w]. */
int64_t ckvo_select_group(const double *q_sel, int32_t n_sel, const double *k,
                          int64_t L, int32_t d, int32_t w, double scale,
                          int32_t pool_mode, int32_t kp, int64_t budget,
                          double *scores, double *pooled, int32_t *idx) {
  if (!q_sel || !k || !scores || n_sel < 1 || w < 1 || L <= w)
    return CKVO_EINVAL;
  if (kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (budget < w) return CKVO_EBUDGET;
  int64_t Ls = L - w;
  double *S = (double *)malloc(sizeof(double) * (size_t)(n_sel * L));
  double *P = (double *)malloc(sizeof(double) * (size_t)Ls);
  if (!S || !P) {
    free(S);
    free(P);
    return CKVO_ENOMEM;
  }
  int rc = ckvo_window_sums(q_sel, n_sel, k, L, d, w, scale, S);
  if (rc == CKVO_OK) {
    for (int64_t j = 0; j < Ls; ++j) scores[j] = 0.0;
    for (int32_t h = 0; h < n_sel; ++h) {
      /* R3: only the prefix columns are pooled and ranked. */
      ckvo_pool(S + (int64_t)h * L, Ls, kp, pool_mode, P);
      if (pooled) memcpy(pooled + (int64_t)h * Ls, P, sizeof(double) * (size_t)Ls);
      for (int64_t j = 0; j < Ls; ++j) scores[j] += P[j];
    }
    for (int64_t j = 0; j < Ls; ++j) scores[j] /= (double)n_sel;
  }
  free(S);
  free(P);
  if (rc != CKVO_OK) return rc;
  if (!idx) return CKVO_OK;
  return ckvo_select_tokens(scores, L, w, budget, idx);
}

/* One layer: every KV group g selects with its own chosen heads (the mask
 * marks chosen query heads; head h belongs to group h / (H / n_kv), R13).
 * q is [H][w][d], k is [n_kv][L][d], scores is [n_kv][L-w], idx is
 * [n_kv][min(budget, L)]. n_threads <= 0 uses the OpenMP default. */
int64_t ckvo_select_layer(const double *q, const uint8_t *mask, int32_t H,
                          int32_t n_kv, const double *k, int64_t L, int32_t d,
                          int32_t w, double scale, int32_t pool_mode, int32_t kp,
                          int64_t budget, double *scores, int32_t *idx,
                          int32_t n_threads) {
  if (!q || !mask || !k || !scores || !idx || H < 1 || n_kv < 1 || H % n_kv)
    return CKVO_EINVAL;
  if (L <= w || w < 1 || d < 1 || kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (budget < w) return CKVO_EBUDGET;
  int32_t G = H / n_kv;
  for (int32_t g = 0; g < n_kv; ++g) {
    int32_t n = 0;
    for (int32_t t = 0; t < G; ++t) n += mask[g * G + t] != 0;
    if (n == 0) return CKVO_EMASK;
  }
  int64_t Ls = L - w, n_ret = budget < L ? budget : L;
  int64_t status = 0;
#ifdef _OPENMP
  if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads)
#endif
  for (int32_t g = 0; g < n_kv; ++g) {
    int32_t n_sel = 0;
    for (int32_t t = 0; t < G; ++t) n_sel += mask[g * G + t] != 0;
    double *q_sel = (double *)malloc(sizeof(double) * (size_t)n_sel * w * d);
    if (!q_sel) {
      status = CKVO_ENOMEM;
      continue;
    }
    int32_t s = 0;
    for (int32_t t = 0; t < G; ++t) {
      int32_t h = g * G + t;
      if (!mask[h]) continue;
      memcpy(q_sel + (int64_t)s * w * d, q + (int64_t)h * w * d,
             sizeof(double) * (size_t)w * d);
      ++s;
    }
    int64_t rc = ckvo_select_group(q_sel, n_sel, k + (int64_t)g * L * d, L, d, w,
                                   scale, pool_mode, kp, budget,
                                   scores + (int64_t)g * Ls, NULL,
                                   idx + (int64_t)g * n_ret);
    if (rc < 0) status = rc;
    free(q_sel);
  }
  return status < 0 ? status : n_ret;
}

/* The paper's own variant of Sec. 3.3: the chosen retrieval heads of the
 * whole layer (marked in mask, from any groups) decide one index set that
 * every attention head of the layer shares. Each chosen head h is scored
 * against the keys of its own group h / (H / n_kv) (R13): its window sums
 * are pooled over the prefix (R6), the pooled vectors of all chosen heads
 * are averaged, and the top-N of that single vector is kept. q is [H][w][d],
 * k is [n_kv][L][d], scores is [L-w], idx gets min(budget, L) entries.
 * n_threads <= 0 uses the OpenMP default (heads run in parallel; their sum is
 * taken afterwards in head order). */
int64_t ckvo_select_layer_shared(const double *q, const uint8_t *mask, int32_t H,
                                 int32_t n_kv, const double *k, int64_t L, int32_t d,
                                 int32_t w, double scale, int32_t pool_mode, int32_t kp,
                                 int64_t budget, double *scores, int32_t *idx,
                                 int32_t n_threads) {
  if (!q || !mask || !k || !scores || !idx || H < 1 || n_kv < 1 || H % n_kv)
    return CKVO_EINVAL;
  if (L <= w || w < 1 || d < 1 || kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (budget < w) return CKVO_EBUDGET;
  int32_t G = H / n_kv, n_chosen = 0;
  for (int32_t h = 0; h < H; ++h) n_chosen += mask[h] != 0;
  if (n_chosen == 0) return CKVO_EMASK;
  int64_t Ls = L - w;
  int32_t *heads = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_chosen);
  double *pooled = (double *)malloc(sizeof(double) * (size_t)n_chosen * (size_t)Ls);
  if (!heads || !pooled) {
    free(heads);
    free(pooled);
    return CKVO_ENOMEM;
  }
  for (int32_t h = 0, c = 0; h < H; ++h)
    if (mask[h]) heads[c++] = h;
  int64_t status = 0;
#ifdef _OPENMP
  if (n_threads <= 0) n_threads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(n_threads)
#endif
  for (int32_t c = 0; c < n_chosen; ++c) {
    int32_t h = heads[c], g = h / G;
    double *S = (double *)malloc(sizeof(double) * (size_t)L);
    if (!S) {
      status = CKVO_ENOMEM;
      continue;
    }
    int rc = ckvo_window_sums(q + (int64_t)h * w * d, 1, k + (int64_t)g * L * d, L, d, w,
                              scale, S);
    if (rc == CKVO_OK) ckvo_pool(S, Ls, kp, pool_mode, pooled + (int64_t)c * Ls);
    else status = rc;
    free(S);
  }
  if (status == 0) {
    for (int64_t j = 0; j < Ls; ++j) {
      double acc = 0.0;
      for (int32_t c = 0; c < n_chosen; ++c) acc += pooled[(int64_t)c * Ls + j];
      scores[j] = acc / (double)n_chosen;
    }
  }
  free(heads);
  free(pooled);
  if (status < 0) return status;
  return ckvo_select_tokens(scores, L, w, budget, idx);
}

/* Selection over the whole prompt, for the keep-window flag off (the
 * alternative of reading R9): the window tokens are not kept by rule but
 * compete with the prefix for the budget. Every column j in [0, L) is scored:
 * a prefix column by all w window rows, a window column L-w+c only by the
 * rows i >= c that see it (the causal window sums of ckvo_window_sums). */

/* The budget tokens of [0, L) with the largest scores a[] (equal scores: the
 * lower index first), written to idx in ascending order; all L when budget >=
 * L. Returns the number written, or a negative code (budget < 1). */
int64_t ckvo_select_tokens_all(const double *a, int64_t L, int64_t budget, int32_t *idx) {
  if (!a || !idx || L < 1) return CKVO_EINVAL;
  if (budget < 1) return CKVO_EBUDGET;
  if (budget >= L) {
    for (int64_t j = 0; j < L; ++j) idx[j] = (int32_t)j;
    return L;
  }
  ckvo_ranked *r = (ckvo_ranked *)malloc(sizeof(ckvo_ranked) * (size_t)L);
  if (!r) return CKVO_ENOMEM;
  for (int64_t j = 0; j < L; ++j) {
    r[j].score = a[j];
    r[j].index = j;
  }
  qsort(r, (size_t)L, sizeof(ckvo_ranked), ckvo_rank_cmp);
  for (int64_t t = 0; t < budget; ++t) idx[t] = (int32_t)r[t].index;
  free(r);
  qsort(idx, (size_t)budget, sizeof(int32_t), ckvo_index_cmp);
  return budget;
}

/* One KV group over the whole prompt: window sums of the chosen heads over
 * [0, L), each pooled over [0, L) (R5's padding at both ends), averaged over
 * the heads (R6), then the budget best tokens of [0, L). scores is [L]; idx
 * gets min(budget, L) entries. */
int64_t ckvo_select_group_all(const double *q_sel, int32_t n_sel, const double *k, int64_t L,
                              int32_t d, int32_t w, double scale, int32_t pool_mode, int32_t kp,
                              int64_t budget, double *scores, int32_t *idx) {
  if (!q_sel || !k || !scores || n_sel < 1 || w < 1 || L <= w) return CKVO_EINVAL;
  if (kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (budget < 1) return CKVO_EBUDGET;
  double *S = (double *)malloc(sizeof(double) * (size_t)(n_sel * L));
  double *P = (double *)malloc(sizeof(double) * (size_t)L);
  if (!S || !P) {
    free(S);
    free(P);
    return CKVO_ENOMEM;
  }
  int rc = ckvo_window_sums(q_sel, n_sel, k, L, d, w, scale, S);
  if (rc == CKVO_OK) {
    for (int64_t j = 0; j < L; ++j) scores[j] = 0.0;
    for (int32_t h = 0; h < n_sel; ++h) {
      ckvo_pool(S + (int64_t)h * L, L, kp, pool_mode, P);
      for (int64_t j = 0; j < L; ++j) scores[j] += P[j];
    }
    for (int64_t j = 0; j < L; ++j) scores[j] /= (double)n_sel;
  }
  free(S);
  free(P);
  if (rc != CKVO_OK) return rc;
  if (!idx) return CKVO_OK;
  return ckvo_select_tokens_all(scores, L, budget, idx);
}

/* The layer-shared selection (see ckvo_select_layer_shared) over the whole
 * prompt: every chosen head's window sums over [0, L) against its own group's
 * keys, pooled over [0, L), averaged over the chosen heads in head order, and
 * the budget best tokens of [0, L). scores is [L]; idx gets min(budget, L)
 * entries. */
int64_t ckvo_select_layer_shared_all(const double *q, const uint8_t *mask, int32_t H,
                                     int32_t n_kv, const double *k, int64_t L, int32_t d,
                                     int32_t w, double scale, int32_t pool_mode, int32_t kp,
                                     int64_t budget, double *scores, int32_t *idx) {
  if (!q || !mask || !k || !scores || !idx || H < 1 || n_kv < 1 || H % n_kv)
    return CKVO_EINVAL;
  if (L <= w || w < 1 || d < 1 || kp < 1 || (kp % 2) == 0) return CKVO_EINVAL;
  if (budget < 1) return CKVO_EBUDGET;
  int32_t G = H / n_kv, n_chosen = 0;
  for (int32_t h = 0; h < H; ++h) n_chosen += mask[h] != 0;
  if (n_chosen == 0) return CKVO_EMASK;
  double *S = (double *)malloc(sizeof(double) * (size_t)L);
  double *P = (double *)malloc(sizeof(double) * (size_t)L);
  if (!S || !P) {
    free(S);
    free(P);
    return CKVO_ENOMEM;
  }
  for (int64_t j = 0; j < L; ++j) scores[j] = 0.0;
  int rc = CKVO_OK;
  for (int32_t h = 0; h < H && rc == CKVO_OK; ++h) {
    if (!mask[h]) continue;
    rc = ckvo_window_sums(q + (int64_t)h * w * d, 1, k + (int64_t)(h / G) * L * d, L, d, w,
                          scale, S);
    if (rc != CKVO_OK) break;
    ckvo_pool(S, L, kp, pool_mode, P);
    for (int64_t j = 0; j < L; ++j) scores[j] += P[j];
  }
  for (int64_t j = 0; j < L; ++j) scores[j] /= (double)n_chosen;
  free(S);
  free(P);
  if (rc != CKVO_OK) return rc;
  return ckvo_select_tokens_all(scores, L, budget, idx);
}

/* Decode attention (Eq. 2 for one query per head): head h attends to the
 * cache of its group g = h / (H / n_kv) (R13), out[h] = sum_j p_j v[g][j]
 * with p the softmax over all n cached keys of scale * <q[h], k[g][j]>.
 * q is [H][d], k and v are [n_kv][n][d], out is [H][d]. */
int ckvo_decode_attention(const double *q, const double *k, const double *v, int32_t H,
                          int32_t n_kv, int64_t n, int32_t d, double scale, double *out) {
  if (!q || !k || !v || !out || H < 1 || n_kv < 1 || H % n_kv || n < 1 || d < 1)
    return CKVO_EINVAL;
  int32_t G = H / n_kv;
  double *p = (double *)malloc(sizeof(double) * (size_t)n);
  if (!p) return CKVO_ENOMEM;
  for (int32_t h = 0; h < H; ++h) {
    const double *kg = k + (int64_t)(h / G) * n * d;
    const double *vg = v + (int64_t)(h / G) * n * d;
    ckvo_attention_row(q + (int64_t)h * d, kg, n, d, scale, p);
    for (int32_t c = 0; c < d; ++c) {
      double acc = 0.0;
      for (int64_t j = 0; j < n; ++j) acc += p[j] * vg[j * d + c];
      out[(int64_t)h * d + c] = acc;
    }
  }
  free(p);
  return CKVO_OK;
}

/* Compression error of one layer (Eq. 6-8): for every decoding step t the
 * attention outputs of all heads, concatenated head-major into an H*d vector,
 * are taken with the full cache and with the compressed cache and projected
 * by W_O ([D][H*d], row-major); the step's term is
 *   || W_O (A_comp,t - A_full,t) || / (|| W_O A_full,t || + eps)
 * (the Frobenius norm of a one-token output is its 2-norm), and e is their
 * sum over the T steps. q_dec is [T][H][d]; k, v [n_kv][L][d]; kc, vc
 * [n_kv][n_c][d]. ratio (optional) receives the T terms. */
int ckvo_layer_error(const double *q_dec, int32_t T, int32_t H, int32_t n_kv, int32_t d,
                     const double *k, const double *v, int64_t L, const double *kc,
                     const double *vc, int64_t n_c, const double *w_o, int32_t D,
                     double scale, double eps, double *ratio, double *e) {
  if (!q_dec || !k || !v || !kc || !vc || !w_o || !e || T < 1 || D < 1) return CKVO_EINVAL;
  int64_t hd = (int64_t)H * d;
  double *af = (double *)malloc(sizeof(double) * (size_t)hd);
  double *ac = (double *)malloc(sizeof(double) * (size_t)hd);
  if (!af || !ac) {
    free(af);
    free(ac);
    return CKVO_ENOMEM;
  }
  double total = 0.0;
  int rc = CKVO_OK;
  for (int32_t t = 0; t < T && rc == CKVO_OK; ++t) {
    const double *qt = q_dec + (int64_t)t * hd;
    rc = ckvo_decode_attention(qt, k, v, H, n_kv, L, d, scale, af);
    if (rc == CKVO_OK) rc = ckvo_decode_attention(qt, kc, vc, H, n_kv, n_c, d, scale, ac);
    if (rc != CKVO_OK) break;
    double num = 0.0, den = 0.0;
    for (int32_t r = 0; r < D; ++r) {
      const double *wr = w_o + (int64_t)r * hd;
      double yf = 0.0, yd = 0.0;
      for (int64_t c = 0; c < hd; ++c) {
        yf += wr[c] * af[c];
        yd += wr[c] * (ac[c] - af[c]);
      }
      num += yd * yd;
      den += yf * yf;
    }
    double term = sqrt(num) / (sqrt(den) + eps);
    if (ratio) ratio[t] = term;
    total += term;
  }
  free(af);
  free(ac);
  if (rc != CKVO_OK) return rc;
  *e = total;
  return CKVO_OK;
}

/* Normalised layer errors from profiling sets (Eq. 10-12): e is
 * [n_sets][n_layers]; each set is L1-normalised over its layers, the sets
 * are averaged, and the average is L1-normalised again into e_tilde. */
int ckvo_normalize_errors(const double *e, int32_t n_sets, int32_t n_layers, double *e_tilde) {
  if (!e || !e_tilde || n_sets < 1 || n_layers < 1) return CKVO_EINVAL;
  for (int32_t l = 0; l < n_layers; ++l) e_tilde[l] = 0.0;
  for (int32_t s = 0; s < n_sets; ++s) {
    double sum = 0.0;
    for (int32_t l = 0; l < n_layers; ++l) sum += e[(int64_t)s * n_layers + l];
    if (!(sum > 0.0)) return CKVO_EINVAL;
    for (int32_t l = 0; l < n_layers; ++l)
      e_tilde[l] += e[(int64_t)s * n_layers + l] / sum / (double)n_sets;
  }
  double sum = 0.0;
  for (int32_t l = 0; l < n_layers; ++l) sum += e_tilde[l];
  for (int32_t l = 0; l < n_layers; ++l) e_tilde[l] /= sum;
  return CKVO_OK;
}

/* Algorithm 1 (Appendix B.1, error-aware layer-adaptive cache allocation),
 * as a proportional share followed by a water-fill of the gap it leaves.
 *
 * Share: every layer gets the floor m plus its part of what is left,
 * R = total - n*m, in proportion to its normalised error e[i] (rounded half to
 * even, R14), clipped to [m, M].
 *
 * Gap: the clipped budgets may miss the total. The algorithm closes the gap
 * one token at a time, giving each missing token to the layer of largest error
 * that is still below M, or taking each extra token from the layer of smallest
 * error still above m (R15: equal errors go to the lower layer). The errors do
 * not change meanwhile, so that rule visits the layers in one fixed order (by
 * error, then by index) and fills or drains each to its bound before it moves
 * to the next; that order is what is computed here.
 *
 * Returns 0 when the budgets sum to total, CKVO_EBUDGET when every layer hit
 * its bound first (B then holds the budgets as far as they got). */
static int alloc_before(const double *e, int32_t a, int32_t b, int largest_first) {
  if (e[a] != e[b]) return largest_first ? e[a] > e[b] : e[a] < e[b];
  return a < b;
}

int ckvo_allocate_budgets(const double *e, int32_t n, int64_t total, int64_t m,
                          int64_t M, int64_t *B) {
  if (!e || !B || n < 1 || m < 0 || M < m) return CKVO_EINVAL;
  const int64_t R = total - (int64_t)n * m;
  int64_t gap = total;
  for (int32_t i = 0; i < n; ++i) {
    const int64_t b = m + (int64_t)nearbyint(e[i] * (double)R);
    B[i] = b < m ? m : (b > M ? M : b);
    gap -= B[i];
  }
  if (gap == 0) return CKVO_OK;
  const int grow = gap > 0;
  int32_t *order = (int32_t *)malloc((size_t)n * sizeof(int32_t));
  if (!order) return CKVO_ENOMEM;
  for (int32_t i = 0; i < n; ++i) {  /* insertion sort into visiting order */
    int32_t k = i;
    while (k > 0 && alloc_before(e, i, order[k - 1], grow)) {
      order[k] = order[k - 1];
      --k;
    }
    order[k] = i;
  }
  for (int32_t k = 0; k < n && gap != 0; ++k) {
    const int32_t i = order[k];
    const int64_t room = grow ? M - B[i] : B[i] - m;
    const int64_t need = grow ? gap : -gap;
    const int64_t moved = need < room ? need : room;
    B[i] += grow ? moved : -moved;
    gap -= grow ? moved : -moved;
  }
  free(order);
  return gap == 0 ? CKVO_OK : CKVO_EBUDGET;
}

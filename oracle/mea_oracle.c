/*
 * Float64 CPU oracle for exact dense softmax attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header or constant with the HIP
 * kernels.
 *
 * What it computes (Rabe & Staats, "Self-attention Does Not Need O(n^2)
 * Memory", arXiv 2112.05682):
 *   - Section 1, attention definition: for one query q and keys/values
 *     k_j, v_j, the scores are s_j = dot(q, k_j), the weights are the softmax
 *     of the scores, and the result is the weight-averaged value vector.
 *   - Section 4 (implementation): the query is divided by sqrt(d) before the
 *     dot product; here that factor is an explicit `scale` argument.
 *   - Section 3 (numerical stability): the softmax is evaluated after
 *     subtracting the largest score of the row, which leaves the weights
 *     unchanged in exact arithmetic.
 *
 * Three independent forward forms are provided so that they can be checked
 * against one another:
 *   direct  - the Section 1 definition, normalising the weights first;
 *   lazy    - the Section 3 single-pass update (running max m*, running
 *             numerator v*, running denominator s*, one division at the end);
 *   chunked - the Section 4 scheme: independent per-chunk summaries
 *             (sum of e^{s-m_c} v, sum of e^{s-m_c}, m_c), rescaled to the
 *             largest chunk max, summed, then divided; queries are processed
 *             in chunks written straight into the output.
 *
 * Backward (hand-derived; the paper differentiates with jax.grad through a
 * checkpointed chunk summary, Section 5.2): with w_ij = softmax_j(s_ij),
 *   dV_j  = sum_i w_ij dO_i
 *   dw_ij = dot(dO_i, v_j)
 *   D_i   = sum_j w_ij dw_ij
 *   dS_ij = w_ij (dw_ij - D_i)
 *   dQ_i  = scale sum_j dS_ij k_j
 *   dK_j  = scale sum_i dS_ij q_i
 * The row maximum is a constant for the gradient (Section 4 stops the
 * gradient through it); the result does not depend on it.
 *
 * Readings where the paper is silent:
 *   - masking: `causal` means key j is visible to query i iff j <= i
 *     (aligned at the top-left, so key 0 is always visible and no row is
 *     empty, also when n_q != n_k);
 *   - key padding: batch b sees only keys j < kv_len[b] (clamped to
 *     [0, n_k]; a NULL kv_len means all n_k), on top of the causal mask; a
 *     row that sees no key has o = 0, lse = -inf and zero gradients, and a
 *     key no row sees has zero dK and dV (the sums over an empty set);
 *   - lse is the natural-log log-sum-exp of the scaled scores of a row;
 *   - layout: contiguous [B, H, n, width], feature index innermost; q and k
 *     have d features, v, o and the upstream gradient d_v (the definition
 *     does not tie the value width to the key width).
 *
 * All sums run in ascending index order in plain double precision.  Rows
 * are distributed over OpenMP threads; each row is computed by one thread.
 *
 * Every entry point returns 0 on success, 1 on an invalid argument and 2 on
 * an allocation failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL 1
#define ORACLE_ENOMEM 2

/* Number of keys visible to query row i: a prefix of the keys, the first
 * n_valid of them (key padding) and, causal, at most the first i + 1. */
static int64_t visible_keys(int64_t i, int64_t n_k, int causal, int64_t n_valid) {
  int64_t n = n_k;
  if (causal && i + 1 < n) n = i + 1;
  return n < n_valid ? n : n_valid;
}

/* Valid keys of (batch, head) slice bh: kv_len[b] clamped to [0, n_k]. */
static int64_t slice_valid(const int64_t* kv_len, int64_t bh, int64_t heads,
                           int64_t n_k) {
  if (!kv_len) return n_k;
  const int64_t l = kv_len[bh / heads];
  return l < 0 ? 0 : (l > n_k ? n_k : l);
}

static double dot(const double* a, const double* b, int64_t d) {
  double acc = 0.0;
  for (int64_t t = 0; t < d; ++t) acc += a[t] * b[t];
  return acc;
}

static int dims_ok(int64_t n_q, int64_t n_k, int64_t d, int64_t d_v) {
  return n_q >= 1 && n_k >= 1 && d >= 1 && d_v >= 1;
}

int mea_oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads used by the calling thread's later parallel loops (n >= 1); for
 * timing the oracle on one core and on all of them in one process. */
void mea_oracle_set_num_threads(int n) {
#ifdef _OPENMP
  omp_set_num_threads(n > 0 ? n : 1);
#else
  (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Direct form (Section 1 definition with the max subtraction of Section 3). */
/* ------------------------------------------------------------------------ */

/* One query row.  s is scratch of length >= n_vis. */
static void direct_row(const double* qi, const double* k, const double* v,
                       int64_t n_vis, int64_t d, int64_t d_v, double scale,
                       double* s, double* out, double* lse) {
  double m = -INFINITY;
  for (int64_t j = 0; j < n_vis; ++j) {
    s[j] = scale * dot(qi, k + j * d, d);
    if (s[j] > m) m = s[j];
  }
  double l = 0.0;
  for (int64_t j = 0; j < n_vis; ++j) l += exp(s[j] - m);
  for (int64_t t = 0; t < d_v; ++t) out[t] = 0.0;
  for (int64_t j = 0; j < n_vis; ++j) {
    const double w = exp(s[j] - m) / l; /* normalised weight, as defined */
    const double* vj = v + j * d_v;
    for (int64_t t = 0; t < d_v; ++t) out[t] += w * vj[t];
  }
  *lse = m + log(l);
}

/* Per-thread scratch: one block of `per_thread` doubles for each OpenMP
 * thread, allocated before the parallel region so that an allocation failure
 * is reported before any work starts. */
static double* thread_scratch(int64_t per_thread) {
  const int64_t n = (int64_t)mea_oracle_num_threads() * per_thread;
  return (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
}

static int thread_id(void) {
#ifdef _OPENMP
  return omp_get_thread_num();
#else
  return 0;
#endif
}

/* One (batch, head) slice, a subset of query rows.  o_rows is [n_rows, d],
 * lse_rows is [n_rows] (either may be NULL). */
int mea_oracle_fwd_rows(int64_t n_q, int64_t n_k, int64_t d, int64_t d_v,
                        const double* q, const double* k, const double* v,
                        double scale, int causal, int64_t n_valid,
                        const int64_t* rows, int64_t n_rows, double* o_rows,
                        double* lse_rows) {
  if (!dims_ok(n_q, n_k, d, d_v) || n_rows < 0 || !q || !k || !v || !rows ||
      n_valid < 0 || n_valid > n_k)
    return ORACLE_EINVAL;
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= n_q) return ORACLE_EINVAL;
  const int64_t per_thread = n_k + d_v;
  double* scratch = thread_scratch(per_thread);
  if (!scratch) return ORACLE_ENOMEM;
#pragma omp parallel for schedule(dynamic, 8)
  for (int64_t r = 0; r < n_rows; ++r) {
    double* s = scratch + thread_id() * per_thread;
    double* out = s + n_k;
    const int64_t i = rows[r];
    double lse;
    direct_row(q + i * d, k, v, visible_keys(i, n_k, causal, n_valid), d, d_v,
               scale, s, out, &lse);
    if (o_rows) memcpy(o_rows + r * d_v, out, sizeof(double) * (size_t)d_v);
    if (lse_rows) lse_rows[r] = lse;
  }
  free(scratch);
  return ORACLE_OK;
}

/* Full [B, H, n_q, d] forward, direct form. */
int mea_oracle_fwd(int64_t batch, int64_t heads, int64_t n_q, int64_t n_k,
                   int64_t d, int64_t d_v, const double* q, const double* k,
                   const double* v, double scale, int causal,
                   const int64_t* kv_len, double* o, double* lse) {
  if (batch < 1 || heads < 1 || !dims_ok(n_q, n_k, d, d_v) || !o || !lse)
    return ORACLE_EINVAL;
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_q);
  if (!rows) return ORACLE_ENOMEM;
  for (int64_t i = 0; i < n_q; ++i) rows[i] = i;
  int err = ORACLE_OK;
  for (int64_t bh = 0; bh < batch * heads && err == ORACLE_OK; ++bh) {
    err = mea_oracle_fwd_rows(n_q, n_k, d, d_v, q + bh * n_q * d,
                              k + bh * n_k * d, v + bh * n_k * d_v, scale,
                              causal, slice_valid(kv_len, bh, heads, n_k), rows,
                              n_q, o + bh * n_q * d_v, lse + bh * n_q);
  }
  free(rows);
  return err;
}

/* ------------------------------------------------------------------------ */
/* Lazy form (Section 3): one pass over the keys in order, keeping a running  */
/* maximum m*, a running numerator v* and a running denominator s*.          */
/* ------------------------------------------------------------------------ */

static void lazy_row(const double* qi, const double* k, const double* v,
                     int64_t n_vis, int64_t d, int64_t d_v, double scale,
                     double* vstar, double* out, double* lse) {
  double sstar = 0.0;
  double mstar = -INFINITY;
  for (int64_t t = 0; t < d_v; ++t) vstar[t] = 0.0;
  for (int64_t j = 0; j < n_vis; ++j) {
    const double sj = scale * dot(qi, k + j * d, d);
    const double mi = (sj > mstar) ? sj : mstar;
    const double old_factor = exp(mstar - mi); /* e^{-inf} = 0 on key 0 */
    const double new_factor = exp(sj - mi);
    const double* vj = v + j * d_v;
    for (int64_t t = 0; t < d_v; ++t)
      vstar[t] = vstar[t] * old_factor + vj[t] * new_factor;
    sstar = sstar * old_factor + new_factor;
    mstar = mi;
  }
  if (n_vis == 0) { /* no visible key: the empty sums give o = 0 */
    for (int64_t t = 0; t < d_v; ++t) out[t] = 0.0;
    *lse = -INFINITY;
    return;
  }
  for (int64_t t = 0; t < d_v; ++t) out[t] = vstar[t] / sstar;
  *lse = mstar + log(sstar);
}

int mea_oracle_fwd_lazy(int64_t batch, int64_t heads, int64_t n_q,
                        int64_t n_k, int64_t d, int64_t d_v, const double* q,
                        const double* k, const double* v, double scale,
                        int causal, const int64_t* kv_len, double* o,
                        double* lse) {
  if (batch < 1 || heads < 1 || !dims_ok(n_q, n_k, d, d_v) || !q || !k ||
      !v || !o || !lse)
    return ORACLE_EINVAL;
  double* scratch = thread_scratch(d_v);
  if (!scratch) return ORACLE_ENOMEM;
  for (int64_t bh = 0; bh < batch * heads; ++bh) {
    const double* qh = q + bh * n_q * d;
    const double* kh = k + bh * n_k * d;
    const double* vh = v + bh * n_k * d_v;
    const int64_t n_valid = slice_valid(kv_len, bh, heads, n_k);
#pragma omp parallel for schedule(dynamic, 8)
    for (int64_t i = 0; i < n_q; ++i)
      lazy_row(qh + i * d, kh, vh, visible_keys(i, n_k, causal, n_valid), d,
               d_v, scale, scratch + thread_id() * d_v,
               o + (bh * n_q + i) * d_v, lse + bh * n_q + i);
  }
  free(scratch);
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Chunked form (Section 4): queries in chunks, keys in chunks, one summary  */
/* per key chunk, then a rescale to the largest chunk maximum and one        */
/* division.  Chunks are true ragged ranges over the visible keys.           */
/* ------------------------------------------------------------------------ */

/* Summaries of the visible keys of one query row, chunk by chunk:
 *   values[c][t] = sum_{j in c} e^{s_j - m_c} v_j[t]
 *   weights[c]   = sum_{j in c} e^{s_j - m_c}
 *   maxes[c]     = max_{j in c} s_j                                         */
static void chunk_summaries(const double* qi, const double* k, const double* v,
                            int64_t n_vis, int64_t d, int64_t d_v, double scale,
                            int64_t key_chunk, double* values, double* weights,
                            double* maxes, double* s) {
  int64_t c = 0;
  for (int64_t j0 = 0; j0 < n_vis; j0 += key_chunk, ++c) {
    const int64_t j1 = (j0 + key_chunk < n_vis) ? j0 + key_chunk : n_vis;
    double m = -INFINITY;
    for (int64_t j = j0; j < j1; ++j) {
      s[j - j0] = scale * dot(qi, k + j * d, d);
      if (s[j - j0] > m) m = s[j - j0];
    }
    double* vc = values + c * d_v;
    for (int64_t t = 0; t < d_v; ++t) vc[t] = 0.0;
    double wsum = 0.0;
    for (int64_t j = j0; j < j1; ++j) {
      const double e = exp(s[j - j0] - m);
      const double* vj = v + j * d_v;
      for (int64_t t = 0; t < d_v; ++t) vc[t] += e * vj[t];
      wsum += e;
    }
    weights[c] = wsum;
    maxes[c] = m;
  }
}

/* Rescale the chunk summaries to the largest chunk maximum, add them up and
 * divide: the combine step of Section 4. */
static void combine_summaries(int64_t n_chunks, int64_t d, double* values,
                              double* weights, const double* maxes,
                              double* out, double* lse) {
  if (n_chunks == 0) { /* no visible key: the empty sums give o = 0 */
    for (int64_t t = 0; t < d; ++t) out[t] = 0.0;
    *lse = -INFINITY;
    return;
  }
  double global_max = -INFINITY;
  for (int64_t c = 0; c < n_chunks; ++c)
    if (maxes[c] > global_max) global_max = maxes[c];
  for (int64_t c = 0; c < n_chunks; ++c) {
    const double f = exp(maxes[c] - global_max);
    for (int64_t t = 0; t < d; ++t) values[c * d + t] *= f;
    weights[c] *= f;
  }
  double all_weights = 0.0;
  for (int64_t t = 0; t < d; ++t) out[t] = 0.0;
  for (int64_t c = 0; c < n_chunks; ++c) {
    for (int64_t t = 0; t < d; ++t) out[t] += values[c * d + t];
    all_weights += weights[c];
  }
  for (int64_t t = 0; t < d; ++t) out[t] /= all_weights;
  *lse = global_max + log(all_weights);
}

int mea_oracle_fwd_chunked(int64_t batch, int64_t heads, int64_t n_q,
                           int64_t n_k, int64_t d, int64_t d_v, const double* q,
                           const double* k, const double* v, double scale,
                           int causal, const int64_t* kv_len,
                           int64_t query_chunk, int64_t key_chunk, double* o,
                           double* lse) {
  if (batch < 1 || heads < 1 || !dims_ok(n_q, n_k, d, d_v) || query_chunk < 1 ||
      key_chunk < 1 || !q || !k || !v || !o || !lse)
    return ORACLE_EINVAL;
  const int64_t max_chunks = (n_k + key_chunk - 1) / key_chunk;
  const int64_t chunk_len = key_chunk < n_k ? key_chunk : n_k;
  /* values [max_chunks, d_v] | weights [max_chunks] | maxes [max_chunks] | s */
  const int64_t per_thread = max_chunks * (d_v + 2) + chunk_len;
  double* scratch = thread_scratch(per_thread);
  if (!scratch) return ORACLE_ENOMEM;
  for (int64_t bh = 0; bh < batch * heads; ++bh) {
    const double* qh = q + bh * n_q * d;
    const double* kh = k + bh * n_k * d;
    const double* vh = v + bh * n_k * d_v;
    const int64_t n_valid = slice_valid(kv_len, bh, heads, n_k);
    /* Outer loop over query chunks; each chunk's rows go straight to o. */
    for (int64_t i0 = 0; i0 < n_q; i0 += query_chunk) {
      const int64_t i1 = (i0 + query_chunk < n_q) ? i0 + query_chunk : n_q;
#pragma omp parallel for schedule(dynamic, 4)
      for (int64_t i = i0; i < i1; ++i) {
        double* values = scratch + thread_id() * per_thread;
        double* weights = values + max_chunks * d_v;
        double* maxes = weights + max_chunks;
        double* s = maxes + max_chunks;
        const int64_t n_vis = visible_keys(i, n_k, causal, n_valid);
        const int64_t n_chunks = (n_vis + key_chunk - 1) / key_chunk;
        chunk_summaries(qh + i * d, kh, vh, n_vis, d, d_v, scale, key_chunk,
                        values, weights, maxes, s);
        combine_summaries(n_chunks, d_v, values, weights, maxes,
                          o + (bh * n_q + i) * d_v, lse + bh * n_q + i);
      }
    }
  }
  free(scratch);
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Backward (hand-derived gradients of o_i = sum_j softmax_j(s_ij) v_j).     */
/* ------------------------------------------------------------------------ */

/* Softmax statistics of one row: max m and denominator l = sum e^{s_j - m},
 * plus D = sum_j w_j dot(dO_i, v_j). */
static void row_stats(const double* qi, const double* doi, const double* k,
                      const double* v, int64_t n_vis, int64_t d, int64_t d_v,
                      double scale, double* s, double* m_out, double* l_out,
                      double* D_out) {
  double m = -INFINITY;
  for (int64_t j = 0; j < n_vis; ++j) {
    s[j] = scale * dot(qi, k + j * d, d);
    if (s[j] > m) m = s[j];
  }
  double l = 0.0;
  for (int64_t j = 0; j < n_vis; ++j) l += exp(s[j] - m);
  double D = 0.0;
  for (int64_t j = 0; j < n_vis; ++j) {
    const double w = exp(s[j] - m) / l;
    D += w * dot(doi, v + j * d_v, d_v);
  }
  *m_out = m;
  *l_out = l;
  *D_out = D;
}

/* dQ for a subset of query rows of one (batch, head) slice.  dq_rows is
 * [n_rows, d]. */
int mea_oracle_bwd_dq_rows(int64_t n_q, int64_t n_k, int64_t d, int64_t d_v,
                           const double* q, const double* k, const double* v,
                           const double* dout, double scale, int causal,
                           int64_t n_valid, const int64_t* rows,
                           int64_t n_rows, double* dq_rows) {
  if (!dims_ok(n_q, n_k, d, d_v) || n_rows < 0 || !q || !k || !v || !dout ||
      !rows || !dq_rows || n_valid < 0 || n_valid > n_k)
    return ORACLE_EINVAL;
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= n_q) return ORACLE_EINVAL;
  double* scratch = thread_scratch(n_k);
  if (!scratch) return ORACLE_ENOMEM;
#pragma omp parallel for schedule(dynamic, 8)
  for (int64_t r = 0; r < n_rows; ++r) {
    double* s = scratch + thread_id() * n_k;
    const int64_t i = rows[r];
    const double* qi = q + i * d;
    const double* doi = dout + i * d_v;
    const int64_t n_vis = visible_keys(i, n_k, causal, n_valid);
    double m, l, D;
    row_stats(qi, doi, k, v, n_vis, d, d_v, scale, s, &m, &l, &D);
    double* dqi = dq_rows + r * d;
    for (int64_t t = 0; t < d; ++t) dqi[t] = 0.0;
    for (int64_t j = 0; j < n_vis; ++j) {
      const double w = exp(s[j] - m) / l;
      const double ds = w * (dot(doi, v + j * d_v, d_v) - D);
      const double* kj = k + j * d;
      for (int64_t t = 0; t < d; ++t) dqi[t] += ds * kj[t];
    }
    for (int64_t t = 0; t < d; ++t) dqi[t] *= scale;
  }
  free(scratch);
  return ORACLE_OK;
}

/* dK and dV for a subset of key rows of one (batch, head) slice.  Needs the
 * softmax statistics of every query row first.  dk_rows, dv_rows are
 * [n_keys, d] (either may be NULL). */
int mea_oracle_bwd_dkdv_keys(int64_t n_q, int64_t n_k, int64_t d, int64_t d_v,
                             const double* q, const double* k, const double* v,
                             const double* dout, double scale, int causal,
                             int64_t n_valid, const int64_t* keys,
                             int64_t n_keys, double* dk_rows, double* dv_rows) {
  if (!dims_ok(n_q, n_k, d, d_v) || n_keys < 0 || !q || !k || !v || !dout ||
      !keys || n_valid < 0 || n_valid > n_k)
    return ORACLE_EINVAL;
  for (int64_t r = 0; r < n_keys; ++r)
    if (keys[r] < 0 || keys[r] >= n_k) return ORACLE_EINVAL;
  double* m = (double*)malloc(sizeof(double) * (size_t)n_q);
  double* l = (double*)malloc(sizeof(double) * (size_t)n_q);
  double* D = (double*)malloc(sizeof(double) * (size_t)n_q);
  if (!m || !l || !D) {
    free(m);
    free(l);
    free(D);
    return ORACLE_ENOMEM;
  }
  double* scratch = thread_scratch(n_k);
  if (!scratch) {
    free(m);
    free(l);
    free(D);
    return ORACLE_ENOMEM;
  }
  /* Pass 1: per-query softmax statistics. */
#pragma omp parallel for schedule(dynamic, 8)
  for (int64_t i = 0; i < n_q; ++i)
    row_stats(q + i * d, dout + i * d_v, k, v,
              visible_keys(i, n_k, causal, n_valid), d, d_v, scale,
              scratch + thread_id() * n_k, &m[i], &l[i], &D[i]);
  free(scratch);
  /* Pass 2: per requested key, sum over the queries that see it. */
#pragma omp parallel for schedule(dynamic, 8)
  for (int64_t r = 0; r < n_keys; ++r) {
    const int64_t j = keys[r];
    const double* kj = k + j * d;
    const double* vj = v + j * d_v;
    double* dkj = dk_rows ? dk_rows + r * d : NULL;
    double* dvj = dv_rows ? dv_rows + r * d_v : NULL;
    if (dkj) for (int64_t t = 0; t < d; ++t) dkj[t] = 0.0;
    if (dvj) for (int64_t t = 0; t < d_v; ++t) dvj[t] = 0.0;
    /* query i sees key j iff j < n_valid and, causal, j <= i */
    const int64_t i_first = j >= n_valid ? n_q : (causal ? j : 0);
    for (int64_t i = i_first; i < n_q; ++i) {
      const double* qi = q + i * d;
      const double* doi = dout + i * d_v;
      const double w = exp(scale * dot(qi, kj, d) - m[i]) / l[i];
      if (dvj) for (int64_t t = 0; t < d_v; ++t) dvj[t] += w * doi[t];
      if (dkj) {
        const double ds = w * (dot(doi, vj, d_v) - D[i]);
        for (int64_t t = 0; t < d; ++t) dkj[t] += ds * qi[t];
      }
    }
    if (dkj) for (int64_t t = 0; t < d; ++t) dkj[t] *= scale;
  }
  free(m);
  free(l);
  free(D);
  return ORACLE_OK;
}

/* Full [B, H, n, d] backward. */
int mea_oracle_bwd(int64_t batch, int64_t heads, int64_t n_q, int64_t n_k,
                   int64_t d, int64_t d_v, const double* q, const double* k,
                   const double* v, const double* dout, double scale,
                   int causal, const int64_t* kv_len, double* dq, double* dk,
                   double* dv) {
  if (batch < 1 || heads < 1 || !dims_ok(n_q, n_k, d, d_v) || !dq || !dk || !dv)
    return ORACLE_EINVAL;
  const int64_t n_max = n_q > n_k ? n_q : n_k;
  int64_t* idx = (int64_t*)malloc(sizeof(int64_t) * (size_t)n_max);
  if (!idx) return ORACLE_ENOMEM;
  for (int64_t i = 0; i < n_max; ++i) idx[i] = i;
  int err = ORACLE_OK;
  for (int64_t bh = 0; bh < batch * heads && err == ORACLE_OK; ++bh) {
    const double* qh = q + bh * n_q * d;
    const double* kh = k + bh * n_k * d;
    const double* vh = v + bh * n_k * d_v;
    const double* doh = dout + bh * n_q * d_v;
    const int64_t n_valid = slice_valid(kv_len, bh, heads, n_k);
    err = mea_oracle_bwd_dq_rows(n_q, n_k, d, d_v, qh, kh, vh, doh, scale,
                                 causal, n_valid, idx, n_q, dq + bh * n_q * d);
    if (err == ORACLE_OK)
      err = mea_oracle_bwd_dkdv_keys(n_q, n_k, d, d_v, qh, kh, vh, doh, scale,
                                     causal, n_valid, idx, n_k,
                                     dk + bh * n_k * d, dv + bh * n_k * d_v);
  }
  free(idx);
  return err;
}

/*
 * Native driver of the float64 oracle for the sanitizer build (test
 * infrastructure): calls every entry point on small seeded inputs -- causal
 * on and off, per-batch valid key lengths, a value width different from the
 * key width, ragged chunk sizes -- and checks that the three forward forms
 * agree, that the row and key subsets reproduce the full functions bit for
 * bit, and that invalid arguments are rejected.  Built with
 * -fsanitize=address,undefined, so any out-of-bounds access or undefined
 * operation on these paths fails the run.  Exit status = number of failures.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int mea_oracle_fwd(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, const double*,
                   const double*, const double*, double, int, const int64_t*, double*, double*);
int mea_oracle_fwd_lazy(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, const double*,
                        const double*, const double*, double, int, const int64_t*, double*, double*);
int mea_oracle_fwd_chunked(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, const double*,
                           const double*, const double*, double, int, const int64_t*, int64_t,
                           int64_t, double*, double*);
int mea_oracle_bwd(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, const double*,
                   const double*, const double*, const double*, double, int, const int64_t*,
                   double*, double*, double*);
int mea_oracle_fwd_rows(int64_t, int64_t, int64_t, int64_t, const double*, const double*,
                        const double*, double, int, int64_t, const int64_t*, int64_t, double*,
                        double*);
int mea_oracle_bwd_dq_rows(int64_t, int64_t, int64_t, int64_t, const double*, const double*,
                           const double*, const double*, double, int, int64_t, const int64_t*,
                           int64_t, double*);
int mea_oracle_bwd_dkdv_keys(int64_t, int64_t, int64_t, int64_t, const double*, const double*,
                             const double*, const double*, double, int, int64_t, const int64_t*,
                             int64_t, double*, double*);

static int failures = 0;
#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      fprintf(stderr, __VA_ARGS__);                        \
      fprintf(stderr, "\n");                               \
      ++failures;                                          \
    }                                                      \
  } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform_pm1(void) { /* xorshift64*, mapped to [-1, 1) */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  const uint64_t x = rng_state * 0x2545F4914F6CDD1Dull;
  return (double)(x >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}
static double* filled(size_t n, double amp) {
  double* p = (double*)malloc(sizeof(double) * (n ? n : 1));
  for (size_t i = 0; i < n; ++i) p[i] = amp * uniform_pm1();
  return p;
}
static double max_rel(const double* a, const double* b, size_t n) {
  double top = 0.0, err = 0.0;
  for (size_t i = 0; i < n; ++i) {
    if (isinf(a[i]) && isinf(b[i]) && (a[i] > 0) == (b[i] > 0)) continue;
    top = fmax(top, fabs(b[i]));
    err = fmax(err, fabs(a[i] - b[i]));
  }
  return top > 0 ? err / top : err;
}

static void one_case(int64_t B, int64_t H, int64_t nq, int64_t nk, int64_t d, int64_t dv,
                     int causal, const int64_t* kv_len, double amp) {
  const double scale = 1.0 / sqrt((double)d);
  const size_t nqd = (size_t)(B * H * nq * d), nkd = (size_t)(B * H * nk * d);
  const size_t nkv = (size_t)(B * H * nk * dv), nqv = (size_t)(B * H * nq * dv);
  const size_t nr = (size_t)(B * H * nq);
  double *q = filled(nqd, amp), *k = filled(nkd, amp), *v = filled(nkv, 1.0), *g = filled(nqv, 1.0);
  double *o1 = filled(nqv, 0), *o2 = filled(nqv, 0), *o3 = filled(nqv, 0);
  double *l1 = filled(nr, 0), *l2 = filled(nr, 0), *l3 = filled(nr, 0);
  CHECK(mea_oracle_fwd(B, H, nq, nk, d, dv, q, k, v, scale, causal, kv_len, o1, l1) == 0, "fwd");
  CHECK(mea_oracle_fwd_lazy(B, H, nq, nk, d, dv, q, k, v, scale, causal, kv_len, o2, l2) == 0, "lazy");
  CHECK(max_rel(o2, o1, nqv) < 1e-12 && max_rel(l2, l1, nr) < 1e-12, "lazy != direct (%g)",
        max_rel(o2, o1, nqv));
  const int64_t chunks[][2] = {{1, 1}, {3, 4}, {nq + 5, nk + 5}, {2, nk}};
  for (int c = 0; c < 4; ++c) {
    CHECK(mea_oracle_fwd_chunked(B, H, nq, nk, d, dv, q, k, v, scale, causal, kv_len, chunks[c][0],
                                 chunks[c][1], o3, l3) == 0, "chunked");
    CHECK(max_rel(o3, o1, nqv) < 1e-12 && max_rel(l3, l1, nr) < 1e-12, "chunked(%ld,%ld) != direct",
          (long)chunks[c][0], (long)chunks[c][1]);
  }
  double *dq = filled(nqd, 0), *dk = filled(nkd, 0), *dvv = filled(nkv, 0);
  CHECK(mea_oracle_bwd(B, H, nq, nk, d, dv, q, k, v, g, scale, causal, kv_len, dq, dk, dvv) == 0, "bwd");
  /* Subsets of one (batch, head) slice reproduce the full functions exactly. */
  const int64_t b = B - 1, h = H - 1, bh = b * H + h;
  const int64_t n_valid = kv_len ? (kv_len[b] < 0 ? 0 : (kv_len[b] > nk ? nk : kv_len[b])) : nk;
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nq > nk ? nq : nk));
  for (int64_t i = 0; i < (nq > nk ? nq : nk); ++i) rows[i] = i;
  const double *qs = q + bh * nq * d, *ks = k + bh * nk * d, *vs = v + bh * nk * dv, *gs = g + bh * nq * dv;
  double *orow = filled((size_t)(nq * dv), 0), *lrow = filled((size_t)nq, 0);
  double *dqr = filled((size_t)(nq * d), 0), *dkr = filled((size_t)(nk * d), 0), *dvr = filled((size_t)(nk * dv), 0);
  CHECK(mea_oracle_fwd_rows(nq, nk, d, dv, qs, ks, vs, scale, causal, n_valid, rows, nq, orow, lrow) == 0, "rows");
  CHECK(memcmp(orow, o1 + bh * nq * dv, sizeof(double) * (size_t)(nq * dv)) == 0, "fwd_rows o differs");
  CHECK(memcmp(lrow, l1 + bh * nq, sizeof(double) * (size_t)nq) == 0, "fwd_rows lse differs");
  CHECK(mea_oracle_bwd_dq_rows(nq, nk, d, dv, qs, ks, vs, gs, scale, causal, n_valid, rows, nq, dqr) == 0,
        "dq_rows");
  CHECK(memcmp(dqr, dq + bh * nq * d, sizeof(double) * (size_t)(nq * d)) == 0, "dq_rows differs");
  CHECK(mea_oracle_bwd_dkdv_keys(nq, nk, d, dv, qs, ks, vs, gs, scale, causal, n_valid, rows, nk, dkr,
                                 dvr) == 0, "dkdv_keys");
  CHECK(memcmp(dkr, dk + bh * nk * d, sizeof(double) * (size_t)(nk * d)) == 0, "dkdv_keys dk differs");
  CHECK(memcmp(dvr, dvv + bh * nk * dv, sizeof(double) * (size_t)(nk * dv)) == 0, "dkdv_keys dv differs");
  /* Invalid arguments are rejected, not read past. */
  int64_t bad_row = nq;
  CHECK(mea_oracle_fwd_rows(nq, nk, d, dv, qs, ks, vs, scale, causal, n_valid, &bad_row, 1, orow, lrow) != 0,
        "row out of range accepted");
  CHECK(mea_oracle_bwd_dkdv_keys(nq, nk, d, dv, qs, ks, vs, gs, scale, causal, nk + 1, rows, 1, dkr, dvr) != 0,
        "n_valid > n_k accepted");
  CHECK(mea_oracle_fwd_chunked(B, H, nq, nk, d, dv, q, k, v, scale, causal, kv_len, 0, 4, o3, l3) != 0,
        "zero chunk accepted");
  free(q); free(k); free(v); free(g); free(o1); free(o2); free(o3); free(l1); free(l2); free(l3);
  free(dq); free(dk); free(dvv); free(rows); free(orow); free(lrow); free(dqr); free(dkr); free(dvr);
}

int main(void) {
  const int64_t lens[2] = {9, 0};
  const int64_t lens3[3] = {1, 40, 17};
  one_case(1, 1, 1, 1, 4, 4, 0, NULL, 1.0);
  one_case(2, 3, 7, 13, 8, 8, 0, NULL, 1.0);
  one_case(2, 3, 7, 13, 8, 8, 1, NULL, 1.0);
  one_case(2, 2, 13, 7, 8, 5, 1, NULL, 1.0);
  one_case(2, 2, 11, 12, 6, 3, 0, lens, 1.0);
  one_case(3, 1, 20, 33, 5, 9, 1, lens3, 1.0);
  one_case(1, 2, 9, 30, 4, 4, 0, NULL, 60.0); /* large logits */
  if (failures == 0) printf("oracle_check ok\n");
  return failures;
}

/*
 * Drives every entry point of oracle/svm_oracle.c on small seeded problems, for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_sanitizers.py compiles both files
 * into one program).  Exits 0 and prints "ok" when every call returned as expected; the
 * sanitizers abort the program on any out-of-bounds access, leak or undefined operation.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t iterations;
  double b, b_up, b_low, dual_obj;
  int64_t n_sv, n_bound;
  int32_t status, pad;
} oracle_result;

double oracle_kernel_value(const float *a, const float *b, int64_t d, int kind, double gamma);
void oracle_kernel_rows(const float *X, int64_t n, int64_t d, const int64_t *rows, int64_t nrows, int kind,
                        double gamma, double *out, int threads);
int oracle_train(const float *X, const int32_t *y, int64_t n, int64_t d, int kind, double C, double gamma,
                 double tol, int64_t max_iter, int64_t cache_bytes, int threads, double *alpha, double *f_out,
                 oracle_result *res, int64_t trace_len, int32_t *trace_ul, double *trace_b, double *trace_gap,
                 int selection);
int oracle_train_ws(const float *X, const int32_t *y, int64_t n, int64_t d, int kind, double C, double gamma,
                    double tol, int64_t q, double frac, int64_t max_inner, int64_t max_iter, int64_t cache_bytes,
                    int threads, double *alpha, double *f_out, oracle_result *res, int64_t *rounds_out,
                    int64_t trace_len, int32_t *trace_ul, double *trace_b, double *trace_margin, int64_t *trace_t,
                    int64_t ws_trace_len, int32_t *ws_trace);
int64_t oracle_ws_select(const double *f, const int32_t *y, const double *alpha, int64_t n, double C, int64_t q,
                         int64_t *B);
void oracle_decision(const float *X, const int32_t *y, const double *alpha, double b, int64_t n, int64_t d, int kind,
                     double gamma, const float *T, int64_t m, double *dec, int threads);
void oracle_f_from_alpha(const float *X, const int32_t *y, const double *alpha, int64_t n, int64_t d, int kind,
                         double gamma, const int64_t *rows, int64_t nrows, double *out, int threads);

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static double urand(void) { /* xorshift64*, uniform in [0, 1) */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (double)((rng_state * 2685821657736338717ull) >> 11) * (1.0 / 9007199254740992.0);
}

#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                   \
    }                                                             \
  } while (0)

static int run(int64_t n, int64_t d, int64_t cache_bytes, int threads) {
  float *X = malloc(sizeof(float) * n * d);
  int32_t *y = malloc(sizeof(int32_t) * n);
  for (int64_t i = 0; i < n; ++i) {
    y[i] = (i % 3 == 0 || i == 0) ? 1 : -1;
    if (i == 1) y[i] = -1;
    for (int64_t k = 0; k < d; ++k) X[i * d + k] = (float)(urand() * 2.0 - 1.0 + 0.4 * y[i]);
  }
  double *alpha = malloc(sizeof(double) * n), *f = malloc(sizeof(double) * n);
  const int64_t tl = 64;
  int32_t *tul = malloc(sizeof(int32_t) * 2 * tl);
  double *tb = malloc(sizeof(double) * 2 * tl), *tg = malloc(sizeof(double) * 2 * tl);
  oracle_result r;
  for (int kind = 0; kind < 2; ++kind)
    for (int sel = 0; sel < 2; ++sel) {
      int st = oracle_train(X, y, n, d, kind, 1.0, 0.5, 1e-3, 100000, cache_bytes, threads, alpha, f, &r, tl, tul, tb,
                            tg, sel);
      CHECK(st == 0 && r.iterations > 0);
    }
  /* a step limit, and invalid input */
  CHECK(oracle_train(X, y, n, d, 0, 1.0, 0.5, 1e-6, 3, cache_bytes, threads, alpha, NULL, &r, 0, NULL, NULL,
                     NULL, 1) == 1);
  CHECK(oracle_train(X, y, n, d, 0, -1.0, 0.5, 1e-3, 10, cache_bytes, threads, alpha, NULL, &r, 0, NULL, NULL,
                     NULL, 0) == -1);
  CHECK(oracle_train(X, y, n, d, 0, 1.0, 0.5, 1e-3, 10, cache_bytes, threads, alpha, NULL, &r, 0, NULL, NULL,
                     NULL, 2) == -1);

  /* working-set rounds: q = 2, a middle size, and q larger than n */
  const int64_t qs[3] = {2, 8, 2 * n + 2};
  for (int qi = 0; qi < 3; ++qi) {
    const int64_t q = qs[qi];
    int64_t rounds = 0;
    double *tm = malloc(sizeof(double) * tl);
    int64_t *tt = malloc(sizeof(int64_t) * tl);
    int32_t *wst = malloc(sizeof(int32_t) * 4 * q);
    int st = oracle_train_ws(X, y, n, d, 0, 1.0, 0.5, 1e-3, q, 0.5, 100 * q, 100000, cache_bytes, threads, alpha, f,
                             &r, &rounds, tl, tul, tb, tm, tt, 4, wst);
    CHECK(st == 0 && rounds > 0);
    int64_t *B = malloc(sizeof(int64_t) * q);
    CHECK(oracle_ws_select(f, y, alpha, n, 1.0, q, B) >= 1);
    free(B);
    free(tm);
    free(tt);
    free(wst);
  }

  /* checkers */
  int64_t rows[5] = {0, n - 1, n / 2, n - 1, 0};
  double *K = malloc(sizeof(double) * 5 * n);
  oracle_kernel_rows(X, n, d, rows, 5, 0, 0.5, K, threads);
  CHECK(K[0] == 1.0 && K[n + n - 1] == 1.0);
  double *fr = malloc(sizeof(double) * 5);
  oracle_f_from_alpha(X, y, alpha, n, d, 0, 0.5, rows, 5, fr, threads);
  CHECK(fabs(fr[0] - fr[4]) == 0.0);
  const int64_t m = 17;
  double *dec = malloc(sizeof(double) * m);
  oracle_decision(X, y, alpha, r.b, n, d, 0, 0.5, X, m, dec, threads);
  CHECK(isfinite(dec[m - 1]));
  CHECK(oracle_kernel_value(X, X, d, 0, 0.5) == 1.0);

  free(K); free(fr); free(dec);
  free(X); free(y); free(alpha); free(f); free(tul); free(tb); free(tg);
  return 0;
}

int main(void) {
  /* full Gram (budget large), then the least-recently-used row cache (budget of a few rows) */
  if (run(61, 5, 1 << 26, 2)) return 1;
  if (run(61, 5, 8 * 61 * 3, 2)) return 1;
  if (run(130, 16, 8 * 130 * 2, 1)) return 1;
  printf("ok\n");
  return 0;
}

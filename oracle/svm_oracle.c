/*
 * svm_oracle.c -- plain, slow CPU reference ("oracle") for kernel-SVM training by SMO.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or load this
 * file or the library built from it; only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark do.  It shares no code, header, table or helper
 * with the HIP library.
 *
 * What it computes (paper, Section III.A and III.B):
 *   - the binary SVM problem on samples x_1..x_n in R^d with labels y_i in {+1,-1}
 *     (Section III.A), made non-linear by a kernel (Section III.A; the Gaussian RBF
 *     kernel is the one named in Section III.C);
 *   - its training QP solved by sequential minimal optimisation: each step picks two
 *     Lagrange multipliers and solves the two-variable sub-problem under the KKT
 *     conditions (Section III.B).  The pair is the maximal violating pair of the
 *     first-order rule the paper cites in Section III.B.
 *
 * Everything is fp64; X is read as fp32 and promoted.  The RBF kernel is evaluated in
 * the direct difference form exp(-gamma * sum_k (a_k - b_k)^2).  The selection scans
 * are serial, so results do not depend on the thread count; OpenMP is used only for
 * per-sample loops whose elements are independent (kernel rows, the f update).
 *
 * Readings where the paper is silent (stated once here, applied below):
 *   dual        max W(a) = sum a - 1/2 sum_ij a_i a_j y_i y_j K_ij, sum a_i y_i = 0, 0<=a<=C
 *   f_i         sum_j a_j y_j K_ij - y_i   (so a = 0 gives f = -y)
 *   I_up        {i : (y_i=+1 and a_i<C) or (y_i=-1 and a_i>0)}
 *   I_low       {i : (y_i=+1 and a_i>0) or (y_i=-1 and a_i<C)}
 *   selection   u = argmin_{I_up} f, l = argmax_{I_low} f; ties go to the smaller index
 *               (or, on request, the second-order rule for l: see oracle_train)
 *   stop        b_low - b_up <= tol
 *   eta         K_uu + K_ll - 2 K_ul, replaced by 1e-12 when <= 0
 *   clipping    box [L,H] on a_l, partner clamped to [0,C], values within 1e-12*C of a
 *               bound snapped onto it
 *   bias        b = (b_up + b_low) / 2 from the terminating selection
 *   decision    d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_RBF = 0, ORACLE_LINEAR = 1 };

typedef struct {
  int64_t iterations;
  double b, b_up, b_low, dual_obj;
  int64_t n_sv, n_bound;
  int32_t status; /* 0 converged, 1 max_iter reached, <0 invalid input */
  int32_t pad;
} oracle_result;

/* Kernel value between two samples (Section III.A; RBF form named in Section III.C). */
double oracle_kernel_value(const float *a, const float *b, int64_t d, int kind, double gamma) {
  double s = 0.0;
  if (kind == ORACLE_LINEAR) {
    for (int64_t k = 0; k < d; ++k) s += (double)a[k] * (double)b[k];
    return s;
  }
  for (int64_t k = 0; k < d; ++k) {
    double t = (double)a[k] - (double)b[k];
    s += t * t;
  }
  return exp(-gamma * s);
}

/* Kernel rows K(x_r, x_j) for j = 0..n-1 and each requested r. out is [nrows][n]. */
void oracle_kernel_rows(const float *X, int64_t n, int64_t d, const int64_t *rows, int64_t nrows, int kind,
                        double gamma, double *out, int threads) {
  for (int64_t q = 0; q < nrows; ++q) {
    const float *xr = X + rows[q] * d;
    double *o = out + q * n;
#pragma omp parallel for num_threads(threads) schedule(static)
    for (int64_t j = 0; j < n; ++j) o[j] = oracle_kernel_value(xr, X + j * d, d, kind, gamma);
  }
}

/* Kernel rows on demand: the full Gram when it fits the byte budget, else a small
 * least-recently-used set of rows.  Either way every value comes from
 * oracle_kernel_value, so the cache changes speed only. */
typedef struct {
  const float *X;
  int64_t n, d;
  int kind, threads;
  double gamma;
  double *gram;      /* n*n or NULL */
  double *slots;     /* cap*n */
  int64_t *slot_row; /* cap */
  int64_t *slot_tick;
  int64_t *row_slot; /* n */
  int64_t cap, tick;
} krows;

static int krows_init(krows *kr, const float *X, int64_t n, int64_t d, int kind, double gamma, int64_t budget,
                      int threads) {
  memset(kr, 0, sizeof(*kr));
  kr->X = X; kr->n = n; kr->d = d; kr->kind = kind; kr->gamma = gamma; kr->threads = threads;
  double need = 8.0 * (double)n * (double)n;
  if (need <= (double)budget) {
    kr->gram = (double *)malloc((size_t)(n * n) * sizeof(double));
    if (!kr->gram) return -1;
#pragma omp parallel for num_threads(threads) schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i)
      for (int64_t j = i; j < n; ++j) {
        double v = oracle_kernel_value(X + i * d, X + j * d, d, kind, gamma);
        kr->gram[i * n + j] = v;
        kr->gram[j * n + i] = v;
      }
    return 0;
  }
  int64_t cap = budget / (8 * n);
  if (cap < 2) cap = 2;
  if (cap > n) cap = n;
  kr->cap = cap;
  kr->slots = (double *)malloc((size_t)(cap * n) * sizeof(double));
  kr->slot_row = (int64_t *)malloc((size_t)cap * sizeof(int64_t));
  kr->slot_tick = (int64_t *)malloc((size_t)cap * sizeof(int64_t));
  kr->row_slot = (int64_t *)malloc((size_t)n * sizeof(int64_t));
  if (!kr->slots || !kr->slot_row || !kr->slot_tick || !kr->row_slot) return -1;
  for (int64_t s = 0; s < cap; ++s) { kr->slot_row[s] = -1; kr->slot_tick[s] = -1; }
  for (int64_t i = 0; i < n; ++i) kr->row_slot[i] = -1;
  return 0;
}

static void krows_free(krows *kr) {
  free(kr->gram); free(kr->slots); free(kr->slot_row); free(kr->slot_tick); free(kr->row_slot);
}

static const double *krows_get(krows *kr, int64_t i) {
  if (kr->gram) return kr->gram + i * kr->n;
  kr->tick++;
  int64_t s = kr->row_slot[i];
  if (s >= 0) { kr->slot_tick[s] = kr->tick; return kr->slots + s * kr->n; }
  int64_t victim = 0;
  for (int64_t q = 1; q < kr->cap; ++q)
    if (kr->slot_tick[q] < kr->slot_tick[victim]) victim = q;
  if (kr->slot_row[victim] >= 0) kr->row_slot[kr->slot_row[victim]] = -1;
  kr->slot_row[victim] = i; kr->slot_tick[victim] = kr->tick; kr->row_slot[i] = victim;
  double *o = kr->slots + victim * kr->n;
  const float *xi = kr->X + i * kr->d;
  const int64_t n = kr->n, d = kr->d;
#pragma omp parallel for num_threads(kr->threads) schedule(static)
  for (int64_t j = 0; j < n; ++j) o[j] = oracle_kernel_value(xi, kr->X + j * d, d, kr->kind, kr->gamma);
  return o;
}

static int in_up(int32_t y, double a, double C) { return (y > 0 && a < C) || (y < 0 && a > 0.0); }
static int in_low(int32_t y, double a, double C) { return (y > 0 && a > 0.0) || (y < 0 && a < C); }

static double clampd(double v, double lo, double hi) { return v < lo ? lo : (v > hi ? hi : v); }

/*
 * Binary SMO training (Section III.B).  Outputs alpha[n]; f[n] if non-NULL; the
 * result summary; and, for the first trace_len steps, the selected pair (u,l), the
 * selection values (b_up,b_low) and the runner-up gaps of both scans.
 *
 * The paper cites two working-pair rules (Section III.B).  selection = 0 takes the maximal
 * violating pair above.  selection = 1 takes the second-order rule for the second index:
 * u as above; l maximises the decrease of the objective that the unclipped two-variable step
 * on (u, t) would give, (f_t - f_u)^2 / a_ut with a_ut = K_uu + K_tt - 2 K_ut (1e-12 when
 * <= 0), over the members t of I_low with f_t > f_u, ties to the smaller index.  The stop
 * rule is the same for both (b_low the largest f over I_low), and so is the step on (u, l).
 * For selection = 1 the second runner-up gap is relative: (g_best - g_second) / g_best.
 */
int oracle_train(const float *X, const int32_t *y, int64_t n, int64_t d, int kind, double C, double gamma,
                 double tol, int64_t max_iter, int64_t cache_bytes, int threads, double *alpha, double *f_out,
                 oracle_result *res, int64_t trace_len, int32_t *trace_ul, double *trace_b, double *trace_gap,
                 int selection) {
  memset(res, 0, sizeof(*res));
  if (!X || !y || !alpha || n < 2 || d < 1 || !(C > 0) || !(tol > 0) || (kind == ORACLE_RBF && !(gamma > 0)) ||
      selection < 0 || selection > 1) {
    res->status = -1;
    return -1;
  }
  int64_t npos = 0, nneg = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (y[i] == 1) npos++;
    else if (y[i] == -1) nneg++;
    else { res->status = -1; return -1; }
  }
  if (!npos || !nneg) { res->status = -1; return -1; }

  krows kr;
  if (krows_init(&kr, X, n, d, kind, gamma, cache_bytes, threads)) { krows_free(&kr); res->status = -2; return -2; }
  double *f = (double *)malloc((size_t)n * sizeof(double));
  /* K_tt of every sample, for the second-order rule */
  double *diag = selection == 1 ? (double *)malloc((size_t)n * sizeof(double)) : NULL;
  if (!f || (selection == 1 && !diag)) { free(f); free(diag); krows_free(&kr); res->status = -2; return -2; }
  if (diag)
    for (int64_t i = 0; i < n; ++i) diag[i] = oracle_kernel_value(X + i * d, X + i * d, d, kind, gamma);

  /* Initial point: a = 0, so f_i = -y_i. */
  for (int64_t i = 0; i < n; ++i) { alpha[i] = 0.0; f[i] = -(double)y[i]; }

  int64_t t = 0;
  double b_up = 0.0, b_low = 0.0;
  int status = 1;
  for (;;) {
    /* Maximal violating pair: first-order selection over I_up and I_low. */
    int64_t u = -1, l = -1, u2 = -1, l2 = -1;
    for (int64_t i = 0; i < n; ++i) {
      if (in_up(y[i], alpha[i], C)) {
        if (u < 0 || f[i] < f[u]) { u2 = u; u = i; }
        else if (u2 < 0 || f[i] < f[u2]) u2 = i;
      }
      if (in_low(y[i], alpha[i], C)) {
        if (l < 0 || f[i] > f[l]) { l2 = l; l = i; }
        else if (l2 < 0 || f[i] > f[l2]) l2 = i;
      }
    }
    if (u < 0 || l < 0) { status = 0; break; }
    b_up = f[u];
    b_low = f[l];
    double gap_l = l2 >= 0 ? b_low - f[l2] : INFINITY;
    /* KKT conditions hold to within tol: stop. */
    const int stop = b_low - b_up <= tol;
    const double *Ku = NULL;
    if (!stop && t < max_iter && selection == 1) {
      /* second-order choice of l among the members of I_low above f_u */
      Ku = krows_get(&kr, u);
      double g1 = -1.0, g2 = -1.0;
      int64_t l1 = -1;
      for (int64_t i = 0; i < n; ++i) {
        if (!in_low(y[i], alpha[i], C) || !(f[i] > b_up)) continue;
        const double bt = f[i] - b_up;
        double at = Ku[u] + diag[i] - 2.0 * Ku[i];
        if (at <= 0.0) at = 1e-12;
        const double g = bt * bt / at;
        if (g > g1) { g2 = g1; g1 = g; l1 = i; }
        else if (g > g2) g2 = g;
      }
      l = l1;
      gap_l = g2 >= 0.0 ? (g1 - g2) / g1 : INFINITY;
    }
    if (t < trace_len) {
      if (trace_ul) { trace_ul[2 * t] = (int32_t)u; trace_ul[2 * t + 1] = (int32_t)l; }
      if (trace_b) { trace_b[2 * t] = b_up; trace_b[2 * t + 1] = b_low; }
      if (trace_gap) {
        trace_gap[2 * t] = u2 >= 0 ? f[u2] - b_up : INFINITY;
        trace_gap[2 * t + 1] = gap_l;
      }
    }
    if (stop) { status = 0; break; }
    if (t >= max_iter) { status = 1; break; }

    /* Two-variable sub-problem on (u, l). */
    if (!Ku) Ku = krows_get(&kr, u);
    const double *Kl = krows_get(&kr, l);
    double eta = Ku[u] + Kl[l] - 2.0 * Ku[l];
    if (eta <= 0.0) eta = 1e-12;
    const double yu = (double)y[u], yl = (double)y[l];
    const double s = yu * yl;
    const double au = alpha[u], al = alpha[l];
    double L, H;
    if (s < 0) { L = fmax(0.0, al - au); H = fmin(C, C + al - au); }
    else { L = fmax(0.0, au + al - C); H = fmin(C, au + al); }
    double al_new = clampd(al + yl * (b_up - f[l]) / eta, L, H);
    double au_new = clampd(au + s * (al - al_new), 0.0, C);
    const double snap = 1e-12 * C;
    if (fabs(al_new) <= snap) al_new = 0.0;
    if (fabs(al_new - C) <= snap) al_new = C;
    if (fabs(au_new) <= snap) au_new = 0.0;
    if (fabs(au_new - C) <= snap) au_new = C;

    /* Gradient update for every sample. */
    const double cu = (au_new - au) * yu, cl = (al_new - al) * yl;
#pragma omp parallel for num_threads(threads) schedule(static)
    for (int64_t j = 0; j < n; ++j) f[j] += cu * Ku[j] + cl * Kl[j];
    alpha[u] = au_new;
    alpha[l] = al_new;
    ++t;
  }

  res->iterations = t;
  res->status = status;
  res->b_up = b_up;
  res->b_low = b_low;
  res->b = 0.5 * (b_up + b_low);
  double sa = 0.0, saf = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    sa += alpha[i];
    saf += alpha[i] * (double)y[i] * f[i];
    if (alpha[i] > 0.0) { res->n_sv++; if (alpha[i] >= C) res->n_bound++; }
  }
  res->dual_obj = 0.5 * sa - 0.5 * saf;
  if (f_out) memcpy(f_out, f, (size_t)n * sizeof(double));
  free(f);
  free(diag);
  krows_free(&kr);
  return status;
}

/*
 * Working-set decomposition (the paper states only the two-multiplier step, Section III.B;
 * this is the reading used for the working-set variant of that step).  Each round:
 *   1. b_up, b_low and the stop rule exactly as in oracle_train;
 *   2. the working set B: the q/2 members of I_up with the smallest (f_i, i), in that order,
 *      then those of the q/2 members of I_low with the largest f_i (ties to the smaller i)
 *      that are not already in B -- between q/2 and q samples;
 *   3. the sub-problem on B, all other multipliers fixed, by the two-multiplier steps of
 *      oracle_train restricted to B (pair, clipping and snapping as there; ties in the
 *      selection to the smaller global index) on a copy of f_B, until its own gap is at most
 *      max(tol, frac * gap of the round) or max_inner steps were taken;
 *   4. f_j += s_j for every j, s_j = sum over p in B (in B's order, c_p != 0) of c_p K(B_p, j)
 *      with c_p = (a_new - a_old) y at B_p, accumulated from zero.
 * With q = 2 a round is one step of oracle_train (same pair, same update, same rounding).
 * iterations counts two-multiplier steps; max_iter bounds their total.  For the first
 * ws_trace_len rounds B is written to ws_trace (q entries per round, -1 padded).  For the first
 * trace_len rounds: the pair (u, l) and (b_up, b_low) of step 1, the steps taken before the
 * round (trace_t), and the round's margin (trace_margin): the smallest distance of any decision
 * taken in the round from the value that would flip it -- the stop test, the boundaries of the
 * two ranked lists at q/2, each pair selection against its runner-up, each local stop test, and
 * each new multiplier against the bounds of its box (relative to C).  A second solver whose
 * values differ from these by less than the margin takes the same decisions.
 */
typedef struct {
  const double *f;
  int64_t sign; /* +1: ascending f, -1: descending f; ties by ascending index either way */
} rank_ctx;

static rank_ctx g_rank;

static int rank_cmp(const void *pa, const void *pb) {
  const int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
  const double fa = (double)g_rank.sign * g_rank.f[a], fb = (double)g_rank.sign * g_rank.f[b];
  if (fa < fb) return -1;
  if (fa > fb) return 1;
  return a < b ? -1 : (a > b ? 1 : 0);
}

/* Step 2 of a round: B from f, y, alpha (scratch up[n], low[n]); returns |B|. */
static int64_t ws_select(const double *f, const int32_t *y, const double *alpha, int64_t n, double C, int64_t q,
                         int64_t *up, int64_t *low, int64_t *B) {
  int64_t nu = 0, nl = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (in_up(y[i], alpha[i], C)) up[nu++] = i;
    if (in_low(y[i], alpha[i], C)) low[nl++] = i;
  }
  g_rank.f = f;
  g_rank.sign = 1;
  qsort(up, (size_t)nu, sizeof(int64_t), rank_cmp);
  g_rank.sign = -1;
  qsort(low, (size_t)nl, sizeof(int64_t), rank_cmp);
  const int64_t h = q / 2;
  int64_t m = 0;
  for (int64_t k = 0; k < nu && k < h; ++k) B[m++] = up[k];
  const int64_t m_up = m;
  for (int64_t k = 0; k < nl && k < h; ++k) {
    int dup = 0;
    for (int64_t r = 0; r < m_up; ++r)
      if (B[r] == low[k]) { dup = 1; break; }
    if (!dup) B[m++] = low[k];
  }
  return m;
}

/* The working set of step 2 alone, for given f and alpha (B has room for q entries). */
int64_t oracle_ws_select(const double *f, const int32_t *y, const double *alpha, int64_t n, double C, int64_t q,
                         int64_t *B) {
  int64_t *up = (int64_t *)malloc((size_t)n * sizeof(int64_t));
  int64_t *low = (int64_t *)malloc((size_t)n * sizeof(int64_t));
  int64_t m = -1;
  if (up && low && q >= 2 && !(q & 1)) m = ws_select(f, y, alpha, n, C, q, up, low, B);
  free(up);
  free(low);
  return m;
}

int oracle_train_ws(const float *X, const int32_t *y, int64_t n, int64_t d, int kind, double C, double gamma,
                    double tol, int64_t q, double frac, int64_t max_inner, int64_t max_iter, int64_t cache_bytes,
                    int threads, double *alpha, double *f_out, oracle_result *res, int64_t *rounds_out,
                    int64_t trace_len, int32_t *trace_ul, double *trace_b, double *trace_margin, int64_t *trace_t,
                    int64_t ws_trace_len, int32_t *ws_trace) {
  memset(res, 0, sizeof(*res));
  if (!X || !y || !alpha || n < 2 || d < 1 || !(C > 0) || !(tol > 0) || (kind == ORACLE_RBF && !(gamma > 0)) ||
      q < 2 || (q & 1) || !(frac >= 0.0 && frac < 1.0) || max_inner < 1) {
    res->status = -1;
    return -1;
  }
  int64_t npos = 0, nneg = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (y[i] == 1) npos++;
    else if (y[i] == -1) nneg++;
    else { res->status = -1; return -1; }
  }
  if (!npos || !nneg) { res->status = -1; return -1; }

  krows kr;
  if (krows_init(&kr, X, n, d, kind, gamma, cache_bytes, threads)) { krows_free(&kr); res->status = -2; return -2; }
  double *f = (double *)malloc((size_t)n * sizeof(double));
  int64_t *up = (int64_t *)malloc((size_t)n * sizeof(int64_t));
  int64_t *low = (int64_t *)malloc((size_t)n * sizeof(int64_t));
  int64_t *B = (int64_t *)malloc((size_t)q * sizeof(int64_t));
  double *KB = (double *)malloc((size_t)(q * q) * sizeof(double));
  double *fB = (double *)malloc((size_t)q * sizeof(double));
  double *aB = (double *)malloc((size_t)q * sizeof(double));
  double *cB = (double *)malloc((size_t)q * sizeof(double));
  double *s = (double *)malloc((size_t)n * sizeof(double));
  if (!f || !up || !low || !B || !KB || !fB || !aB || !cB || !s) {
    free(f); free(up); free(low); free(B); free(KB); free(fB); free(aB); free(cB); free(s);
    krows_free(&kr);
    res->status = -2;
    return -2;
  }
  for (int64_t i = 0; i < n; ++i) { alpha[i] = 0.0; f[i] = -(double)y[i]; }

  int64_t t = 0, rounds = 0;
  double b_up = 0.0, b_low = 0.0;
  int status = 1;
  for (;;) {
    /* 1. maximal violating pair of the whole problem and the stop rule */
    int64_t u = -1, l = -1;
    for (int64_t i = 0; i < n; ++i) {
      if (in_up(y[i], alpha[i], C) && (u < 0 || f[i] < f[u])) u = i;
      if (in_low(y[i], alpha[i], C) && (l < 0 || f[i] > f[l])) l = i;
    }
    if (u < 0 || l < 0) { status = 0; break; }
    b_up = f[u];
    b_low = f[l];
    double margin = fabs((b_low - b_up) - tol);
    if (rounds < trace_len) {
      if (trace_ul) { trace_ul[2 * rounds] = (int32_t)u; trace_ul[2 * rounds + 1] = (int32_t)l; }
      if (trace_b) { trace_b[2 * rounds] = b_up; trace_b[2 * rounds + 1] = b_low; }
      if (trace_t) trace_t[rounds] = t;
      if (trace_margin) trace_margin[rounds] = margin;
    }
    if (b_low - b_up <= tol) { status = 0; break; }
    if (t >= max_iter) { status = 1; break; }

    /* 2. working set */
    const int64_t m = ws_select(f, y, alpha, n, C, q, up, low, B);
    if (rounds < ws_trace_len && ws_trace)
      for (int64_t k = 0; k < q; ++k) ws_trace[rounds * q + k] = k < m ? (int32_t)B[k] : -1;
    {
      /* the ranked lists' boundaries (up and low are sorted by ws_select) */
      int64_t nu = 0, nl = 0;
      for (int64_t i = 0; i < n; ++i) {
        nu += in_up(y[i], alpha[i], C);
        nl += in_low(y[i], alpha[i], C);
      }
      const int64_t h = q / 2;
      /* (from a = 0 every f is exactly -y, so the ties of round 0 are exact in any solver) */
      if (rounds > 0 && nu > h) margin = fmin(margin, f[up[h]] - f[up[h - 1]]);
      if (rounds > 0 && nl > h) margin = fmin(margin, f[low[h - 1]] - f[low[h]]);
    }

    /* 3. sub-problem on B */
    for (int64_t a = 0; a < m; ++a) {
      const double *Ka = krows_get(&kr, B[a]);
      for (int64_t b = 0; b < m; ++b) KB[a * m + b] = Ka[B[b]];
      fB[a] = f[B[a]];
      aB[a] = alpha[B[a]];
    }
    const double tol_loc = fmax(tol, frac * (b_low - b_up));
    for (int64_t inner = 0; inner < max_inner && t < max_iter; ++inner) {
      int64_t pu = -1, pl = -1;
      for (int64_t a = 0; a < m; ++a) {
        const int32_t ya = y[B[a]];
        if (in_up(ya, aB[a], C) && (pu < 0 || fB[a] < fB[pu] || (fB[a] == fB[pu] && B[a] < B[pu]))) pu = a;
        if (in_low(ya, aB[a], C) && (pl < 0 || fB[a] > fB[pl] || (fB[a] == fB[pl] && B[a] < B[pl]))) pl = a;
      }
      if (pu >= 0 && pl >= 0) {
        margin = fmin(margin, fabs((fB[pl] - fB[pu]) - tol_loc));
        /* the first step of round 0 sees f = -y exactly: its ties are exact in any solver */
        for (int64_t a = 0; a < m && !(rounds == 0 && inner == 0); ++a) {
          const int32_t ya = y[B[a]];
          if (a != pu && in_up(ya, aB[a], C)) margin = fmin(margin, fabs(fB[a] - fB[pu]));
          if (a != pl && in_low(ya, aB[a], C)) margin = fmin(margin, fabs(fB[pl] - fB[a]));
        }
      }
      if (pu < 0 || pl < 0 || fB[pl] - fB[pu] <= tol_loc) break;
      double eta = KB[pu * m + pu] + KB[pl * m + pl] - 2.0 * KB[pu * m + pl];
      if (eta <= 0.0) eta = 1e-12;
      const double yu = (double)y[B[pu]], yl = (double)y[B[pl]];
      const double sg = yu * yl;
      const double au = aB[pu], al = aB[pl];
      double L, H;
      if (sg < 0) { L = fmax(0.0, al - au); H = fmin(C, C + al - au); }
      else { L = fmax(0.0, au + al - C); H = fmin(C, au + al); }
      const double al_raw = al + yl * (fB[pu] - fB[pl]) / eta;
      margin = fmin(margin, fmin(fabs(al_raw - L), fabs(al_raw - H)) / C);
      double al_new = clampd(al_raw, L, H);
      double au_new = clampd(au + sg * (al - al_new), 0.0, C);
      const double snap = 1e-12 * C;
      if (fabs(al_new) <= snap) al_new = 0.0;
      if (fabs(al_new - C) <= snap) al_new = C;
      if (fabs(au_new) <= snap) au_new = 0.0;
      if (fabs(au_new - C) <= snap) au_new = C;
      const double cu = (au_new - au) * yu, cl = (al_new - al) * yl;
      for (int64_t a = 0; a < m; ++a) fB[a] += cu * KB[pu * m + a] + cl * KB[pl * m + a];
      aB[pu] = au_new;
      aB[pl] = al_new;
      ++t;
    }

    /* 4. gradient update of every sample from the change of the multipliers in B */
    for (int64_t a = 0; a < m; ++a) cB[a] = (aB[a] - alpha[B[a]]) * (double)y[B[a]];
    for (int64_t j = 0; j < n; ++j) s[j] = 0.0;
    for (int64_t a = 0; a < m; ++a) {
      if (cB[a] == 0.0) continue;
      const double *Ka = krows_get(&kr, B[a]);
      const double c = cB[a];
#pragma omp parallel for num_threads(threads) schedule(static)
      for (int64_t j = 0; j < n; ++j) s[j] += c * Ka[j];
    }
    for (int64_t j = 0; j < n; ++j) f[j] += s[j];
    for (int64_t a = 0; a < m; ++a) alpha[B[a]] = aB[a];
    if (rounds < trace_len && trace_margin) trace_margin[rounds] = margin;
    ++rounds;
  }

  res->iterations = t;
  res->status = status;
  res->b_up = b_up;
  res->b_low = b_low;
  res->b = 0.5 * (b_up + b_low);
  double sa = 0.0, saf = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    sa += alpha[i];
    saf += alpha[i] * (double)y[i] * f[i];
    if (alpha[i] > 0.0) { res->n_sv++; if (alpha[i] >= C) res->n_bound++; }
  }
  res->dual_obj = 0.5 * sa - 0.5 * saf;
  if (rounds_out) *rounds_out = rounds;
  if (f_out) memcpy(f_out, f, (size_t)n * sizeof(double));
  free(f); free(up); free(low); free(B); free(KB); free(fB); free(aB); free(cB); free(s);
  krows_free(&kr);
  return status;
}

/* Decision values d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b, summed in index order. */
void oracle_decision(const float *X, const int32_t *y, const double *alpha, double b, int64_t n, int64_t d, int kind,
                     double gamma, const float *T, int64_t m, double *dec, int threads) {
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t q = 0; q < m; ++q) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i)
      if (alpha[i] > 0.0) s += alpha[i] * (double)y[i] * oracle_kernel_value(X + i * d, T + q * d, d, kind, gamma);
    dec[q] = s - b;
  }
}

/* f_i = sum_j a_j y_j K_ij - y_i recomputed from alpha, for the listed rows only. */
void oracle_f_from_alpha(const float *X, const int32_t *y, const double *alpha, int64_t n, int64_t d, int kind,
                         double gamma, const int64_t *rows, int64_t nrows, double *out, int threads) {
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t q = 0; q < nrows; ++q) {
    const int64_t i = rows[q];
    double s = 0.0;
    for (int64_t j = 0; j < n; ++j)
      if (alpha[j] != 0.0) s += alpha[j] * (double)y[j] * oracle_kernel_value(X + i * d, X + j * d, d, kind, gamma);
    out[q] = s - (double)y[i];
  }
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/*
 * svmx.h -- C ABI of libsvmx.so: kernel-SVM training by SMO on one AMD Instinct MI355X (gfx950).
 *
 * The problem (paper, Section III.A): samples X = {x_1..x_n}, x_i in R^d, labels y_i in {+1,-1};
 * find the maximum-margin separator, made non-linear by a kernel.  The kernel here is the
 * Gaussian RBF K(a,b) = exp(-gamma * |a-b|^2) (the kernel the paper names, Section III.C).
 * Training solves the dual QP by sequential minimal optimisation: each step updates two
 * Lagrange multipliers under the KKT conditions (Section III.B).  Multiclass training is
 * one-against-one: m classes give m(m-1)/2 independent binary problems (Section III.A).
 *
 * The dual solved:  max W(a) = sum_i a_i - 1/2 sum_ij a_i a_j y_i y_j K_ij
 *                   s.t. sum_i a_i y_i = 0,  0 <= a_i <= C.
 * With f_i = sum_j a_j y_j K_ij - y_i the working pair of each step is the maximal violating
 * pair u = argmin_{I_up} f, l = argmax_{I_low} f (ties to the smaller index), where
 *   I_up  = {i : (y_i=+1 and a_i<C) or (y_i=-1 and a_i>0)},
 *   I_low = {i : (y_i=+1 and a_i>0) or (y_i=-1 and a_i<C)};
 * training stops when b_low - b_up <= tol (b_up = f_u, b_low = f_l) and returns
 * b = (b_up + b_low)/2.  Decision values are d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b; the
 * predicted label is +1 iff d(x) > 0.
 *
 * Conventions for every entry point:
 *  - "device" pointers are HIP device memory of the current device; "host" pointers are
 *    ordinary host memory.  X arrays are fp32, row-major [rows][d], rows contiguous.
 *  - The caller owns every buffer, including the device workspace, whose size is given by
 *    the matching *_workspace_bytes query.  The library keeps no state between calls
 *    except the loaded code object, a thread-local error message, and (svm_train_static only)
 *    its static device scratch and that scratch's address on each device.
 *  - All device work is enqueued on options->stream (a hipStream_t; NULL = the null stream).
 *    Every call returns only after its outputs are complete.
 *  - Negative status: nothing was written to the outputs that can be relied upon, nothing
 *    leaks; svm_last_error() explains.  SVM_NOT_CONVERGED (positive) means the iteration
 *    limit was reached: alpha is feasible (0 <= a <= C, sum a y = 0) and b is the current
 *    midpoint.
 *  - Calls on one device that overlap in time must use distinct workspaces.  Training calls
 *    (svm_train, svm_train_ovo) should not overlap in time on one device: each solver launch
 *    expects all of its workgroups to run at once, and one that has to wait longer than the
 *    device-side wait limit (2 s) for workgroups held back by another call's launch ends with
 *    SVM_EDEVICE.
 */
#ifndef SVMX_H
#define SVMX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SVM_OK = 0,
  SVM_NOT_CONVERGED = 1,
  SVM_EINVAL = -1,     /* invalid argument */
  SVM_ENOMEM = -2,     /* problem too large for the device, or n beyond the 32-bit sample index
                          (n > 2^31 - 2) */
  SVM_EDEVICE = -3,    /* a HIP call failed, or a device-side wait exceeded its time limit */
  SVM_EWORKSPACE = -4  /* workspace NULL or smaller than the size query returned */
} svm_status;

/* Where kernel rows come from during the solve. */
typedef enum {
  SVM_GRAM_AUTO = 0, /* full Gram when it fits gram_budget_bytes, else row path */
  SVM_GRAM_ON = 1,   /* precompute the full fp32 Gram (MFMA) and read rows from it */
  SVM_GRAM_OFF = 2   /* row path: evaluate the two kernel rows from X at every step */
} svm_gram_mode;

/* Which MFMA instruction computes the Gram's dot products (the Gram path and svm_gram). */
typedef enum {
  SVM_MFMA_SPLIT_F16 = 0, /* every row scaled by a power of two and split into two fp16 halves;
                             three fp16 MFMA products per fp32 product (v_mfma_f32_16x16x32_f16),
                             fp32 accumulation; values as accurate as SVM_MFMA_F32 */
  SVM_MFMA_F32 = 1        /* fp32 inputs on v_mfma_f32_16x16x4f32 */
} svm_gram_mfma;

/* How the working pair of each step is chosen (the paper cites two rules, Section III.B). */
typedef enum {
  SVM_SELECT_MVP = 0,         /* maximal violating pair: u = argmin_{I_up} f, l = argmax_{I_low} f */
  SVM_SELECT_SECOND_ORDER = 1 /* u as above; l = the member t of I_low with f_t > f_u that maximises
                                 (f_t - f_u)^2 / a_ut, a_ut = K_uu + K_tt - 2 K_ut (1e-12 when not
                                 positive), ties to the smaller index: the decrease of the objective
                                 the unclipped step on (u, t) would give.  The stop rule is unchanged
                                 (b_low = max_{I_low} f).  Gram path only (each step reads row u
                                 before l is known); not with working_set */
} svm_selection;

#define SVM_WORKING_SET_AUTO (-1) /* svm_options.working_set: decided per problem (see there) */

typedef struct {
  int32_t struct_size;       /* = sizeof(svm_options); set by svm_default_options */
  int32_t gram;              /* svm_gram_mode */
  int64_t gram_budget_bytes; /* AUTO picks the Gram when 4*n*ld <= budget (ld = n rounded up to 64);
                                0 = 200 GiB */
  int64_t row_cache_bytes;   /* row path: HBM bytes for cached kernel rows; 0 = none */
  int64_t max_iter;          /* 0 = max(10^7, 100 n) SMO steps */
  int32_t check_every;       /* SMO steps per device launch between host convergence checks
                                (the host-side check "every set of iterations", Section III.B);
                                0 = 65536.  Results do not depend on it. */
  int32_t trace_len;         /* record the selection of the first trace_len steps */
  int32_t *trace_ws;         /* host [2*trace_len]: (u, l) of each step, or NULL */
  double *trace_b;           /* host [2*trace_len]: (b_up, b_low) of each step, or NULL */
  double *f_out;             /* device [n]: final f, or NULL (binary training only) */
  void *stream;              /* hipStream_t, or NULL */
  int32_t workgroups;        /* solver workgroups per problem; 0 = automatic */
  int32_t exchange_levels;   /* levels of the cross-workgroup exchange: 1, 2, or 0 = automatic
                                (two levels above 128 workgroups per problem) */
  int32_t gram_mfma;         /* svm_gram_mfma */
  int32_t working_set;       /* 0 = one maximal violating pair per step with f updated every step
                                (Section III.B).  SVM_WORKING_SET_AUTO (-1): binary training with
                                the first-order rule, no trace and automatic workgroups, n > 4096:
                                rounds of q = 64 with a Gram and 128 without (rows of 256 features
                                or more), else 32, for the first 128 rounds, continued if they took
                                at least as many pair steps per round as a round costs (Gram path:
                                10 at q = 64, 4.25 at 32; row path: 12.5 at q = 128, 4.5 at 32,
                                measured on MI355X), else the per-step solver
                                takes over from their state (svm_stats.schedule says which); every
                                other case per-step.  Deterministic: the rule reads the state after
                                a fixed number of rounds, not the host check cadence.
                                q = 2..128, even: working-set rounds -- B = the
                                q/2 smallest f of I_up and the q/2 largest of I_low (ties to the
                                smaller index), pair steps on B alone until its gap is at most
                                max(tol, 0.5 x the round's gap) or 100 q steps, then f updated once
                                from the round's change.  Gram path: n <= 261,120 (255
                                workgroups of up to 1,024 samples).  Row path: every round
                                evaluates K(B, .) from X in one pass, n <= 255 x min(1024,
                                16384 / q).  Binary training only.  The trace then holds the
                                maximal violating pair of every round. */
  int32_t resident_rows;     /* binary training, row path, per-step solver: rows of X each solver
                                workgroup keeps in LDS for the whole launch (the first rows of its
                                slice), read from there instead of from HBM at every step; 0 = as
                                many as fit, -1 = none, k > 0 = at most k.  Results do not depend
                                on it. */
  int32_t selection;         /* svm_selection (binary and one-vs-one training) */
  int32_t reserved;          /* must be 0 */
  const double *alpha_init;  /* binary training: device [n] multipliers to start from instead of 0
                                (a warm start, e.g. to resume a call stopped by max_iter), or NULL.
                                Must be finite with 0 <= a_i <= C and |sum a_i y_i| <= 1e-9 C n
                                (the equality constraint), else SVM_EINVAL.  The buffer may be the
                                alpha argument itself; it is read before the call writes alpha.
                                svm_train_ovo rejects it (SVM_EINVAL). */
  const double *f_init;      /* with alpha_init: device [n] values f_i = sum_j a_j y_j K_ij - y_i
                                that go with it (a previous call's f_out), or NULL: recomputed on
                                the device from alpha_init -- from the Gram on the Gram path, from X
                                with the exact fp64 kernel otherwise.  With the f_out of a call
                                stopped by max_iter, the resumed call takes the steps the
                                uninterrupted one would have taken.  Must be finite. */
} svm_options;

typedef struct {
  int64_t iterations;   /* SMO steps taken */
  int64_t n_sv;         /* samples with a_i > 0 */
  int64_t n_bound_sv;   /* samples with a_i = C */
  double b_up, b_low;   /* selection values of the final step */
  double dual_obj;      /* W(a) = 1/2 sum a - 1/2 sum a y f */
  int32_t gram_used;    /* 1 if the full Gram was precomputed */
  int32_t launches;     /* solver launches (host convergence checks) */
  double t_gram;        /* seconds of the precompute: the Gram build, or the squared row norms
                           of the row path */
  double t_solve, t_finalize, t_total; /* seconds */
  double t_kernel;      /* seconds the solver kernel ran, summed over its launches (HIP events on
                           the launch stream) */
  int64_t rounds;       /* working-set rounds (0 for the per-step solver) */
  int32_t resident_rows; /* rows of X each solver workgroup kept in LDS (binary row path) */
  int32_t schedule;     /* binary training: 0 = per-step solver, 1 = working-set rounds, 2 = rounds
                           (the automatic probe), then the per-step solver */
  double t_upload;      /* seconds of input validation and staging before the precompute: the
                           labels copied to the host and checked (one-vs-one: and class-sorted),
                           the problem descriptors copied to the device, the device-side scan of X
                           for values that are not finite (one-vs-one: and the class-sorted copy of
                           X).  The inputs themselves are device buffers, so no copy of X over
                           PCIe is part of any call. */
} svm_stats;

/* Fill *o with the defaults above. */
void svm_default_options(svm_options *o);

/* Device workspace bytes svm_train needs for an n x d problem under options o (NULL =
 * defaults); -1 if the sizes overflow or are invalid. */
int64_t svm_train_workspace_bytes(int64_t n, int64_t d, const svm_options *o);

/*
 * Binary training (Sections III.A and III.B).
 *   X      device fp32 [n][d]          training samples
 *   y      device int32 [n]            labels, each +1 or -1, both present
 *   C      > 0, finite                  box constraint
 *   gamma  > 0, finite                  RBF width
 *   tol    > 0, finite                  stopping tolerance on b_low - b_up
 *   alpha  device fp64 [n], out        Lagrange multipliers
 *   b      host double, out            bias of d(x) = sum a y K - b
 *   workspace/workspace_bytes          device scratch of at least svm_train_workspace_bytes
 *   o      options or NULL;  st  host stats out or NULL
 * EINVAL: n<2, d<1, non-finite or non-positive C/gamma/tol, NULL pointers, a label not in
 * {+1,-1} or only one class present, a value of X that is not finite (checked on the device
 * before any other work), byte counts of n*d or of the n^2 Gram that overflow int64.
 */
svm_status svm_train(const float *X, const int32_t *y, int64_t n, int64_t d, double C, double gamma, double tol,
                     double *alpha, double *b, void *workspace, int64_t workspace_bytes, const svm_options *o,
                     svm_stats *st);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): svm_train without a workspace argument.  Its device
 * scratch is a library-owned static array of SVM_STATIC_SCRATCH_BYTES on each device the library
 * runs on (held until the process ends); it calls no hipMalloc/hipFree and creates no HIP events
 * (t_gram, t_solve, t_finalize and t_kernel of *st are reported as 0).  Arguments, outputs and
 * results are those of svm_train with the same options, except that SVM_GRAM_AUTO takes the Gram
 * only when the whole plan fits the scratch (else the row path).  SVM_EWORKSPACE when the plan
 * does not fit: on the Gram path beyond n = 4,060 at 16 features (3,712 at 784); the row path
 * needs about 16 bytes a sample, within the scratch up to its own limit of 1,048,576 samples.
 * Every call on one device uses that device's one array and leaves the last call's
 * contents in it (each call initialises what it reads): calls that overlap in time on one device
 * race, and must not be made.
 */
#define SVM_STATIC_SCRATCH_BYTES (64LL * 1024 * 1024)
svm_status svm_train_static(const float *X, const int32_t *y, int64_t n, int64_t d, double C, double gamma,
                            double tol, double *alpha, double *b, const svm_options *o, svm_stats *st);

/* Device workspace bytes svm_predict needs. */
int64_t svm_predict_workspace_bytes(int64_t n, int64_t d, int64_t m);

/*
 * Decision values d(x_q) = sum_{a_i>0} a_i y_i K(x_i, x_q) - b for m test samples.
 *   X_train device fp32 [n][d], y device int32 [n], alpha device fp64 [n], b host value,
 *   X_test device fp32 [m][d], dec device fp64 [m] out.  m = 0 is allowed (nothing written).
 */
svm_status svm_predict(const float *X_train, const int32_t *y, const double *alpha, double b, int64_t n, int64_t d,
                       double gamma, const float *X_test, int64_t m, double *dec, void *workspace,
                       int64_t workspace_bytes, const svm_options *o);

/* Device workspace bytes svm_train_ovo needs for n samples in k classes. */
int64_t svm_train_ovo_workspace_bytes(int64_t n, int64_t d, int32_t k, const svm_options *o);

/*
 * One-against-one training (Section III.A; the binary problems run side by side on the one
 * device, Section III.B).  P = k(k-1)/2 pairs (a<b) in lexicographic order; in pair (a,b)
 * class a is +1 and class b is -1, and the pair's local sample order is the class-a samples
 * by increasing original index followed by the class-b samples likewise.
 *   label  device int32 [n], values 0..k-1, every class present
 *   alpha  device fp64 [(k-1)*n] out: the pairs' multipliers packed in pair order, each pair
 *          in its local sample order (pair p occupies n_a + n_b entries)
 *   b      host double [P] out;  st  host svm_stats [P] out or NULL
 * EINVAL as for svm_train (a label outside 0..k-1, a class without samples and a value of X
 * that is not finite included).
 */
svm_status svm_train_ovo(const float *X, const int32_t *label, int64_t n, int64_t d, int32_t k, double C,
                         double gamma, double tol, double *alpha, double *b, void *workspace,
                         int64_t workspace_bytes, const svm_options *o, svm_stats *st);

/* Device workspace bytes svm_predict_ovo needs. */
int64_t svm_predict_ovo_workspace_bytes(int64_t n, int64_t d, int32_t k, int64_t m);

/*
 * One-against-one prediction with the outputs of svm_train_ovo.
 *   dec   device fp64 [m][P] out: decision value of every pair
 *   pred  device int32 [m] out: class with most votes (pair (a,b) votes a iff d>0, else b);
 *         ties go to the smaller class id
 */
svm_status svm_predict_ovo(const float *X, const int32_t *label, int64_t n, int64_t d, int32_t k,
                           const double *alpha, const double *b, double gamma, const float *X_test, int64_t m,
                           double *dec, int32_t *pred, void *workspace, int64_t workspace_bytes,
                           const svm_options *o);

/*
 * The kernel rows of the hot path, exposed for verification:
 * out[q][j] = K(x_{rows[q]}, x_j) for j < n, evaluated the way the row path evaluates them.
 *   rows device int64 [r] (each in [0,n)), out device fp32 [r][n].
 */
svm_status svm_kernel_rows(const float *X, int64_t n, int64_t d, double gamma, const int64_t *rows, int64_t r,
                           float *out, const svm_options *o);

/*
 * The full fp32 RBF Gram the Gram path precomputes (MFMA X X^T with a row-norm epilogue, on the
 * instruction o->gram_mfma selects): G[i*ld + j] = K(x_i, x_j) for i, j < n; ld >= n.  G device
 * fp32 [n][ld].  workspace: device scratch of svm_gram_workspace_bytes(n, d, o) bytes (the split
 * fp16 rows, scales and norms; 0 bytes for SVM_MFMA_F32, where workspace may be NULL).
 */
int64_t svm_gram_workspace_bytes(int64_t n, int64_t d, const svm_options *o);
svm_status svm_gram(const float *X, int64_t n, int64_t d, double gamma, float *G, int64_t ld, void *workspace,
                    int64_t workspace_bytes, const svm_options *o);

/* Thread-local message for the last non-OK status of this thread ("" if none). */
const char *svm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SVMX_H */

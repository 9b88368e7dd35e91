// common.hpp -- internal definitions shared by the host solver and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

typedef unsigned long long u64;

// Problem status kept in Ctl::status.
enum : int32_t { ST_RUNNING = 0, ST_CONVERGED = 1, ST_MAXITER = 2, ST_TIMEOUT = -1 };

// Per-problem control block (device memory).  Written only by workgroup 0 of the problem.
struct Ctl {
  int64_t t;         // SMO steps taken so far
  int32_t status;    // ST_*
  int32_t pad;
  double b_up, b_low;
  int64_t u, l;      // last selection
};

// One binary sub-problem of a solver launch.  A binary training run is one problem; a
// one-vs-one run is one problem per class pair.  Local sample j maps to the global sample
// (row of the Gram / of X) off0 + j for j < len0, else off1 + (j - len0).
struct Prob {
  int64_t n;          // local samples
  int64_t off0, len0, off1;
  const int32_t *y;   // binary: labels by global index; NULL: +1 for j < len0, else -1
  double *alpha;      // [n] local order
  double *f;          // [n]
  Ctl *ctl;
  u64 *slots;         // exchange words [2][nwg][SLOT_WORDS]
  u64 *slots2;        // second exchange level [2][ng][SLOT_WORDS], or NULL
  int32_t *trace_ul;  // [2*trace_len] or NULL
  double *trace_b;    // [2*trace_len] or NULL
  int64_t trace_len;
  int32_t wg0, nwg;   // workgroups [wg0, wg0+nwg) of the launch serve this problem
  int32_t per_wg;     // local samples per workgroup
  int32_t g1;         // workgroups per first-level exchange group (0 = one level)
  int32_t ng;         // number of first-level groups
  int32_t pad;
};

constexpr int SLOT_WORDS = 16;  // 10 used; a record fills one 128-byte line

// Launch-wide parameters of the persistent solver.
struct SolveParams {
  const Prob *probs;
  const int32_t *wg_prob;  // workgroup -> problem
  double C, tol, gamma;
  int64_t max_iter;        // absolute step limit per problem
  int64_t steps;           // steps this launch may take per problem
  // Gram path
  const float *gram;       // [N][ld] or NULL
  int64_t ld;
  // Row path
  const float *X;          // [N][d] (global order)
  const double *sqn;       // [N] squared row norms of X (row_norms_k)
  int64_t d;
  float *cache;            // [cap][ld] row slices, or NULL
  int32_t *cache_tags;     // [nwg_total][cap] per-workgroup tag copies
  int32_t cache_cap;
  int32_t pad;
  uint64_t spin_limit;     // wall-clock ticks (100 MHz) a wait may last
  int32_t *error;          // set to 1 on a wait time-out
};

// Kernel launchers (defined in the .hip files).
hipError_t launch_gram(const float *X, int64_t n, int64_t d, float gamma, float *G, int64_t ld, hipStream_t s);
hipError_t launch_kernel_rows(const float *X, int64_t n, int64_t d, double gamma, const int64_t *rows, int64_t r,
                              float *out, hipStream_t s);
// Rows of X scaled by powers of two and split into two fp16 halves (gram_split.hip): hi and lo
// [n][dp] (dp = d rounded up to 32, zero padded), the row scales and the row norms.
struct SplitX {
  _Float16 *hi, *lo;
  float *scale, *nrm;
  int64_t dp;
};
SplitX split_views(void *scratch, int64_t n, int64_t d);
hipError_t launch_split_rows(const float *X, int64_t n, int64_t d, const SplitX &s, hipStream_t st);

// Split-fp16 Gram (gram_split.hip): scratch bytes, and the build into G.
int64_t gram_split_scratch_bytes(int64_t n, int64_t d);
hipError_t launch_gram_split(const float *X, int64_t n, int64_t d, float gamma, float *G, int64_t ld, void *scratch,
                             hipStream_t st);
hipError_t launch_row_norms(const float *X, int64_t n, int64_t d, double *sqn, hipStream_t s);
hipError_t launch_gather_rows(const float *X, int64_t d, const int32_t *perm, int64_t n, float *Xs, hipStream_t s);
hipError_t launch_solver_init(const Prob *probs, int32_t nprob, int64_t max_n, hipStream_t s);
// total_wg <= 0 only reports in *max_coresident how many workgroups of the variant fit at once.
hipError_t launch_solver(const SolveParams &p, int32_t total_wg, int32_t per_thread, bool gram, hipStream_t s,
                         int32_t *max_coresident);
hipError_t launch_finalize(const Prob *probs, int32_t nprob, double C, double *out /*[nprob][4]*/, hipStream_t s);
// Device scratch of one prediction: compacted support vectors and per-split partial sums.
struct PredictScratch {
  int32_t *sv_row;  // [ntr]
  double *sv_coef;  // [ntr]
  int64_t *count;   // [1]
  double *part;     // [predict_splits(m, ntr)][m]
  const SplitX *split_train = nullptr;  // split rows of the training X and of the test samples
  const SplitX *split_test = nullptr;   // (both set: the split-fp16 kernel; host pointers)
};
int predict_splits(int64_t m, int64_t nsv_max);
// Decision values for training samples addressed like Prob (local j -> row off0+j or
// off1+j-len0, then through perm when perm != NULL); labels from y by that row, or by range.
hipError_t launch_predict_map(const float *Xtr, int64_t d, int64_t off0, int64_t len0, int64_t off1,
                              const int32_t *y, const int32_t *perm, const double *alpha, int64_t ntr, double gamma,
                              const float *T, int64_t m, double b, double *dec, int64_t dec_stride,
                              const PredictScratch &ws, hipStream_t s);
hipError_t launch_ovo_vote(const double *dec, int64_t m, int32_t k, int32_t *pred, hipStream_t s);

int solver_block_size(bool gram);
int max_per_thread(bool gram);

}  // namespace svmx

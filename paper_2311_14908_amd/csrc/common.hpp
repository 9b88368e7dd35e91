// common.hpp -- internal definitions shared by the host solver and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "solver_params.hpp"

namespace svmx {

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

// Kernel value from the fp32 accumulation of the split-fp16 product of rows i and j (row i the
// MFMA's first operand): the scales, |x_i|^2 + |x_j|^2 - 2 x_i.x_j with one fused multiply-add,
// clamped at 0, exp2(c t), c = -gamma log2(e) (one fused multiply-add, written out, so the
// rounding does not depend on what the compiler contracts).
__device__ __forceinline__ float split_rbf(float acc, float si, float sj, float ni, float nj, float c) {
  const float dot = (acc * si) * sj;
  float t = __builtin_fmaf(-2.0f, dot, ni + nj);
  t = t > 0.f ? t : 0.f;
  return __builtin_amdgcn_exp2f(c * t);
}
hipError_t launch_split_rows(const float *X, int64_t n, int64_t d, const SplitX &s, hipStream_t st);

// Split-fp16 Gram (gram_split.hip): scratch bytes, and the build into G.
int64_t gram_split_scratch_bytes(int64_t n, int64_t d);
hipError_t launch_gram_split(const float *X, int64_t n, int64_t d, float gamma, float *G, int64_t ld, void *scratch,
                             hipStream_t st);
hipError_t launch_row_norms(const float *X, int64_t n, int64_t d, double *sqn, hipStream_t s);
// flag[0] = 1 when a value of X[0 .. count) is not finite (flag left as it is otherwise).
hipError_t launch_check_finite(const float *X, int64_t count, int32_t *flag, hipStream_t s);
hipError_t launch_gather_rows(const float *X, int64_t d, const int32_t *perm, int64_t n, float *Xs, hipStream_t s);
hipError_t launch_solver_init(const Prob *probs, int32_t nprob, int64_t max_n, hipStream_t s);
// total_wg <= 0 only reports in *max_coresident how many workgroups of the variant fit at once.
hipError_t launch_solver(const SolveParams &p, int32_t total_wg, int32_t per_thread, bool gram, hipStream_t s,
                         int32_t *max_coresident);
// Row path: how many rows of X a solver workgroup can keep resident in LDS next to its other
// LDS data (p's max_per_wg, cache_cap and d; per_thread as for launch_solver), or -1 on a HIP
// error.
int64_t solver_res_rows_max(const SolveParams &p, int32_t per_thread);
hipError_t launch_finalize(const Prob *probs, int32_t nprob, double C, double *out /*[nprob][4]*/, hipStream_t s);
// Device scratch of a prediction: compacted support vectors and per-split partial sums of
// every problem of one launch, and the problems' descriptions.
struct PredictScratch {
  int32_t *sv_row;  // [sum of the problems' ntr]
  double *sv_coef;  // [sum of the problems' ntr]
  int64_t *count;   // [problems]
  double *part;     // [sum of the problems' nsplit][m]
  struct PredPair *pairs;  // [problems], device
  const SplitX *split_train = nullptr;  // split rows of the training X and of the test samples
  const SplitX *split_test = nullptr;   // (both set: the split-fp16 kernel; host pointers)
};
int predict_splits(int64_t m, int64_t nsv_max);
// One problem of a prediction launch: its training samples addressed like Prob (local j -> row
// off0+j or off1+j-len0, then through perm when perm != NULL; labels from y by that row, or by
// range), its multipliers alpha[alpha_off ..][ntr], where its support vectors and partial sums
// go, its bias and split count (predict_splits(m, ntr)).
struct PredPair {
  int64_t off0, len0, off1;
  const int32_t *y;
  const int32_t *perm;
  int64_t alpha_off, ntr, sv_off, part_off;
  double b;
  int32_t nsplit, pad;
};
// Decision values of npairs problems in one launch per stage: dec[q * dec_stride + p] for test
// sample q and problem p (pairs[] already on the device, in ws.pairs); nsplit_max = the
// largest nsplit among them.
hipError_t launch_predict_pairs(const float *Xtr, int64_t d, int32_t npairs, int nsplit_max, const double *alpha,
                                double gamma, const float *T, int64_t m, double *dec, int64_t dec_stride,
                                const PredictScratch &ws, hipStream_t s);
hipError_t launch_ovo_vote(const double *dec, int64_t m, int32_t k, int32_t *pred, hipStream_t s);

// Working-set solver (ws_smo.hip): one problem per launch, nwg sample-owning workgroups plus,
// when nwg > 1, one solving workgroup (launch nwg + 1).  Gram path, or row path (sp.gram NULL:
// every round each owner evaluates K(B, own samples) from the split rows; needs nwg >= 2 and
// q * per_wg <= ws_row_cap()).  Prob::slots holds
// [2][nwg][ws_list_words()] candidate words, Prob::slots2 [2][ng][ws_list_words()] group
// lists followed by ws_bcast_words() words for the solving workgroup's results; Ctl::t counts
// pair steps; rounds[problem] counts rounds (ws_slice_max() samples per workgroup at most; q
// even, 2..ws_q_max(); at most 16 lists per merge, so nwg <= 255 with g1 = ceil(sqrt(nwg))).
struct WsParams {
  SolveParams sp;    // steps = pair steps a launch may start rounds within
  int64_t *rounds;   // [nprob]
  double frac;       // local tolerance factor
  int32_t q;         // working-set size
  int32_t max_inner; // pair steps per round at most
  SplitX split;      // row path (sp.gram == NULL): split-fp16 rows of X, scales and norms
  float cexp;        // row path: -gamma * log2(e)
  int32_t pad;
  int64_t round_end; // a launch also ends once this many rounds are done
};
hipError_t launch_ws_solver(const WsParams &p, int32_t total_wg, hipStream_t s, int32_t *max_coresident);
int ws_slice_max();
int ws_q_max();
int64_t ws_list_words();
int64_t ws_bcast_words();
int ws_row_cap();

int solver_block_size(bool gram);
int max_per_thread(bool gram);

}  // namespace svmx

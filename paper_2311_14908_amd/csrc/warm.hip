// warm.hip -- f recomputed from given multipliers, for the warm start of a binary training:
// f_i = sum_j a_j y_j K_ij - y_i (the gradient of the dual the SMO steps keep, Section III.B),
// summed over the support vectors only (a_j > 0) in increasing index, one thread per sample.
#include "warm.hpp"

#include <math.h>

namespace svmx {

constexpr int WBS = 256;

__global__ void __launch_bounds__(WBS) f_from_alpha_k(const int32_t *__restrict__ sv, const double *__restrict__ coef,
                                                      int64_t nsv, const int32_t *__restrict__ y, int64_t n,
                                                      const float *__restrict__ G, int64_t ld,
                                                      const float *__restrict__ X, int64_t d, double gamma,
                                                      double *__restrict__ f) {
#pragma clang fp contract(off)
  const int64_t i = blockIdx.x * (int64_t)WBS + threadIdx.x;
  if (i >= n) return;
  double s = 0.0;
  for (int64_t k = 0; k < nsv; ++k) {
    const int64_t j = sv[k];
    double kij;
    if (G) {
      kij = (double)G[j * ld + i];
    } else {
      const float *xi = X + i * d, *xj = X + j * d;
      double d2 = 0.0;
      for (int64_t t = 0; t < d; ++t) {
        const double df = (double)xi[t] - (double)xj[t];
        d2 += df * df;
      }
      kij = exp(-gamma * d2);
    }
    s += coef[k] * kij;
  }
  f[i] = s - (double)y[i];
}

hipError_t launch_f_from_alpha(const int32_t *sv, const double *coef, int64_t nsv, const int32_t *y, int64_t n,
                               const float *G, int64_t ld, const float *X, int64_t d, double gamma, double *f,
                               hipStream_t s) {
  const int64_t blocks = (n + WBS - 1) / WBS;
  hipLaunchKernelGGL(f_from_alpha_k, dim3((unsigned)blocks), dim3(WBS), 0, s, sv, coef, nsv, y, n, G, ld, X, d, gamma,
                     f);
  return hipGetLastError();
}

}  // namespace svmx

// warm.hpp -- the warm start of a binary training (svm_options.alpha_init).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

// f_i = sum_k coef_k K(x_i, x_{sv_k}) - y_i for i < n, the sum over k in increasing order in fp64
// (coef_k = a y of support vector sv_k, the support vectors in increasing index).  K comes from
// the Gram (row sv_k, pitch ld) when G is not NULL, else from X [n][d] with the exact kernel
// exp(-gamma sum_t (x_it - x_jt)^2), the squared distance summed in fp64.
hipError_t launch_f_from_alpha(const int32_t *sv, const double *coef, int64_t nsv, const int32_t *y, int64_t n,
                               const float *G, int64_t ld, const float *X, int64_t d, double gamma, double *f,
                               hipStream_t s);

}  // namespace svmx

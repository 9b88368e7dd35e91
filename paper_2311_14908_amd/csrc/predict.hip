// predict.hip -- decision values d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b and one-vs-one votes.
//
// A workgroup stages TQ test samples in LDS and streams the training samples past them: a
// group of lanes takes one training sample with a_i > 0, accumulates its squared distance to
// each staged test sample in fp64, and adds a_i y_i exp(-gamma d^2) into per-group fp64 sums;
// the group sums are then combined in a fixed order, so results are deterministic.
#include "common.hpp"

#include <math.h>

namespace svmx {

constexpr int PBS = 256;
constexpr int TQ = 8;

struct PredMap {  // local training index j -> row of X, and its label
  int64_t off0, len0, off1;
  const int32_t *y;     // labels by row, or NULL: +1 for j < len0, else -1
  const int32_t *perm;  // sorted position -> row of X, or NULL (identity)
};

__device__ __forceinline__ int64_t pm_row(const PredMap &m, int64_t j) {
  const int64_t r = j < m.len0 ? m.off0 + j : m.off1 + (j - m.len0);
  return m.perm ? (int64_t)m.perm[r] : r;
}
__device__ __forceinline__ double pm_label(const PredMap &m, int64_t j) {
  return m.y ? (double)m.y[pm_row(m, j)] : (j < m.len0 ? 1.0 : -1.0);
}

template <int GS>
__global__ void __launch_bounds__(PBS) predict_k(const float *__restrict__ Xtr, int64_t d, PredMap map,
                                                 const double *__restrict__ alpha, int64_t ntr, double gamma,
                                                 const float *__restrict__ T, int64_t m, double b, double *dec,
                                                 int64_t dec_stride) {
  extern __shared__ float4 st4[];  // [TQ][d]
  float *st = reinterpret_cast<float *>(st4);
  __shared__ double part[PBS / GS][TQ];
  const int64_t q0 = (int64_t)blockIdx.x * TQ;
  const int nq = (int)(m - q0 < TQ ? m - q0 : TQ);
  for (int64_t e = threadIdx.x; e < (int64_t)TQ * d; e += PBS) {
    const int64_t q = e / d, k = e - q * d;
    st[e] = q < nq ? T[(q0 + q) * d + k] : 0.f;
  }
  __syncthreads();
  const int lig = threadIdx.x % GS, grp = threadIdx.x / GS;
  constexpr int NG = PBS / GS;
  double acc[TQ];
#pragma unroll
  for (int q = 0; q < TQ; ++q) acc[q] = 0.0;
  for (int64_t i = grp; i < ntr; i += NG) {
    const double ai = alpha[i];
    if (!(ai > 0.0)) continue;
    const float *xi = Xtr + pm_row(map, i) * d;
    double ds[TQ];
#pragma unroll
    for (int q = 0; q < TQ; ++q) ds[q] = 0.0;
    for (int64_t k = lig; k < d; k += GS) {
      const double v = (double)xi[k];
#pragma unroll
      for (int q = 0; q < TQ; ++q) {
        const double e = v - (double)st[q * d + k];
        ds[q] += e * e;
      }
    }
#pragma unroll
    for (int q = 0; q < TQ; ++q) {
      for (int o = GS >> 1; o > 0; o >>= 1) ds[q] += __shfl_xor(ds[q], o);
    }
    const double coef = ai * pm_label(map, i);
#pragma unroll
    for (int q = 0; q < TQ; ++q) acc[q] += coef * exp(-gamma * ds[q]);
  }
  if (lig == 0) {
#pragma unroll
    for (int q = 0; q < TQ; ++q) part[grp][q] = acc[q];
  }
  __syncthreads();
  if (threadIdx.x < nq) {
    double s = 0.0;
    for (int g = 0; g < NG; ++g) s += part[g][threadIdx.x];
    dec[(q0 + threadIdx.x) * dec_stride] = s - b;
  }
}

hipError_t launch_predict_map(const float *Xtr, int64_t d, int64_t off0, int64_t len0, int64_t off1,
                              const int32_t *y, const int32_t *perm, const double *alpha, int64_t ntr, double gamma,
                              const float *T, int64_t m, double b, double *dec, int64_t dec_stride, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  PredMap map{off0, len0, off1, y, perm};
  const int64_t blocks = (m + TQ - 1) / TQ;
  const size_t shmem = (size_t)TQ * d * sizeof(float);
  int gs = 1;
  while (gs < d && gs < 64) gs <<= 1;
  const void *fn;
  switch (gs) {
    case 1: fn = reinterpret_cast<const void *>(&predict_k<1>); break;
    case 2: fn = reinterpret_cast<const void *>(&predict_k<2>); break;
    case 4: fn = reinterpret_cast<const void *>(&predict_k<4>); break;
    case 8: fn = reinterpret_cast<const void *>(&predict_k<8>); break;
    case 16: fn = reinterpret_cast<const void *>(&predict_k<16>); break;
    case 32: fn = reinterpret_cast<const void *>(&predict_k<32>); break;
    default: fn = reinterpret_cast<const void *>(&predict_k<64>); break;
  }
  if (shmem > 48 * 1024) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return e;
  }
  void *args[] = {(void *)&Xtr, &d, &map, (void *)&alpha, &ntr, &gamma, (void *)&T, &m, &b, &dec, &dec_stride};
  return hipLaunchKernel(fn, dim3((unsigned)blocks), dim3(PBS), args, shmem, s);
}

// pred[q] = class with most votes over the k(k-1)/2 pairs (a<b, lexicographic), pair (a,b)
// voting a iff its decision value is > 0; ties to the smaller class.
__global__ void ovo_vote_k(const double *__restrict__ dec, int64_t m, int32_t k, int32_t *__restrict__ pred) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (q >= m) return;
  const int P = k * (k - 1) / 2;
  int votes[64];
  for (int c = 0; c < k; ++c) votes[c] = 0;
  int p = 0;
  for (int a = 0; a < k; ++a)
    for (int bb = a + 1; bb < k; ++bb, ++p) votes[dec[q * P + p] > 0.0 ? a : bb]++;
  int best = 0;
  for (int c = 1; c < k; ++c)
    if (votes[c] > votes[best]) best = c;
  pred[q] = best;
}

hipError_t launch_ovo_vote(const double *dec, int64_t m, int32_t k, int32_t *pred, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  hipLaunchKernelGGL(ovo_vote_k, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, s, dec, m, k, pred);
  return hipGetLastError();
}

}  // namespace svmx

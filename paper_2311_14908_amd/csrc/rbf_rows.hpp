// rbf_rows.hpp -- device routines that evaluate RBF kernel values between two staged rows
// (x_u, x_l) and samples of X.  Shared by the solver's row path, its K_ul, and the exposed
// kernel-row entry point, so all of them produce bit-identical values.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace svmx {

// Lanes per sample: a power of two covering d (float4 units when VEC4), at most 64.
__device__ __forceinline__ int group_size_for(int64_t d, bool vec4) {
  const int64_t units = vec4 ? (d + 3) / 4 : d;
  int gs = 1;
  while (gs < units && gs < 64) gs <<= 1;
  return gs;
}

__device__ __forceinline__ double sqdiff_acc(float v, float a, double acc) {
  const float e = v - a;  // fp32 difference (relative error 6e-8), squared and summed in fp64
  return __builtin_fma((double)e, (double)e, acc);
}

// Squared distances from x_u (sxu) and x_l (sxl) to nb <= SB samples xs[0..nb), computed by a
// group of gs lanes: lane `lig` accumulates the features k = lig, lig+gs, ... (float4 units
// when VEC4) in increasing order, then the group combines its partial sums by the butterfly
// xor gs/2, ..., 1, leaving the totals in every lane of the group.  The per-sample arithmetic
// does not depend on SB or on which samples share a batch.
template <bool VEC4, int SB>
__device__ __forceinline__ void dist2_batch(const float *const *xs, int nb, const float *sxu, const float *sxl, int64_t d,
                                            int lig, int gs, double *du, double *dl) {
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    du[s] = 0.0;
    dl[s] = 0.0;
  }
  if (VEC4) {
    const int64_t d4 = d >> 2;
    const float4 *u4 = reinterpret_cast<const float4 *>(sxu);
    const float4 *l4 = reinterpret_cast<const float4 *>(sxl);
    for (int64_t k = lig; k < d4; k += gs) {
      const float4 a = u4[k], b = l4[k];
      float4 v[SB];
#pragma unroll
      for (int s = 0; s < SB; ++s)
        if (s < nb) v[s] = reinterpret_cast<const float4 *>(xs[s])[k];
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        if (s < nb) {
          du[s] = sqdiff_acc(v[s].x, a.x, du[s]);
          du[s] = sqdiff_acc(v[s].y, a.y, du[s]);
          du[s] = sqdiff_acc(v[s].z, a.z, du[s]);
          du[s] = sqdiff_acc(v[s].w, a.w, du[s]);
          dl[s] = sqdiff_acc(v[s].x, b.x, dl[s]);
          dl[s] = sqdiff_acc(v[s].y, b.y, dl[s]);
          dl[s] = sqdiff_acc(v[s].z, b.z, dl[s]);
          dl[s] = sqdiff_acc(v[s].w, b.w, dl[s]);
        }
      }
    }
  } else {
    for (int64_t k = lig; k < d; k += gs) {
      const float a = sxu[k], b = sxl[k];
      float v[SB];
#pragma unroll
      for (int s = 0; s < SB; ++s)
        if (s < nb) v[s] = xs[s][k];
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        if (s < nb) {
          du[s] = sqdiff_acc(v[s], a, du[s]);
          dl[s] = sqdiff_acc(v[s], b, dl[s]);
        }
      }
    }
  }
  for (int o = gs >> 1; o > 0; o >>= 1) {
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      du[s] += __shfl_xor(du[s], o);
      dl[s] += __shfl_xor(dl[s], o);
    }
  }
}

// K = exp(-gamma d^2) rounded to fp32.
__device__ __forceinline__ float rbf_of(double d2, double gamma) { return (float)exp(-gamma * d2); }

// Value v (0..2*SB) of a batch: the u row for v < SB, else the l row.
template <int SB>
__device__ __forceinline__ double batch_value(const double *du, const double *dl, int v) {
  double r = 0.0;
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    r = (v == s) ? du[s] : r;
    r = (v == SB + s) ? dl[s] : r;
  }
  return r;
}

}  // namespace svmx

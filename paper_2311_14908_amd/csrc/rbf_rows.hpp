// rbf_rows.hpp -- device routines that evaluate RBF kernel values between two rows (x_u, x_l)
// and samples of X.  Shared by the solver's row path, its K_ul, and the exposed kernel-row
// entry point, so all of them produce bit-identical values.
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

// Sum of `v` over aligned groups of gs lanes (gs a power of two <= 64), in every lane of the
// group.  Levels 1, 2, 4, 8 use DPP (quad permutes, half-row and row mirrors: after each level
// all lanes of the combined block hold the same value, so a mirror partner is as good as the
// xor partner); levels 16 and 32 use lane permutes.  fp64 addition is commutative, so every
// lane ends with the same bits.
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int hi = __builtin_amdgcn_update_dpp((int)(b >> 32), (int)(b >> 32), CTRL, 0xf, 0xf, false);
  const int lo = __builtin_amdgcn_update_dpp((int)b, (int)b, CTRL, 0xf, 0xf, false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double group_sum(double v, int gs) {
  if (gs > 1) v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  if (gs > 2) v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  if (gs > 4) v += dpp_d<0x141>(v);  // row_half_mirror
  if (gs > 8) v += dpp_d<0x140>(v);  // row_mirror
  if (gs > 16) v += __shfl_xor(v, 16);
  if (gs > 32) v += __shfl_xor(v, 32);
  return v;
}

// Squared distances from x_u (xu) and x_l (xl) to nb <= SB samples xs[0..nb), computed by a
// group of gs lanes: lane `lig` accumulates the features k = lig, lig+gs, ... (float4 units
// when VEC4) in increasing order -- all loads of a chunk of MAXM such positions are issued
// before any arithmetic -- then the group sums its lanes with group_sum.  The arithmetic of a
// sample does not depend on SB, on the batch it shares, or on where x_u / x_l are read from.
// Called with the whole wave active (nb, gs uniform per group).
template <bool VEC4, int SB, int MAXM>
__device__ __forceinline__ void dist2_batch(const float *const *xs, int nb, const float *xu, const float *xl, int64_t d,
                                            int lig, int gs, double *du, double *dl) {
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    du[s] = 0.0;
    dl[s] = 0.0;
  }
  if (VEC4) {
    const int64_t d4 = d >> 2;
    const float4 *u4 = reinterpret_cast<const float4 *>(xu);
    const float4 *l4 = reinterpret_cast<const float4 *>(xl);
    for (int64_t k0 = lig; k0 < d4; k0 += (int64_t)gs * MAXM) {
      float4 a[MAXM], b[MAXM], v[SB][MAXM];
#pragma unroll
      for (int m = 0; m < MAXM; ++m) {
        const int64_t k = k0 + (int64_t)m * gs;
        if (k < d4) {
          a[m] = u4[k];
          b[m] = l4[k];
#pragma unroll
          for (int s = 0; s < SB; ++s)
            if (s < nb) v[s][m] = reinterpret_cast<const float4 *>(xs[s])[k];
        }
      }
#pragma unroll
      for (int m = 0; m < MAXM; ++m) {
        if (k0 + (int64_t)m * gs < d4) {
#pragma unroll
          for (int s = 0; s < SB; ++s) {
            if (s < nb) {
              du[s] = sqdiff_acc(v[s][m].x, a[m].x, du[s]);
              du[s] = sqdiff_acc(v[s][m].y, a[m].y, du[s]);
              du[s] = sqdiff_acc(v[s][m].z, a[m].z, du[s]);
              du[s] = sqdiff_acc(v[s][m].w, a[m].w, du[s]);
              dl[s] = sqdiff_acc(v[s][m].x, b[m].x, dl[s]);
              dl[s] = sqdiff_acc(v[s][m].y, b[m].y, dl[s]);
              dl[s] = sqdiff_acc(v[s][m].z, b[m].z, dl[s]);
              dl[s] = sqdiff_acc(v[s][m].w, b[m].w, dl[s]);
            }
          }
        }
      }
    }
  } else {
    for (int64_t k0 = lig; k0 < d; k0 += (int64_t)gs * MAXM) {
      float a[MAXM], b[MAXM], v[SB][MAXM];
#pragma unroll
      for (int m = 0; m < MAXM; ++m) {
        const int64_t k = k0 + (int64_t)m * gs;
        if (k < d) {
          a[m] = xu[k];
          b[m] = xl[k];
#pragma unroll
          for (int s = 0; s < SB; ++s)
            if (s < nb) v[s][m] = xs[s][k];
        }
      }
#pragma unroll
      for (int m = 0; m < MAXM; ++m) {
        if (k0 + (int64_t)m * gs < d) {
#pragma unroll
          for (int s = 0; s < SB; ++s) {
            if (s < nb) {
              du[s] = sqdiff_acc(v[s][m], a[m], du[s]);
              dl[s] = sqdiff_acc(v[s][m], b[m], dl[s]);
            }
          }
        }
      }
    }
  }
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    du[s] = group_sum(du[s], gs);
    dl[s] = group_sum(dl[s], gs);
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

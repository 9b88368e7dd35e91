// rbf_rows.hpp -- device routine that evaluates RBF kernel values between staged rows and
// samples of X.  Shared by the solver's row path and by the exposed kernel-row entry point,
// so both produce bit-identical values.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

// Row path: squared distances from x_u and x_l (staged in LDS) to the workgroup's own
// samples, by groups of GS lanes per sample; fp64 accumulation, fp32 result exp(-g d^2).
// The same routine gives K_ul, so a kernel value never depends on which side computed it.
__device__ __forceinline__ int group_size_for(int64_t d, bool vec4) {
  int64_t units = vec4 ? (d + 3) / 4 : d;
  int gs = 1;
  while (gs < units && gs < 64) gs <<= 1;
  return gs;
}

template <bool VEC4>
__device__ __forceinline__ void dist2_group(const float *__restrict__ xj, const float *sxu, const float *sxl, int64_t d,
                                            int lane_in_group, int gs, double &du, double &dl) {
  du = 0.0;
  dl = 0.0;
  if (VEC4) {
    const int64_t d4 = d >> 2;
    const float4 *x4 = reinterpret_cast<const float4 *>(xj);
    const float4 *u4 = reinterpret_cast<const float4 *>(sxu);
    const float4 *l4 = reinterpret_cast<const float4 *>(sxl);
    for (int64_t k = lane_in_group; k < d4; k += gs) {
      const float4 v = x4[k], a = u4[k], b = l4[k];
      double e;
      e = (double)v.x - (double)a.x; du += e * e;
      e = (double)v.y - (double)a.y; du += e * e;
      e = (double)v.z - (double)a.z; du += e * e;
      e = (double)v.w - (double)a.w; du += e * e;
      e = (double)v.x - (double)b.x; dl += e * e;
      e = (double)v.y - (double)b.y; dl += e * e;
      e = (double)v.z - (double)b.z; dl += e * e;
      e = (double)v.w - (double)b.w; dl += e * e;
    }
  } else {
    for (int64_t k = lane_in_group; k < d; k += gs) {
      const double v = (double)xj[k];
      double e = v - (double)sxu[k];
      du += e * e;
      e = v - (double)sxl[k];
      dl += e * e;
    }
  }
  for (int o = gs >> 1; o > 0; o >>= 1) {
    du += __shfl_xor(du, o);
    dl += __shfl_xor(dl, o);
  }
}

}  // namespace svmx

// rbf_rows.hpp -- device routines that evaluate RBF kernel values between two rows (x_u, x_l)
// and samples of X as a GEMV: fp32 dot products against both rows in one pass over the
// samples, combined with squared norms computed the same way.  Shared by the solver's row
// path, its K_ul, and
// the exposed kernel-row entry point, so all of them produce bit-identical values.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "solver_params.hpp"

namespace svmx {

// Feature positions (float4 units when VEC4) each lane of a group takes in the first register
// block of a row evaluation.
constexpr int ROW_POSITIONS = 4;

// Lanes per sample: the smallest power of two gs with ROW_POSITIONS * gs covering the row's
// units, at most 64 (longer rows continue in later blocks).  So a short row does not leave most
// of a lane's positions masked: its lanes each take up to ROW_POSITIONS units, and a wave holds
// 64 / gs samples at once.
__host__ __device__ __forceinline__ int group_size_for(int64_t d, bool vec4) {
  const int64_t units = vec4 ? (d + 3) / 4 : d;
  int gs = 1;
  while ((int64_t)ROW_POSITIONS * gs < units && gs < 64) gs <<= 1;
  return gs;
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

// Per-lane operand type: a float4 of features when VEC4, else one float.
template <bool VEC4> struct Lane;
template <> struct Lane<true> {
  typedef float4 T;
  static __device__ __forceinline__ float4 scale(float4 v, float m) { return make_float4(v.x * m, v.y * m, v.z * m, v.w * m); }
  static __device__ __forceinline__ float dot(float4 v, float4 a, float acc) {
    acc = __builtin_fmaf(v.x, a.x, acc);
    acc = __builtin_fmaf(v.y, a.y, acc);
    acc = __builtin_fmaf(v.z, a.z, acc);
    return __builtin_fmaf(v.w, a.w, acc);
  }
};
template <> struct Lane<false> {
  typedef float T;
  static __device__ __forceinline__ float scale(float v, float m) { return v * m; }
  static __device__ __forceinline__ float dot(float v, float a, float acc) { return __builtin_fmaf(v, a, acc); }
};

// Squared norm of row x, computed exactly as dot_batch computes the dot product of a sample
// with itself (a group of gs lanes; lane `lig` accumulates positions lig, lig+gs, ... in
// increasing order in fp32, the group sums the partials in fp64).  So |x|^2 + |x|^2 - 2 x.x is
// exactly 0 for identical rows (K = 1 on the diagonal and between duplicates), and every caller
// gets the same bits for a row.
template <bool VEC4>
__device__ __forceinline__ double sq_norm(const float *x, int64_t d, int lig, int gs) {
  typedef typename Lane<VEC4>::T T;
  const SVMX_GLOBAL T *p = gp(reinterpret_cast<const T *>(x));
  const int64_t units = VEC4 ? (d >> 2) : d;
  float acc = 0.f;
  for (int64_t k = lig; k < units; k += gs) acc = Lane<VEC4>::dot(p[k], p[k], acc);
  return group_sum((double)acc, gs);
}

// Operands of a pair of rows (x_u, x_l) held by one lane for the first MAXM positions
// k = lig + m*gs (float4 units when VEC4); positions past d are zeroed and masked.
template <bool VEC4, int MAXM>
struct RowPair {
  typename Lane<VEC4>::T a[MAXM], b[MAXM];
  float mk[MAXM];  // 1 inside d, 0 past it
};

template <bool VEC4, int MAXM>
__device__ __forceinline__ void load_pair(RowPair<VEC4, MAXM> &r, const float *xu, const float *xl, int64_t d, int lig,
                                          int gs) {
  typedef typename Lane<VEC4>::T T;
  const int64_t units = VEC4 ? (d >> 2) : d;
#pragma unroll
  for (int m = 0; m < MAXM; ++m) {
    const int64_t k = lig + (int64_t)m * gs;
    const int64_t kk = k < units ? k : units - 1;
    r.mk[m] = k < units ? 1.f : 0.f;
    r.a[m] = Lane<VEC4>::scale(gp(reinterpret_cast<const T *>(xu))[kk], r.mk[m]);
    r.b[m] = Lane<VEC4>::scale(gp(reinterpret_cast<const T *>(xl))[kk], r.mk[m]);
  }
}

// Unit k of a sample row; XLDS: the row sits in LDS (the pointer is addressed as LDS, so the
// load is an LDS read even where the compiler cannot trace the pointer to its array).
// (The host pass of the compiler has no LDS address space and never runs this.)
template <bool XLDS, typename T>
__device__ __forceinline__ T row_unit(const float *row, int64_t k) {
#if __HIP_DEVICE_COMPILE__
  if constexpr (XLDS) return ((__attribute__((address_space(3))) const T *)row)[k];
#endif
  return gp(reinterpret_cast<const T *>(row))[k];
}

// Block 0 of nb <= SB samples xs[0..nb): positions k = lig + m*gs, m < MAXM (float4 units when
// VEC4), for one lane of a group of gs lanes.  Loads are unconditional (clamped positions and
// samples), so they issue back to back; the sample rows may sit in HBM or in LDS.
template <bool VEC4, int SB, int MAXM, bool XLDS = false>
__device__ __forceinline__ void load_block0(typename Lane<VEC4>::T (&v)[SB][MAXM], const float *const *xs, int nb,
                                            int64_t d, int lig, int gs) {
  typedef typename Lane<VEC4>::T T;
  const int64_t units = VEC4 ? (d >> 2) : d;
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    const float *row = xs[s < nb ? s : nb - 1];
#pragma unroll
    for (int m = 0; m < MAXM; ++m) {
      const int64_t k = lig + (int64_t)m * gs;
      v[s][m] = row_unit<XLDS, T>(row, k < units ? k : units - 1);
    }
  }
}

// fp32 partial dot products of one lane against x_u (fu) and x_l (fl): block 0 from v (as
// loaded by load_block0), later blocks of MAXM positions loaded here.  The lane accumulates the
// products of its positions k = lig, lig+gs, ... in increasing order, so a sample's partials do
// not depend on SB, on the batch it shares, on where its row is read from, or on which of the
// two rows is x_u.
template <bool VEC4, int SB, int MAXM, bool XLDS = false>
__device__ __forceinline__ void dot_partials(const typename Lane<VEC4>::T (&v0)[SB][MAXM], const float *const *xs,
                                             int nb, const float *xu, const float *xl, int64_t d, int lig, int gs,
                                             const RowPair<VEC4, MAXM> &r, float (&fu)[SB], float (&fl)[SB]) {
  typedef typename Lane<VEC4>::T T;
  const int64_t units = VEC4 ? (d >> 2) : d;
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    fu[s] = 0.f;
    fl[s] = 0.f;
#pragma unroll
    for (int m = 0; m < MAXM; ++m) {  // r.a / r.b are zero past d (X is finite)
      fu[s] = Lane<VEC4>::dot(v0[s][m], r.a[m], fu[s]);
      fl[s] = Lane<VEC4>::dot(v0[s][m], r.b[m], fl[s]);
    }
  }
  // Later blocks: MAXL positions at a time (fewer registers than block 0; they occur only for
  // rows longer than MAXM * gs units).
  constexpr int MAXL = MAXM > 2 ? 2 : MAXM;
  for (int64_t k0 = lig + (int64_t)gs * MAXM; k0 < units; k0 += (int64_t)gs * MAXL) {
    T a[MAXL], b[MAXL], v[SB][MAXL];
    float mk[MAXL];
#pragma unroll
    for (int m = 0; m < MAXL; ++m) {
      const int64_t k = k0 + (int64_t)m * gs;
      const int64_t kk = k < units ? k : units - 1;
      mk[m] = k < units ? 1.f : 0.f;
      a[m] = gp(reinterpret_cast<const T *>(xu))[kk];
      b[m] = gp(reinterpret_cast<const T *>(xl))[kk];
#pragma unroll
      for (int s = 0; s < SB; ++s) v[s][m] = row_unit<XLDS, T>(xs[s < nb ? s : nb - 1], kk);
    }
#pragma unroll
    for (int m = 0; m < MAXL; ++m) {
      const T am = Lane<VEC4>::scale(a[m], mk[m]), bm = Lane<VEC4>::scale(b[m], mk[m]);
#pragma unroll
      for (int s = 0; s < SB; ++s) {
        fu[s] = Lane<VEC4>::dot(v[s][m], am, fu[s]);
        fl[s] = Lane<VEC4>::dot(v[s][m], bm, fl[s]);
      }
    }
  }
}

// Dot products of nb <= SB samples xs[0..nb) with x_u (pu) and x_l (pl), computed by a group
// of gs lanes: the lanes' fp32 partials (dot_partials) summed over the group in fp64
// (group_sum).  Called with the whole wave active (nb, gs uniform per group).
template <bool VEC4, int SB, int MAXM>
__device__ __forceinline__ void dot_batch(const float *const *xs, int nb, const float *xu, const float *xl, int64_t d,
                                          int lig, int gs, const RowPair<VEC4, MAXM> &r, double *pu, double *pl) {
  typename Lane<VEC4>::T v[SB][MAXM];
  load_block0<VEC4, SB, MAXM>(v, xs, nb, d, lig, gs);
  float fu[SB], fl[SB];
  dot_partials<VEC4, SB, MAXM>(v, xs, nb, xu, xl, d, lig, gs, r, fu, fl);
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    pu[s] = group_sum((double)fu[s], gs);
    pl[s] = group_sum((double)fl[s], gs);
  }
}

// a + b of the two results of a gfx950 lane swap of the 64-bit values x (as the instruction's
// destination) and y (its source): permlane16_swap exchanges the odd rows of 16 of x with the
// even rows of y, permlane32_swap the high half of x with the low half of y.  So with D = 16,
// a lane of an even row gets x(own) + x(lane + 16) and a lane of an odd row y(lane - 16) +
// y(own); with D = 32 likewise for the halves.
template <int D>
__device__ __forceinline__ double swap_sum(double x, double y) {
  const unsigned long long bx = (unsigned long long)__double_as_longlong(x);
  const unsigned long long by = (unsigned long long)__double_as_longlong(y);
  unsigned a_hi, a_lo, b_hi, b_lo;
  if (D == 16) {
    const auto h = __builtin_amdgcn_permlane16_swap((unsigned)(bx >> 32), (unsigned)(by >> 32), false, false);
    const auto l = __builtin_amdgcn_permlane16_swap((unsigned)bx, (unsigned)by, false, false);
    a_hi = h[0]; b_hi = h[1]; a_lo = l[0]; b_lo = l[1];
  } else {
    const auto h = __builtin_amdgcn_permlane32_swap((unsigned)(bx >> 32), (unsigned)(by >> 32), false, false);
    const auto l = __builtin_amdgcn_permlane32_swap((unsigned)bx, (unsigned)by, false, false);
    a_hi = h[0]; b_hi = h[1]; a_lo = l[0]; b_lo = l[1];
  }
  const double a = __longlong_as_double((long long)(((unsigned long long)a_hi << 32) | a_lo));
  const double b = __longlong_as_double((long long)(((unsigned long long)b_hi << 32) | b_lo));
  return a + b;
}

// The group sums of the fp32 partials of nb <= SB samples, written to du[s] (against x_u) and
// dl[s] (against x_l), s < nb.  The same butterfly as group_sum, and so the same bits (fp64
// addition is commutative, and every level adds the same two partial sums), but for gs >= 32
// the levels across rows and halves are lane swaps that also transpose: after level 16 the
// lanes of even rows hold the u sums and those of odd rows the l sums, after level 32 the low
// half holds sample s and the high half sample s + 1.  That halves the work of those levels.
template <int SB>
__device__ __forceinline__ void group_sums_store(const float (&fu)[SB], const float (&fl)[SB], int nb, int gs, int lig,
                                                 double *du, double *dl) {
  double u[SB], l[SB];
#pragma unroll
  for (int s = 0; s < SB; ++s) {
    u[s] = (double)fu[s];
    l[s] = (double)fl[s];
    if (gs > 1) { u[s] += dpp_d<0xB1>(u[s]); l[s] += dpp_d<0xB1>(l[s]); }    // quad_perm [1,0,3,2]
    if (gs > 2) { u[s] += dpp_d<0x4E>(u[s]); l[s] += dpp_d<0x4E>(l[s]); }    // quad_perm [2,3,0,1]
    if (gs > 4) { u[s] += dpp_d<0x141>(u[s]); l[s] += dpp_d<0x141>(l[s]); }  // row_half_mirror
    if (gs > 8) { u[s] += dpp_d<0x140>(u[s]); l[s] += dpp_d<0x140>(l[s]); }  // row_mirror
  }
  if (gs <= 16) {
    if (lig == 0) {
#pragma unroll
      for (int s = 0; s < SB; ++s)
        if (s < nb) { du[s] = u[s]; dl[s] = l[s]; }
    }
    return;
  }
  double t[SB];
#pragma unroll
  for (int s = 0; s < SB; ++s) t[s] = swap_sum<16>(u[s], l[s]);
  double *const side = (lig & 16) ? dl : du;
  if (gs == 32) {
    if ((lig & 15) == 0) {
#pragma unroll
      for (int s = 0; s < SB; ++s)
        if (s < nb) side[s] = t[s];
    }
    return;
  }
  const int half = lig >> 5;
#pragma unroll
  for (int s = 0; s < SB; s += 2) {
    const double v = swap_sum<32>(t[s], s + 1 < SB ? t[s + 1] : t[s]);
    const int ss = s + half;
    if ((lig & 15) == 0 && ss < nb && ss < SB) side[ss] = v;
  }
}

// K = exp(-gamma d^2) rounded to fp32, with d^2 = (|x|^2 + |y|^2) - 2 x.y from the norms and
// the dot product (clamped at 0 against cancellation).  Not contracted, so the bits do not
// depend on the caller; (|x|^2 + |y|^2) is symmetric in x and y.
__device__ __forceinline__ float rbf_from_dot(double nx, double ny, double dot, double gamma) {
#pragma clang fp contract(off)
  double d2 = (nx + ny) - 2.0 * dot;
  d2 = d2 > 0.0 ? d2 : 0.0;
  return (float)exp(-gamma * d2);
}

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

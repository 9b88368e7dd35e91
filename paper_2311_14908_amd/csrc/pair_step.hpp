// pair_step.hpp -- device pieces shared by the solver kernels: DPP wave reductions with
// index tie-breaking, relaxed agent-scope word access for the exchanges, and the
// two-multiplier step (paper, Section III.B) with its gradient update.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "solver_params.hpp"

namespace svmx {

constexpr int IBIG = 0x7fffffff;

__device__ __forceinline__ bool lt_min(double v2, int i2, double v, int i) { return v2 < v || (v2 == v && i2 < i); }
__device__ __forceinline__ bool gt_max(double v2, int i2, double v, int i) { return v2 > v || (v2 == v && i2 < i); }

__device__ __forceinline__ double readlane_d(double v, int lane) {
  const long long b = __double_as_longlong(v);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(b >> 32), lane);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)b, lane);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_mov(int v) {
  return __builtin_amdgcn_update_dpp(v, v, CTRL, ROW_MASK, 0xf, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_mov_d(double v) {
  const long long b = __double_as_longlong(v);
  const unsigned hi = (unsigned)dpp_mov<CTRL, ROW_MASK>((int)(b >> 32));
  const unsigned lo = (unsigned)dpp_mov<CTRL, ROW_MASK>((int)b);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

template <int CTRL>
__device__ __forceinline__ double dpp_full_d(double v) {  // every lane reads its source lane
  const long long b = __double_as_longlong(v);
  const unsigned hi = (unsigned)__builtin_amdgcn_mov_dpp((int)(b >> 32), CTRL, 0xF, 0xF, false);
  const unsigned lo = (unsigned)__builtin_amdgcn_mov_dpp((int)b, CTRL, 0xF, 0xF, false);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Wave-wide min (MAX = false) or max (MAX = true) of v, returned to every lane.  DPP row
// operations (xor 1 and 2 inside quads, rotations by 4 and 8 inside rows of 16, then the
// row-15 and row-31 broadcasts) leave the result in lane 63.  Lanes outside a broadcast's row
// mask keep their own value, which min/max leaves unchanged.  Compare and select: the values
// are finite or +-inf, so fmin/fmax's quieting of NaN inputs is not needed (either zero may
// come out of -0 against +0; callers compare with ==, for which they are equal).
template <bool MAX>
__device__ __forceinline__ double wave_extreme(double v) {
#define SVMX_EXT_FULL(CTRL)                           \
  {                                                   \
    const double o = dpp_full_d<CTRL>(v);             \
    v = MAX ? (o > v ? o : v) : (o < v ? o : v);      \
  }
#define SVMX_EXT_MASK(CTRL, RM)                       \
  {                                                   \
    const double o = dpp_mov_d<CTRL, RM>(v);          \
    v = MAX ? (o > v ? o : v) : (o < v ? o : v);      \
  }
  SVMX_EXT_FULL(0xB1)         // quad_perm [1,0,3,2]
  SVMX_EXT_FULL(0x4E)         // quad_perm [2,3,0,1]
  SVMX_EXT_FULL(0x124)        // row_ror:4
  SVMX_EXT_FULL(0x128)        // row_ror:8
  SVMX_EXT_MASK(0x142, 0xA)   // row_bcast:15 -> rows 1, 3
  SVMX_EXT_MASK(0x143, 0xC)   // row_bcast:31 -> rows 2, 3
#undef SVMX_EXT_FULL
#undef SVMX_EXT_MASK
  return readlane_d(v, 63);
}

// Wave-wide min of a and max of b, returned to every lane: the DPP pattern of wave_extreme
// (quad permutes, row rotations, then the row-15 and row-31 broadcasts into lane 63) with
// compare-and-select (the values are finite or +-inf, so no NaN canonicalization) and the
// two chains interleaved round by round.
__device__ __forceinline__ void wave_minmax(double &a, double &b) {
#define SVMX_MM_FULL(CTRL)                       \
  {                                              \
    const double oa = dpp_full_d<CTRL>(a);       \
    const double ob = dpp_full_d<CTRL>(b);       \
    a = oa < a ? oa : a;                         \
    b = ob > b ? ob : b;                         \
  }
#define SVMX_MM_MASK(CTRL, RM)                   \
  {                                              \
    const double oa = dpp_mov_d<CTRL, RM>(a);    \
    const double ob = dpp_mov_d<CTRL, RM>(b);    \
    a = oa < a ? oa : a;                         \
    b = ob > b ? ob : b;                         \
  }
  SVMX_MM_FULL(0xB1)      // quad_perm [1,0,3,2]
  SVMX_MM_FULL(0x4E)      // quad_perm [2,3,0,1]
  SVMX_MM_FULL(0x124)     // row_ror:4
  SVMX_MM_FULL(0x128)     // row_ror:8
  SVMX_MM_MASK(0x142, 0xA)  // row_bcast:15 -> rows 1, 3
  SVMX_MM_MASK(0x143, 0xC)  // row_bcast:31 -> rows 2, 3
#undef SVMX_MM_FULL
#undef SVMX_MM_MASK
  a = readlane_d(a, 63);
  b = readlane_d(b, 63);
}

// Wave-wide min of an int, returned to every lane (same DPP pattern).
__device__ __forceinline__ int wave_min_int(int v) {
  v = min(v, dpp_mov<0xB1, 0xF>(v));
  v = min(v, dpp_mov<0x4E, 0xF>(v));
  v = min(v, dpp_mov<0x124, 0xF>(v));
  v = min(v, dpp_mov<0x128, 0xF>(v));
  v = min(v, dpp_mov<0x142, 0xA>(v));
  v = min(v, dpp_mov<0x143, 0xC>(v));
  return __builtin_amdgcn_readlane(v, 63);
}

// Lane of the winner among the lanes with `hit` (those holding the extreme value): the one with
// the smallest index i; an index reduction runs only when several lanes tie.
__device__ __forceinline__ int tie_lane(bool hit, int i) {
  const unsigned long long tie = (unsigned long long)__ballot(hit);
  if (__popcll(tie) == 1) return __ffsll(tie) - 1;
  const int best = wave_min_int(hit ? i : IBIG);
  return __ffsll((unsigned long long)__ballot(hit && i == best)) - 1;
}

// Lane holding the winner of one side: the extreme value, then the smallest index among the
// lanes holding it.  This is the (value, index) lexicographic order: -0 and +0 compare equal.
template <bool MAX>
__device__ __forceinline__ int winner_lane(double v, int i) {
  const double rv = wave_extreme<MAX>(v);
  return tie_lane(v == rv, i);
}

__device__ __forceinline__ void st_word(u64 *p, u64 v) {
  __hip_atomic_store(gp(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ u64 ld_word(const u64 *p) {
  return __hip_atomic_load(gp(const_cast<u64 *>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 2x2 sub-problem on (u, l): eta = K_uu + K_ll - 2 K_ul with K_uu = K_ll = 1 for the RBF
// kernel, the box [L, H] on a_l, the partner clamped to [0, C], values within 1e-12 C of a
// bound snapped onto it.  Written without contraction so the fp64 rounding is that of the
// plain expression.
struct PairStep {
  double au, al;  // new multipliers of u and l
};

__device__ __forceinline__ PairStep solve_pair(double C, double bu, double bl, double au, double al, double yu,
                                               double yl, double kul) {
#pragma clang fp contract(off)
  double eta = (1.0 + 1.0) - 2.0 * kul;
  if (eta <= 0.0) eta = 1e-12;
  const double s = yu * yl;
  double L, H;
  if (s < 0) {
    L = fmax(0.0, al - au);
    H = fmin(C, C + al - au);
  } else {
    L = fmax(0.0, au + al - C);
    H = fmin(C, au + al);
  }
  double aln = al + yl * (bu - bl) / eta;
  aln = aln < L ? L : (aln > H ? H : aln);
  double aun = au + s * (al - aln);
  aun = aun < 0.0 ? 0.0 : (aun > C ? C : aun);
  const double snap = 1e-12 * C;
  if (fabs(aln) <= snap) aln = 0.0;
  if (fabs(aln - C) <= snap) aln = C;
  if (fabs(aun) <= snap) aun = 0.0;
  if (fabs(aun - C) <= snap) aun = C;
  return PairStep{aun, aln};
}

// f_j + (c_u K_uj + c_l K_lj), rounded as written (no contraction), so that every solver
// variant -- whatever its unrolling -- produces the same bits.
__device__ __forceinline__ double f_update(double f, double cu, float ku, double cl, float kl) {
#pragma clang fp contract(off)
  return f + (cu * (double)ku + cl * (double)kl);
}

}  // namespace svmx

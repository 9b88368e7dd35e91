// solver_params.hpp -- the data the persistent SMO solver kernel reads: per-problem control
// blocks, problem descriptors and launch parameters (shared by the host and the kernel).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

typedef unsigned long long u64;

// Global-memory view of a pointer.  The kernels reach global memory through pointers held in
// parameter blocks and descriptors; the compiler cannot tell their address space and would use
// FLAT instructions, which also count against the LDS wait counter, so every wait for an LDS
// access (each barrier, each LDS hand-off) would wait for outstanding global loads and stores
// as well.  Accesses through gp() are global instructions.
#if defined(__HIP_DEVICE_COMPILE__) && __HIP_DEVICE_COMPILE__
#define SVMX_GLOBAL __attribute__((address_space(1)))
#else
#define SVMX_GLOBAL
#endif
template <class T>
__host__ __device__ __forceinline__ SVMX_GLOBAL T *gp(T *p) {
  return (SVMX_GLOBAL T *)p;
}

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

constexpr int SLOT_WORDS = 16;  // 6 used; a record sits alone in one 128-byte line

// Rank that reduces the records (or merges the lists) of first-level group g, whose members are
// ranks g g1 .. min(nwg, g g1 + g1) - 1: the member whose workgroup runs on XCD g mod 8 (a launch
// deals its workgroups to the eight XCDs in turn), so that the groups' work spreads over the
// XCDs; the first rank of each group would put every one of them on one XCD whenever g1 and
// wg0 are multiples of 8.  Which member it is does not change any value.
__host__ __device__ __forceinline__ int32_t group_leader(const Prob &P, int32_t g) {
  const int32_t q0 = g * P.g1, size = (P.nwg < q0 + P.g1 ? P.nwg : q0 + P.g1) - q0;
  const int32_t off = ((g & 7) - ((P.wg0 + q0) & 7) + 8) & 7;
  return q0 + (off < size ? off : 0);
}

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
  int32_t res_rows;        // row path: rows of X each workgroup keeps in LDS (the first of its slice)
  int32_t max_per_wg;      // row path: largest per_wg of the launch's problems (sizes the LDS)
  int32_t second_order;    // Gram path: 1 = the second index of each pair by the second-order rule
  uint64_t spin_limit;     // wall-clock ticks (100 MHz) a wait may last
  int32_t *error;          // set to 1 on a wait time-out
};

}  // namespace svmx

// gram.hip -- RBF Gram precompute on MFMA, kernel rows from X, and row gathers (gfx950).
//
// G_ij = exp(-gamma * max(0, |x_i|^2 + |x_j|^2 - 2 x_i.x_j)): the dot products form the
// contraction X X^T, run on v_mfma_f32_16x16x4f32 with fp32 inputs and accumulation over the
// upper-triangle tiles only (G is symmetric); the row norms are accumulated from the same LDS
// tiles and the RBF map is the epilogue, whose stores are non-temporal (the Gram is not read
// again here, so its lines should not displace the operand slabs from L2).  The kernel is the
// Gaussian RBF the paper names (Section III.C).
#include "common.hpp"
#include "rbf_rows.hpp"
#include "tile_order.hpp"
#include "tile_store.hpp"

#include <math.h>

namespace svmx {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int GT = 128;       // tile edge (rows and columns)
constexpr int GKC = 16;       // k per LDS stage
constexpr int GPAD = GT + 16; // LDS row pitch in floats (keeps the MFMA operand reads conflict-free)
constexpr int GBS = 256;      // 4 waves, 2x2 over the tile, 64x64 each

// Load a 128 x 16 slab of X (rows r0.., columns k0..) into LDS transposed to [k][row], and
// add the slab's squares into this thread's norm partials.  Thread t covers rows t/4 and
// 64 + t/4, columns k0 + 4*(t%4) .. +3, so the partials of a row always meet in the same
// order and a sample's norm does not depend on which tile role loaded it.
template <bool VEC4>
__device__ __forceinline__ void load_slab(const float *__restrict__ X, int64_t n, int64_t d, int64_t r0, int64_t k0,
                                          float (*S)[GPAD], float nacc[2]) {
  const int t = threadIdx.x;
  const int kq = (t & 3) * 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int row = h * 64 + (t >> 2);
    const int64_t gr = r0 + row;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (gr < n) {
      const float *src = X + gr * d + k0 + kq;
      if (VEC4 && k0 + kq + 3 < d) {
        const float4 q = *reinterpret_cast<const float4 *>(src);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (k0 + kq + e < d) v[e] = src[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      S[kq + e][row] = v[e];
      nacc[h] += v[e] * v[e];
    }
  }
}

// One 128x128 tile (rows i0.., columns j0..) of the Gram for each tile with ti <= tj (the
// upper triangle); a tile off the diagonal is stored twice, as itself and mirrored.  Tiles are
// handed out XCD-major in super-tile order (tile_order.hpp): the workgroups one XCD holds at
// once share their row and column slabs in that XCD's L2.  The RBF map is exp2(c * t) with
// c = -gamma * log2(e) and t = |x_i|^2 + |x_j|^2 - 2 x_i.x_j clamped at 0 (v_exp_f32).
template <bool VEC4, bool STORE4>
__global__ void __launch_bounds__(GBS) gram_rbf_mfma(const float *__restrict__ X, int64_t n, int64_t d, float c,
                                                     float *__restrict__ G, int64_t ld, int64_t nt, int64_t ntiles) {
  __shared__ float As[GKC][GPAD];
  __shared__ float Bs[GKC][GPAD];
  __shared__ float nA[GT], nB[GT];
  // XCD-major swizzle of the linear tile index, then (ti, tj) in super-tile order
  const int64_t per_xcd = (ntiles + 7) / 8;
  const int64_t b = (int64_t)blockIdx.x;
  const int64_t lin = (b % 8) * per_xcd + b / 8;
  if (lin >= ntiles) return;
  int64_t ti, tj;
  upper_tile_super(lin, nt, ti, tj);
  const int64_t i0 = ti * GT, j0 = tj * GT;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  v4f acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) acc[a][bb] = (v4f){0.f, 0.f, 0.f, 0.f};
  float na[2] = {0.f, 0.f}, nb[2] = {0.f, 0.f};

  for (int64_t k0 = 0; k0 < d; k0 += GKC) {
    load_slab<VEC4>(X, n, d, i0, k0, As, na);
    load_slab<VEC4>(X, n, d, j0, k0, Bs, nb);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GKC; kk += 4) {
      float av[4], bv[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) av[m] = As[kk + (lane >> 4)][wm * 64 + m * 16 + (lane & 15)];
#pragma unroll
      for (int m = 0; m < 4; ++m) bv[m] = Bs[kk + (lane >> 4)][wn * 64 + m * 16 + (lane & 15)];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int bb = 0; bb < 4; ++bb)
          acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[bb], acc[a][bb], 0, 0, 0);
    }
    __syncthreads();
  }
  // norms: combine the four partials of each row (lanes 4r..4r+3 of a wave)
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    na[h] += __shfl_xor(na[h], 1);
    na[h] += __shfl_xor(na[h], 2);
    nb[h] += __shfl_xor(nb[h], 1);
    nb[h] += __shfl_xor(nb[h], 2);
  }
  if ((threadIdx.x & 3) == 0) {
    nA[threadIdx.x >> 2] = na[0];
    nA[64 + (threadIdx.x >> 2)] = na[1];
    nB[threadIdx.x >> 2] = nb[0];
    nB[64 + (threadIdx.x >> 2)] = nb[1];
  }
  __syncthreads();
  // epilogue: lane holds D[4*(lane/16)+e][lane%16] of each 16x16 block
  const bool mirror = ti != tj;
  const int kq = lane >> 4, r16 = lane & 15;
  float kv[4][4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int lr0 = wm * 64 + a * 16 + 4 * kq;
    const int64_t gr0 = i0 + lr0;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const int lc = wn * 64 + bb * 16 + r16;
      const int64_t gc = j0 + lc;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float t = nA[lr0 + e] + nB[lc] - 2.0f * acc[a][bb][e];
        t = t > 0.f ? t : 0.f;
        kv[a][bb][e] = (gr0 + e == gc) ? 1.0f : __builtin_amdgcn_exp2f(c * t);
      }
      if (!mirror && gc < n) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (gr0 + e < n) __builtin_nontemporal_store(kv[a][bb][e], &G[(gr0 + e) * ld + gc]);
      }
    }
  }
  if (mirror) store_tile_128<STORE4>(G, ld, n, i0 + wm * 64, j0 + wn * 64, kq, r16, kv);
}

hipError_t launch_gram(const float *X, int64_t n, int64_t d, float gamma, float *G, int64_t ld, hipStream_t s) {
  const int64_t nt = (n + GT - 1) / GT;
  const int64_t ntiles = nt * (nt + 1) / 2;
  const int64_t grid = ((ntiles + 7) / 8) * 8;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  const float c = -gamma * 1.4426950408889634f;
  const bool vec4 = (d % 4 == 0) && ((reinterpret_cast<uintptr_t>(X) & 15) == 0);
  const bool st4 = (ld % 4 == 0) && ((reinterpret_cast<uintptr_t>(G) & 15) == 0);
  if (vec4 && st4)
    hipLaunchKernelGGL((gram_rbf_mfma<true, true>), dim3((unsigned)grid), dim3(GBS), 0, s, X, n, d, c, G, ld, nt, ntiles);
  else if (vec4)
    hipLaunchKernelGGL((gram_rbf_mfma<true, false>), dim3((unsigned)grid), dim3(GBS), 0, s, X, n, d, c, G, ld, nt, ntiles);
  else if (st4)
    hipLaunchKernelGGL((gram_rbf_mfma<false, true>), dim3((unsigned)grid), dim3(GBS), 0, s, X, n, d, c, G, ld, nt, ntiles);
  else
    hipLaunchKernelGGL((gram_rbf_mfma<false, false>), dim3((unsigned)grid), dim3(GBS), 0, s, X, n, d, c, G, ld, nt, ntiles);
  return hipGetLastError();
}

// out[q][j] = K(x_rows[q], x_j), evaluated with the row path's routines (pairs of rows, the
// sample norms computed here with the routine that fills the solver's norm table).
template <bool VEC4>
__global__ void __launch_bounds__(256) kernel_rows_k(const float *__restrict__ X, int64_t n, int64_t d, double gamma,
                                                      const int64_t *__restrict__ rows, int64_t r,
                                                      float *__restrict__ out) {
  constexpr int SB = 2, MAXM = ROW_POSITIONS;
  const int64_t q0 = 2 * (int64_t)blockIdx.y;
  const int64_t q1 = q0 + 1 < r ? q0 + 1 : q0;
  const int64_t ru = rows[q0], rl = rows[q1];
  const float *xu = X + ru * d, *xl = X + rl * d;
  const int gs = group_size_for(d, VEC4);
  const int lig = threadIdx.x & (gs - 1);
  const int ngroups = 256 / gs;
  const int grp = threadIdx.x / gs;
  const double nu = sq_norm<VEC4>(xu, d, lig, gs), nl = sq_norm<VEC4>(xl, d, lig, gs);
  RowPair<VEC4, MAXM> rp;
  load_pair(rp, xu, xl, d, lig, gs);
  const int64_t chunk = (int64_t)ngroups * SB;
  for (int64_t j0 = (int64_t)blockIdx.x * chunk + (int64_t)grp * SB; j0 < n; j0 += (int64_t)gridDim.x * chunk) {
    const int nb = (int)(n - j0 < SB ? n - j0 : SB);
    const float *xs[SB];
    double nj[SB];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
      xs[b] = X + (j0 + (b < nb ? b : nb - 1)) * d;
      nj[b] = sq_norm<VEC4>(xs[b], d, lig, gs);
    }
    double du[SB], dl[SB];
    dot_batch<VEC4, SB, MAXM>(xs, nb, xu, xl, d, lig, gs, rp, du, dl);
    for (int v = lig; v < 2 * SB; v += gs) {
      const int b = v < SB ? v : v - SB;
      if (b >= nb) continue;
      const float kv = rbf_from_dot(v < SB ? nu : nl, nj[b], batch_value<SB>(du, dl, v), gamma);
      if (v < SB)
        out[q0 * n + j0 + b] = kv;
      else if (q1 != q0)
        out[q1 * n + j0 + b] = kv;
    }
  }
}

// flag[0] = 1 if any of the count values at X is not finite (a plain store: every writer
// stores the same value, so no atomic is needed).
__global__ void __launch_bounds__(256) nonfinite_k(const float *__restrict__ X, int64_t count, int32_t *flag) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += stride) bad |= !__builtin_isfinite(X[i]);
  if (bad) *flag = 1;
}

hipError_t launch_check_finite(const float *X, int64_t count, int32_t *flag, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(nonfinite_k, dim3((unsigned)blocks), dim3(256), 0, s, X, count, flag);
  return hipGetLastError();
}

// sqn[j] = |x_j|^2, one group of lanes per row (the routine kernel_rows_k uses).
template <bool VEC4>
__global__ void __launch_bounds__(256) row_norms_k(const float *__restrict__ X, int64_t n, int64_t d,
                                                    double *__restrict__ sqn) {
  const int gs = group_size_for(d, VEC4);
  const int lig = threadIdx.x & (gs - 1);
  const int64_t groups = (int64_t)gridDim.x * (256 / gs);
  for (int64_t j = (int64_t)blockIdx.x * (256 / gs) + threadIdx.x / gs; j < n; j += groups) {
    const double v = sq_norm<VEC4>(X + j * d, d, lig, gs);
    if (lig == 0) sqn[j] = v;
  }
}

hipError_t launch_row_norms(const float *X, int64_t n, int64_t d, double *sqn, hipStream_t s) {
  const bool vec4 = (d % 4 == 0) && ((reinterpret_cast<uintptr_t>(X) & 15) == 0);
  int64_t blocks = (n + 3) / 4;  // at least four rows per block (64-lane groups); grid-stride beyond
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  if (vec4)
    hipLaunchKernelGGL(row_norms_k<true>, dim3((unsigned)blocks), dim3(256), 0, s, X, n, d, sqn);
  else
    hipLaunchKernelGGL(row_norms_k<false>, dim3((unsigned)blocks), dim3(256), 0, s, X, n, d, sqn);
  return hipGetLastError();
}

hipError_t launch_kernel_rows(const float *X, int64_t n, int64_t d, double gamma, const int64_t *rows, int64_t r,
                              float *out, hipStream_t s) {
  const int64_t pairs = (r + 1) / 2;
  if (pairs > 65535) return hipErrorInvalidValue;
  int64_t bx = (n + 255) / 256;
  if (bx > 1024) bx = 1024;
  const bool vec4 = (d % 4 == 0) && ((reinterpret_cast<uintptr_t>(X) & 15) == 0);
  if (vec4)
    hipLaunchKernelGGL(kernel_rows_k<true>, dim3((unsigned)bx, (unsigned)pairs), dim3(256), 0, s, X, n, d, gamma,
                       rows, r, out);
  else
    hipLaunchKernelGGL(kernel_rows_k<false>, dim3((unsigned)bx, (unsigned)pairs), dim3(256), 0, s, X, n, d, gamma,
                       rows, r, out);
  return hipGetLastError();
}

// Xs[r] = X[perm[r]] (row gather, e.g. into class-sorted order).
__global__ void gather_rows_k(const float *__restrict__ X, int64_t d, const int32_t *__restrict__ perm, int64_t n,
                              float *__restrict__ Xs) {
  const int64_t total = n * d;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / d, k = e - r * d;
    Xs[e] = X[(int64_t)perm[r] * d + k];
  }
}

hipError_t launch_gather_rows(const float *X, int64_t d, const int32_t *perm, int64_t n, float *Xs, hipStream_t s) {
  int64_t blocks = (n * d + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(gather_rows_k, dim3((unsigned)blocks), dim3(256), 0, s, X, d, perm, n, Xs);
  return hipGetLastError();
}

}  // namespace svmx

// gram_split.hip -- RBF Gram on the fp16 MFMA path with fp32 accuracy (gfx950).
//
// G_ij = exp(-gamma * max(0, |x_i|^2 + |x_j|^2 - 2 x_i.x_j)) as in gram.hip (the Gaussian RBF
// the paper names, Section III.C), but the contraction X X^T runs on v_mfma_f32_16x16x32_f16:
// every row is scaled by a power of two s_i (so that |x| < 1), split as x = h + l with h, l fp16
// (h the nearest fp16, l the nearest fp16 to the remainder; together 22 significant bits), and
// x_i.x_j = s_i s_j (h_i.h_j + h_i.l_j + l_i.h_j) up to the l_i.l_j term (2^-22 relative) and
// the rounding of l; all three products go into one fp32 accumulator per output, as in an fp32
// contraction.  Three fp16 MFMA products per fp32 product on a 2.5 PFLOP/s path instead of one
// fp32 product on the 157 TFLOP/s path; measured against the fp64 difference form, the values
// are as accurate as those of the fp32 MFMA kernel.  The row norms are fp64 sums of the fp32
// inputs.
#include "common.hpp"
#include "tile_order.hpp"
#include "tile_store.hpp"

#include <math.h>

namespace svmx {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int ST = 128;   // tile edge (rows and columns)
constexpr int SKS = 32;   // k per stage: one MFMA K
constexpr int SBS = 256;  // 4 waves, 2x2 over the tile, 64x64 each

int64_t split_pitch(int64_t d) { return (d + SKS - 1) / SKS * SKS; }

// Scratch of the split Gram: hi and lo halves [n][dp] (dp = d rounded up to 32, zero padded),
// the power-of-two row scales and the row norms.
int64_t gram_split_scratch_bytes(int64_t n, int64_t d) {
  const int64_t dp = split_pitch(d);
  return 2 * (2 * n * dp) + 8 * n + 256;
}

SplitX split_views(void *scratch, int64_t n, int64_t d) {
  SplitX s;
  s.dp = split_pitch(d);
  char *p = static_cast<char *>(scratch);
  s.hi = reinterpret_cast<_Float16 *>(p);
  s.lo = s.hi + n * s.dp;
  s.scale = reinterpret_cast<float *>(s.lo + n * s.dp);
  s.nrm = s.scale + n;
  return s;
}

// One wave per row: s = 2^e with max|x| < 2^e, h = fp16(x / s), l = fp16(x / s - h), and the
// norm |x|^2 as an fp64 sum rounded to fp32.
__global__ void __launch_bounds__(256) gram_split_k(const float *__restrict__ X, int64_t n, int64_t d, SplitX s) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * 4;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += waves) {
    const float *x = X + r * d;
    float m = 0.f;
    double q = 0.0;
    for (int64_t k = lane; k < d; k += 64) {
      const float v = x[k];
      m = fmaxf(m, fabsf(v));
      q = __builtin_fma((double)v, (double)v, q);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      m = fmaxf(m, __shfl_xor(m, o));
      q += __shfl_xor(q, o);
    }
    int e = 0;
    if (m > 0.f) (void)frexpf(m, &e);  // m = f 2^e, f in [0.5, 1)
    const float inv = ldexpf(1.0f, -e);
    _Float16 *hr = s.hi + r * s.dp, *lr = s.lo + r * s.dp;
    for (int64_t k = lane; k < s.dp; k += 64) {
      const float v = k < d ? x[k] * inv : 0.f;  // exact (power of two)
      const _Float16 h = (_Float16)v;
      hr[k] = h;
      lr[k] = (_Float16)(v - (float)h);  // v - h is exact in fp32
    }
    if (lane == 0) {
      s.scale[r] = ldexpf(1.0f, e);
      s.nrm[r] = (float)q;
    }
  }
}

// LDS stage: [slab: A hi, A lo, B hi, B lo][k chunk of 8][row] of 16-byte vectors, so the 16
// lanes that read one MFMA operand read 256 contiguous bytes.
struct SplitStage {
  h8 v[4][SKS / 8][ST];
};

// This thread's share of one stage: rows t/2 of the A and B tiles, k chunks 2*(t%2), +1.
__device__ __forceinline__ void split_load(const SplitX &s, int64_t n, int64_t i0, int64_t j0, int64_t k0, h8 (&r)[8]) {
  const int t = threadIdx.x;
  const int row = t >> 1, kq = (t & 1) * 2;
#pragma unroll
  for (int sl = 0; sl < 4; ++sl) {
    const int64_t g = (sl < 2 ? i0 : j0) + row;
    const _Float16 *base = (sl & 1) ? s.lo : s.hi;
    if (g < n) {
      const h8 *p = reinterpret_cast<const h8 *>(base + g * s.dp + k0) + kq;
      r[2 * sl] = p[0];
      r[2 * sl + 1] = p[1];
    } else {
      r[2 * sl] = (h8){};
      r[2 * sl + 1] = (h8){};
    }
  }
}

__device__ __forceinline__ void split_store(SplitStage &S, const h8 (&r)[8]) {
  const int t = threadIdx.x;
  const int row = t >> 1, kq = (t & 1) * 2;
#pragma unroll
  for (int sl = 0; sl < 4; ++sl) {
    S.v[sl][kq][row] = r[2 * sl];
    S.v[sl][kq + 1][row] = r[2 * sl + 1];
  }
}

// One 128x128 tile of the upper triangle per workgroup; workgroup b runs on XCD b % 8 and takes
// tile b / 8 of that XCD's contiguous share of the super-tile order (tile_order.hpp), so the
// tiles an XCD holds at once share their row and column slabs in its L2.  An off-diagonal
// tile is stored twice, as itself and mirrored.  The stores are non-temporal: the Gram is not
// read again by this kernel, so its lines should not displace the operand slabs from L2
// (measured: 12.0 -> 9.8 ms for the 60,000 x 784 Gram, 1.35 -> 1.16 ms at 20,000 x 784,
// 3.67 -> 3.30 ms at 50,000 x 128, 12.6 -> 12.2 ms at 100,000 x 32).  Lane l of an MFMA holds
// D[4*(l/16) + e][l%16] of each 16x16 block.
template <bool STORE4>
__global__ void __launch_bounds__(SBS) gram_rbf_f16x3(SplitX s, int64_t n, float c, float *__restrict__ G, int64_t ld,
                                                      int64_t nt, int64_t ntiles) {
  __shared__ SplitStage S[2];
  __shared__ float sA[ST], sB[ST], nA[ST], nB[ST];
  const int64_t per_xcd = (ntiles + 7) / 8;
  const int64_t b = (int64_t)blockIdx.x;
  const int64_t lin = (b % 8) * per_xcd + b / 8;
  if (lin >= ntiles) return;
  int64_t ti, tj;
  upper_tile_super(lin, nt, ti, tj);
  const int64_t i0 = ti * ST, j0 = tj * ST;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int kq = lane >> 4, r16 = lane & 15;

  if (threadIdx.x < ST) {
    const int64_t gi = i0 + threadIdx.x, gj = j0 + threadIdx.x;
    sA[threadIdx.x] = gi < n ? s.scale[gi] : 0.f;
    nA[threadIdx.x] = gi < n ? s.nrm[gi] : 0.f;
    sB[threadIdx.x] = gj < n ? s.scale[gj] : 0.f;
    nB[threadIdx.x] = gj < n ? s.nrm[gj] : 0.f;
  }
  v4f acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) acc[a][bb] = (v4f){0.f, 0.f, 0.f, 0.f};
  h8 r[8];
  split_load(s, n, i0, j0, 0, r);
  split_store(S[0], r);
  __syncthreads();
  const int64_t stages = s.dp / SKS;
  for (int64_t st = 0; st < stages; ++st) {
    const int cur = (int)(st & 1);
    if (st + 1 < stages) split_load(s, n, i0, j0, (st + 1) * SKS, r);
    h8 ah[4], al[4], bh[4], bl[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      ah[a] = S[cur].v[0][kq][wm * 64 + a * 16 + r16];
      al[a] = S[cur].v[1][kq][wm * 64 + a * 16 + r16];
      bh[a] = S[cur].v[2][kq][wn * 64 + a * 16 + r16];
      bl[a] = S[cur].v[3][kq][wn * 64 + a * 16 + r16];
    }
    // the three products of a block go into one accumulator; each sweep over the 16 blocks
    // keeps 16 independent MFMAs between two uses of an accumulator
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bh[bb], acc[a][bb], 0, 0, 0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bl[bb], acc[a][bb], 0, 0, 0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[a], bh[bb], acc[a][bb], 0, 0, 0);
    if (st + 1 < stages) split_store(S[cur ^ 1], r);
    __syncthreads();
  }

  const bool diag = ti == tj;
  // A diagonal tile holds both K(x_r, x_c) and K(x_c, x_r).  The cross products h.l and l.h
  // are accumulated in the order of the operand roles, so the two can differ in the last bit;
  // the upper one (row index <= column index, the role every off-diagonal tile uses) is
  // mirrored into the lower one through LDS (the stage buffers, free after the loop), so that
  // K(x_i, x_j) of i < j is always computed with x_i as the row operand.
  float(*T)[ST] = reinterpret_cast<float(*)[ST]>(&S[0]);
  static_assert(sizeof(S) >= sizeof(float) * ST * ST, "mirror tile does not fit the stage buffers");
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
      for (int e = 0; e < 4; ++e)
        kv[a][bb][e] = (gr0 + e == gc) ? 1.0f : split_rbf(acc[a][bb][e], sA[lr0 + e], sB[lc], nA[lr0 + e], nB[lc], c);
      if (diag) {
#pragma unroll
        for (int e = 0; e < 4; ++e) T[lr0 + e][lc] = kv[a][bb][e];
      }
    }
  }
  if (!diag) {
    store_tile_128<STORE4>(G, ld, n, i0 + wm * 64, j0 + wn * 64, kq, r16, kv);
    return;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < ST * ST; q += SBS) {
    const int r = q / ST, cc = q % ST;
    const int64_t gr = i0 + r, gcc = j0 + cc;
    if (gr < n && gcc < n) __builtin_nontemporal_store(r <= cc ? T[r][cc] : T[cc][r], &G[gr * ld + gcc]);
  }
}

// One LDS stage (32 KB, loaded, then multiplied, no register prefetch) instead of two, so four
// workgroups share a CU instead of two; a diagonal tile writes each upper value to both of its
// places instead of mirroring through LDS.  Same products in the same order, so the same
// values.  Short rows are bound by the stores, and four workgroups a CU keep twice as many in
// flight: 13.9 -> 11.3-11.7 ms at 100,000 x 32 (40 GB), 3.5 -> 3.3 ms at 50,000 x 128.  Long
// rows are bound by the stage loads and the MFMA schedule, and there the other workgroups'
// products cover each one's loads better than one stage of register prefetch in two:
// 1.34 -> 1.12 ms at 20,000 x 784, 10.95 -> 9.73 ms at 60,000 x 784, 0.66 -> 0.53 ms at
// 20,000 x 256.  The two-stage kernel remains for a Gram whose row pitch or base does not
// allow float4 stores.
__global__ void __launch_bounds__(SBS, 4) gram_rbf_f16x3_lds1(SplitX s, int64_t n, float c, float *__restrict__ G,
                                                             int64_t ld, int64_t nt, int64_t ntiles, int64_t sup) {
  __shared__ SplitStage S[1];
  __shared__ float sA[ST], sB[ST], nA[ST], nB[ST];
  const int64_t per_xcd = (ntiles + 7) / 8;
  const int64_t b = (int64_t)blockIdx.x;
  const int64_t lin = (b % 8) * per_xcd + b / 8;
  if (lin >= ntiles) return;
  int64_t ti, tj;
  upper_tile_super(lin, nt, ti, tj, sup);
  const int64_t i0 = ti * ST, j0 = tj * ST;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int kq = lane >> 4, r16 = lane & 15;
  if (threadIdx.x < ST) {
    const int64_t gi = i0 + threadIdx.x, gj = j0 + threadIdx.x;
    sA[threadIdx.x] = gi < n ? s.scale[gi] : 0.f;
    nA[threadIdx.x] = gi < n ? s.nrm[gi] : 0.f;
    sB[threadIdx.x] = gj < n ? s.scale[gj] : 0.f;
    nB[threadIdx.x] = gj < n ? s.nrm[gj] : 0.f;
  }
  v4f acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) acc[a][bb] = (v4f){0.f, 0.f, 0.f, 0.f};
  const int64_t stages = s.dp / SKS;
  for (int64_t stg = 0; stg < stages; ++stg) {
    {
      h8 r[8];
      split_load(s, n, i0, j0, stg * SKS, r);
      if (stg > 0) __syncthreads();  // the previous stage's operands have been read
      split_store(S[0], r);
    }
    __syncthreads();
    h8 ah[4], al[4], bh[4], bl[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      ah[a] = S[0].v[0][kq][wm * 64 + a * 16 + r16];
      al[a] = S[0].v[1][kq][wm * 64 + a * 16 + r16];
      bh[a] = S[0].v[2][kq][wn * 64 + a * 16 + r16];
      bl[a] = S[0].v[3][kq][wn * 64 + a * 16 + r16];
    }
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bh[bb], acc[a][bb], 0, 0, 0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bl[bb], acc[a][bb], 0, 0, 0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) acc[a][bb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[a], bh[bb], acc[a][bb], 0, 0, 0);
  }
  const bool diag = ti == tj;
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
      for (int e = 0; e < 4; ++e)
        kv[a][bb][e] = (gr0 + e == gc) ? 1.0f : split_rbf(acc[a][bb][e], sA[lr0 + e], sB[lc], nA[lr0 + e], nB[lc], c);
      if (diag && gc < n) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (gr0 + e < n && lr0 + e <= lc) {
            __builtin_nontemporal_store(kv[a][bb][e], &G[(gr0 + e) * ld + gc]);
            if (lr0 + e < lc) __builtin_nontemporal_store(kv[a][bb][e], &G[gc * ld + gr0 + e]);
          }
        }
      }
    }
  }
  if (!diag) store_tile_128<true>(G, ld, n, i0 + wm * 64, j0 + wn * 64, kq, r16, kv);
}

hipError_t launch_split_rows(const float *X, int64_t n, int64_t d, const SplitX &s, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t pb = (n + 3) / 4;
  if (pb > 8192) pb = 8192;
  hipLaunchKernelGGL(gram_split_k, dim3((unsigned)pb), dim3(256), 0, st, X, n, d, s);
  return hipGetLastError();
}

hipError_t launch_gram_split(const float *X, int64_t n, int64_t d, float gamma, float *G, int64_t ld, void *scratch,
                             hipStream_t st) {
  const SplitX s = split_views(scratch, n, d);
  hipError_t e = launch_split_rows(X, n, d, s, st);
  if (e != hipSuccess) return e;
  const int64_t nt = (n + ST - 1) / ST;
  const int64_t ntiles = nt * (nt + 1) / 2;
  const int64_t grid = ((ntiles + 7) / 8) * 8;
  if (grid > 0x7fffffffLL) return hipErrorInvalidValue;
  const float c = -gamma * 1.4426950408889634f;
  const bool st4 = (ld % 4 == 0) && ((reinterpret_cast<uintptr_t>(G) & 15) == 0);
  if (st4) {
    // super-tiles of 32 x 32 tiles for rows of up to 128 features, whose build is bound by its
    // stores (measured: 8.7 -> 7.7 ms at 100,000 x 32, 16.6 -> 13.2 ms at 130,000 x 32, 2.44 ->
    // 2.37 ms at 50,000 x 128), 8 x 8 for longer rows (1.09 against 1.25 ms at 20,000 x 784)
    const int64_t sup = s.dp <= 4 * SKS ? 32 : 8;
    hipLaunchKernelGGL(gram_rbf_f16x3_lds1, dim3((unsigned)grid), dim3(SBS), 0, st, s, n, c, G, ld, nt, ntiles, sup);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((gram_rbf_f16x3<false>), dim3((unsigned)grid), dim3(SBS), 0, st, s, n, c, G, ld, nt, ntiles);
  return hipGetLastError();
}

}  // namespace svmx

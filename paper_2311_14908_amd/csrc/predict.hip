// predict.hip -- decision values d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b and one-vs-one votes.
//
// 1. sv_compact: the support vectors (a_i > 0) in increasing local index, as rows of X with
//    coefficient a_i y_i (one workgroup, ballot prefix sums; deterministic order).
// 2. predict_mfma: 128 test samples x 128 support vectors per tile; the dot products run on
//    v_mfma_f32_16x16x4f32 (fp32 in, fp32 accumulate), norms come from the same LDS slabs,
//    K = exp2(c * max(0, |t|^2 + |x|^2 - 2 t.x)) with c = -gamma log2(e), and each test row
//    sums coef * K in fp64 over the tile in a fixed tree.  Support-vector tiles are split
//    over `nsplit` workgroups per test tile; each split writes its own partial sums.
//    By default the contraction runs instead on v_mfma_f32_16x16x32_f16 with the rows scaled by
//    powers of two and split into two fp16 halves, three products per fp32 product, as in the
//    Gram build (predict_f16x3); `gram_mfma = SVM_MFMA_F32` keeps the fp32 kernel.
// 3. predict_final: dec = sum over splits (fixed order) - b.
// Results are deterministic: no atomics touch values.
#include "common.hpp"

#include <math.h>

namespace svmx {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int PT = 128;        // tile edge
constexpr int PKC = 16;        // k per LDS stage
constexpr int PPAD = PT + 16;  // LDS pitch (conflict-free operand reads)
constexpr int PBS = 256;

__device__ __forceinline__ int64_t pm_pos(const PredPair &m, int64_t j) {
  return j < m.len0 ? m.off0 + j : m.off1 + (j - m.len0);
}

// One workgroup of 1024 threads per problem (blockIdx.x): stable compaction of its samples
// with a > 0.
__global__ void __launch_bounds__(1024) sv_compact_k(const double *__restrict__ alpha_all,
                                                     const PredPair *__restrict__ pairs, int32_t *__restrict__ sv_row_all,
                                                     double *__restrict__ sv_coef_all, int64_t *__restrict__ count_all) {
  const PredPair map = pairs[blockIdx.x];
  const double *alpha = alpha_all + map.alpha_off;
  const int64_t n = map.ntr;
  int32_t *sv_row = sv_row_all + map.sv_off;
  double *sv_coef = sv_coef_all + map.sv_off;
  int64_t *count = count_all + blockIdx.x;
  __shared__ int wave_cnt[16];
  __shared__ int64_t s_base;
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int64_t c0 = 0; c0 < n; c0 += 1024) {
    const int64_t j = c0 + threadIdx.x;
    const double a = j < n ? alpha[j] : 0.0;
    const bool sv = a > 0.0;
    const unsigned long long mask = __ballot(sv);
    const int before = __popcll(mask & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[w] = __popcll(mask);
    __syncthreads();
    int off = 0;
    for (int q = 0; q < w; ++q) off += wave_cnt[q];
    int tot = 0;
    for (int q = 0; q < 16; ++q) tot += wave_cnt[q];
    if (sv) {
      const int64_t pos = pm_pos(map, j);
      const int64_t row = map.perm ? (int64_t)map.perm[pos] : pos;
      const double y = map.y ? (double)map.y[row] : (j < map.len0 ? 1.0 : -1.0);
      const int64_t dst = s_base + off + before;
      sv_row[dst] = (int32_t)row;
      sv_coef[dst] = a * y;
    }
    __syncthreads();
    if (threadIdx.x == 0) s_base += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) *count = s_base;
}

// Load 128 rows x 16 columns into LDS transposed to [k][row] and add the squares into the
// thread's norm partials (thread t: rows t/4 and 64 + t/4, columns 4*(t%4) .. +3).  Rows come
// from `idx` (row numbers of X) when given, else r0.. directly; rows at or past `nrows` are 0.
template <bool VEC4>
__device__ __forceinline__ void load_rows(const float *__restrict__ X, const int32_t *__restrict__ idx, int64_t nrows,
                                          int64_t d, int64_t r0, int64_t k0, float (*S)[PPAD], float nacc[2]) {
  const int t = threadIdx.x;
  const int kq = (t & 3) * 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int row = h * 64 + (t >> 2);
    const int64_t r = r0 + row;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < nrows) {
      const int64_t xr = idx ? (int64_t)idx[r] : r;
      const float *src = X + xr * d + k0 + kq;
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

template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int hi = __builtin_amdgcn_update_dpp((int)(b >> 32), (int)(b >> 32), CTRL, 0xf, 0xf, false);
  const int lo = __builtin_amdgcn_update_dpp((int)b, (int)b, CTRL, 0xf, 0xf, false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the same bits.
__device__ __forceinline__ double row16_sum(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  v += dpp_d<0x140>(v);  // row_mirror
  return v;
}

// Workgroup (x, y, z): test rows 128 x .. +128, split y of problem z's support-vector tiles.
template <bool VEC4>
__global__ void __launch_bounds__(PBS) predict_mfma_k(const float *__restrict__ T, int64_t m, const float *__restrict__ X,
                                                      const PredPair *__restrict__ pairs,
                                                      const int32_t *__restrict__ sv_row_all,
                                                      const double *__restrict__ sv_coef_all,
                                                      const int64_t *__restrict__ sv_count, int64_t d, float c,
                                                      double *__restrict__ part_all) {
  const PredPair pp = pairs[blockIdx.z];
  const int nsplit = pp.nsplit;
  if ((int)blockIdx.y >= nsplit) return;
  const int32_t *sv_row = sv_row_all + pp.sv_off;
  const double *sv_coef = sv_coef_all + pp.sv_off;
  double *part = part_all + pp.part_off;
  __shared__ float As[PKC][PPAD];
  __shared__ float Bs[PKC][PPAD];
  __shared__ float nA[PT], nB[PT];
  __shared__ double cB[PT];
  __shared__ double rs[2][PT];
  const int64_t nsv = sv_count[blockIdx.z];
  const int64_t q0 = (int64_t)blockIdx.x * PT;
  const int split = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  double row_acc = 0.0;  // thread t < 128 owns test row q0 + t
  const int64_t ntile = (nsv + PT - 1) / PT;
  for (int64_t st = split; st < ntile; st += nsplit) {
    const int64_t s0 = st * PT;
    v4f acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = (v4f){0.f, 0.f, 0.f, 0.f};
    float na[2] = {0.f, 0.f}, nb[2] = {0.f, 0.f};
    for (int64_t k0 = 0; k0 < d; k0 += PKC) {
      load_rows<VEC4>(T, nullptr, m, d, q0, k0, As, na);
      load_rows<VEC4>(X, sv_row + s0, nsv - s0, d, 0, k0, Bs, nb);
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < PKC; kk += 4) {
        float av[4], bv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) av[q] = As[kk + (lane >> 4)][wm * 64 + q * 16 + (lane & 15)];
#pragma unroll
        for (int q = 0; q < 4; ++q) bv[q] = Bs[kk + (lane >> 4)][wn * 64 + q * 16 + (lane & 15)];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[a], bv[b], acc[a][b], 0, 0, 0);
      }
      __syncthreads();
    }
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
    if (threadIdx.x < PT) cB[threadIdx.x] = s0 + threadIdx.x < nsv ? sv_coef[s0 + threadIdx.x] : 0.0;
    __syncthreads();
    // per test row: sum over this wave's 64 columns (4 blocks x 16 lanes), then the two halves
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int lr = wm * 64 + a * 16 + 4 * (lane >> 4) + e;
        double sacc = 0.0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int lc = wn * 64 + b * 16 + (lane & 15);
          float t = nA[lr] + nB[lc] - 2.0f * acc[a][b][e];
          t = t > 0.f ? t : 0.f;
          sacc = __builtin_fma(cB[lc], (double)__builtin_amdgcn_exp2f(c * t), sacc);
        }
        sacc = row16_sum(sacc);
        if ((lane & 15) == 0) rs[wn][lr] = sacc;
      }
    }
    __syncthreads();
    if (threadIdx.x < PT) row_acc += rs[0][threadIdx.x] + rs[1][threadIdx.x];
    __syncthreads();
  }
  if (threadIdx.x < PT && q0 + threadIdx.x < m) part[(int64_t)split * m + q0 + threadIdx.x] = row_acc;
}

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
constexpr int PKS = 32;  // k per stage of the split kernel (one MFMA K)

struct PredStage {
  h8 v[4][PKS / 8][PT];  // [A hi, A lo, B hi, B lo][k chunk of 8][row]
};

// This thread's share of one stage: rows t/2 of the test tile (A, rows q0..) and of the
// support-vector tile (B, rows sv_row[s0..]), k chunks 2*(t%2), +1.  Rows past the end are 0.
__device__ __forceinline__ void pred_split_load(const SplitX &st, const SplitX &sx, int64_t m, int64_t q0,
                                                const int32_t *__restrict__ sv_row, int64_t nsv, int64_t s0, int64_t k0,
                                                h8 (&r)[8]) {
  const int t = threadIdx.x;
  const int row = t >> 1, kq = (t & 1) * 2;
  const int64_t qa = q0 + row, qb = s0 + row;
  const bool va = qa < m, vb = qb < nsv;
  const int64_t rb = vb ? (int64_t)sv_row[qb] : 0;
#pragma unroll
  for (int sl = 0; sl < 4; ++sl) {
    const bool v = sl < 2 ? va : vb;
    const SplitX &S = sl < 2 ? st : sx;
    const int64_t g = sl < 2 ? qa : rb;
    const _Float16 *base = (sl & 1) ? S.lo : S.hi;
    if (v) {
      const h8 *p = reinterpret_cast<const h8 *>(base + g * S.dp + k0) + kq;
      r[2 * sl] = p[0];
      r[2 * sl + 1] = p[1];
    } else {
      r[2 * sl] = (h8){};
      r[2 * sl + 1] = (h8){};
    }
  }
}

__device__ __forceinline__ void pred_split_store(PredStage &S, const h8 (&r)[8]) {
  const int t = threadIdx.x;
  const int row = t >> 1, kq = (t & 1) * 2;
#pragma unroll
  for (int sl = 0; sl < 4; ++sl) {
    S.v[sl][kq][row] = r[2 * sl];
    S.v[sl][kq + 1][row] = r[2 * sl + 1];
  }
}

// predict_mfma_k on the split representation: st holds the test rows, sx the training rows
// (support vectors addressed through sv_row); dot = acc * s_q * s_j.  One LDS stage (loaded,
// then multiplied) instead of two with register prefetch, so three workgroups share a CU
// instead of two and each one's stage loads run under the others' products; same products in
// the same order, so the same values.  Measured at 10,000 test rows: 1.41 -> 1.38 ms with
// 15,016 support vectors of 784 features, 0.55 -> 0.44 ms with 20,000 of 128, 0.36 -> 0.32 ms
// with 13,500 of 32.
__global__ void __launch_bounds__(PBS, 3) predict_f16x3_k(SplitX st, int64_t m, SplitX sx,
                                                       const PredPair *__restrict__ pairs,
                                                       const int32_t *__restrict__ sv_row_all,
                                                       const double *__restrict__ sv_coef_all,
                                                       const int64_t *__restrict__ sv_count, float c,
                                                       double *__restrict__ part_all) {
  const PredPair pp = pairs[blockIdx.z];
  const int nsplit = pp.nsplit;
  if ((int)blockIdx.y >= nsplit) return;
  const int32_t *sv_row = sv_row_all + pp.sv_off;
  const double *sv_coef = sv_coef_all + pp.sv_off;
  double *part = part_all + pp.part_off;
  __shared__ PredStage S[1];
  __shared__ float sA[PT], nA[PT], sB[PT], nB[PT];
  __shared__ double cB[PT];
  __shared__ double rs[2][PT];
  const int64_t nsv = sv_count[blockIdx.z];
  const int64_t q0 = (int64_t)blockIdx.x * PT;
  const int split = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int kq = lane >> 4, r16 = lane & 15;
  if (threadIdx.x < PT) {
    const int64_t q = q0 + threadIdx.x;
    sA[threadIdx.x] = q < m ? st.scale[q] : 0.f;
    nA[threadIdx.x] = q < m ? st.nrm[q] : 0.f;
  }
  double row_acc = 0.0;  // thread t < 128 owns test row q0 + t
  const int64_t ntile = (nsv + PT - 1) / PT;
  const int64_t stages = st.dp / PKS;
  for (int64_t tile = split; tile < ntile; tile += nsplit) {
    const int64_t s0 = tile * PT;
    if (threadIdx.x < PT) {
      const int64_t q = s0 + threadIdx.x;
      const int64_t rr = q < nsv ? (int64_t)sv_row[q] : -1;
      sB[threadIdx.x] = rr >= 0 ? sx.scale[rr] : 0.f;
      nB[threadIdx.x] = rr >= 0 ? sx.nrm[rr] : 0.f;
      cB[threadIdx.x] = rr >= 0 ? sv_coef[q] : 0.0;
    }
    v4f acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = (v4f){0.f, 0.f, 0.f, 0.f};
    for (int64_t sg = 0; sg < stages; ++sg) {
      {
        h8 r[8];
        pred_split_load(st, sx, m, q0, sv_row, nsv, s0, sg * PKS, r);
        if (sg > 0) __syncthreads();  // the previous stage's operands have been read
        pred_split_store(S[0], r);
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
        for (int b = 0; b < 4; ++b) {
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bh[b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bl[b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[a], bh[b], acc[a][b], 0, 0, 0);
        }
    }
    // per test row: sum over this wave's 64 columns (4 blocks x 16 lanes), then the two halves
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int lr = wm * 64 + a * 16 + 4 * kq + e;
        double sacc = 0.0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int lc = wn * 64 + b * 16 + r16;
          const float dot = (acc[a][b][e] * sA[lr]) * sB[lc];
          float t = nA[lr] + nB[lc] - 2.0f * dot;
          t = t > 0.f ? t : 0.f;
          sacc = __builtin_fma(cB[lc], (double)__builtin_amdgcn_exp2f(c * t), sacc);
        }
        sacc = row16_sum(sacc);
        if (r16 == 0) rs[wn][lr] = sacc;
      }
    }
    __syncthreads();
    if (threadIdx.x < PT) row_acc += rs[0][threadIdx.x] + rs[1][threadIdx.x];
    __syncthreads();
  }
  if (threadIdx.x < PT && q0 + threadIdx.x < m) part[(int64_t)split * m + q0 + threadIdx.x] = row_acc;
}

// dec[q * stride + p] = the sum of problem p's (blockIdx.y) split partials - its bias.
__global__ void predict_final_k(const double *__restrict__ part_all, int64_t m, const PredPair *__restrict__ pairs,
                                double *dec, int64_t stride) {
  const int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (q >= m) return;
  const PredPair pp = pairs[blockIdx.y];
  const double *part = part_all + pp.part_off;
  double s = 0.0;
  for (int k = 0; k < pp.nsplit; ++k) s += part[(int64_t)k * m + q];
  dec[q * stride + blockIdx.y] = s - pp.b;
}

int predict_splits(int64_t m, int64_t nsv_max) {
  if (m <= 0) return 1;
  const int64_t row_tiles = (m + PT - 1) / PT;
  const int64_t sv_tiles = nsv_max > 0 ? (nsv_max + PT - 1) / PT : 1;
  int64_t s = (512 + row_tiles - 1) / row_tiles;
  if (s > sv_tiles) s = sv_tiles;
  if (s > 64) s = 64;
  if (s < 1) s = 1;
  return (int)s;
}

hipError_t launch_predict_pairs(const float *Xtr, int64_t d, int32_t npairs, int nsplit_max, const double *alpha,
                                double gamma, const float *T, int64_t m, double *dec, int64_t dec_stride,
                                const PredictScratch &ws, hipStream_t s) {
  if (m <= 0 || npairs <= 0) return hipSuccess;
  const bool split = ws.split_test != nullptr && ws.split_train != nullptr;
  hipLaunchKernelGGL(sv_compact_k, dim3((unsigned)npairs), dim3(1024), 0, s, alpha, ws.pairs, ws.sv_row, ws.sv_coef,
                     ws.count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float c = (float)(-gamma * 1.4426950408889634);
  dim3 grid((unsigned)((m + PT - 1) / PT), (unsigned)nsplit_max, (unsigned)npairs);
  const bool vec4 = (d % 4 == 0) && ((reinterpret_cast<uintptr_t>(T) & 15) == 0) &&
                    ((reinterpret_cast<uintptr_t>(Xtr) & 15) == 0);
  if (split)
    hipLaunchKernelGGL(predict_f16x3_k, grid, dim3(PBS), 0, s, *ws.split_test, m, *ws.split_train, ws.pairs,
                       ws.sv_row, ws.sv_coef, ws.count, c, ws.part);
  else if (vec4)
    hipLaunchKernelGGL(predict_mfma_k<true>, grid, dim3(PBS), 0, s, T, m, Xtr, ws.pairs, ws.sv_row, ws.sv_coef,
                       ws.count, d, c, ws.part);
  else
    hipLaunchKernelGGL(predict_mfma_k<false>, grid, dim3(PBS), 0, s, T, m, Xtr, ws.pairs, ws.sv_row, ws.sv_coef,
                       ws.count, d, c, ws.part);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(predict_final_k, dim3((unsigned)((m + 255) / 256), (unsigned)npairs), dim3(256), 0, s, ws.part,
                     m, ws.pairs, dec, dec_stride);
  return hipGetLastError();
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

// tile_store.hpp -- stores of a 128 x 128 Gram tile held in MFMA 16 x 16 output layout (four
// waves of 64 x 64), shared by the split-fp16 and the fp32 MFMA Gram kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace svmx {

typedef float tile_v4f __attribute__((ext_vector_type(4)));

// Value of lane (lane ^ 16) and of lane (lane ^ 1): the gfx950 lane swap across rows of 16,
// and the DPP quad permute [1, 0, 3, 2].
__device__ __forceinline__ float lane_xor16(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return __builtin_bit_cast(float, (threadIdx.x & 16) ? r[0] : r[1]);
}
__device__ __forceinline__ float lane_xor1(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, x),
                                                               __builtin_bit_cast(int, x), 0xB1, 0xF, 0xF, false));
}

// Stores of an off-diagonal tile and of its mirror in 128-byte row segments.  A wave holds a
// 64 x 64 block, lane (kq, r16) the values kv[a][bb][e] of row 16 a + 4 kq + e (from r0) and
// column 16 bb + r16 (from c0): the MFMA 16 x 16 layout, in which one store instruction would
// write 64-byte pieces of rows, and a stream of 64-byte pieces reaches about 3.3 TB/s against
// 5.5 TB/s for 128-byte ones (measured on 40 GB).  So the lanes trade values first.  Direct
// tile: lanes kq and kq ^ 1 (xor 16) swap one of two neighbouring 16-column blocks, after which
// lanes 0-31 (and 32-63) hold 32 consecutive columns of one row.  Mirror: lanes r16 and r16 ^ 1
// (xor 1) swap one of two neighbouring 16-row blocks, after which eight lanes hold 32
// consecutive entries of one mirrored row as float4s.  The values stored are the same.
template <bool STORE4>
__device__ __forceinline__ void store_tile_128(float *__restrict__ G, int64_t ld, int64_t n, int64_t r0, int64_t c0,
                                               int kq, int r16, const float (&kv)[4][4][4]) {
  const bool odd = kq & 1;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int jp = 0; jp < 2; ++jp)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float A = kv[a][2 * jp][e], B = kv[a][2 * jp + 1][e];
        const float recv = lane_xor16(odd ? A : B);
        const int64_t row1 = r0 + a * 16 + 4 * (kq & 2) + e, row2 = row1 + 4;
        const int64_t col = c0 + (2 * jp + (odd ? 1 : 0)) * 16 + r16;
        if (col < n) {
          if (row1 < n) __builtin_nontemporal_store(odd ? recv : A, &G[row1 * ld + col]);
          if (row2 < n) __builtin_nontemporal_store(odd ? B : recv, &G[row2 * ld + col]);
        }
      }
  const bool odd1 = r16 & 1;
#pragma unroll
  for (int ap = 0; ap < 2; ++ap)
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      float v1[4], v2[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float P = kv[2 * ap][bb][e], Q = kv[2 * ap + 1][bb][e];
        const float recv = lane_xor1(odd1 ? P : Q);
        v1[e] = odd1 ? recv : P;
        v2[e] = odd1 ? Q : recv;
      }
      const int64_t mr1 = c0 + bb * 16 + (r16 & ~1), mr2 = mr1 + 1;
      const int64_t mc = r0 + 32 * ap + (odd1 ? 16 : 0) + 4 * kq;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t mr = h ? mr2 : mr1;
        const float *v = h ? v2 : v1;
        if (mr >= n) continue;
        float *dst = G + mr * ld + mc;
        if (STORE4 && mc + 3 < n) {
          __builtin_nontemporal_store((tile_v4f){v[0], v[1], v[2], v[3]}, reinterpret_cast<tile_v4f *>(dst));
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (mc + e < n) __builtin_nontemporal_store(v[e], &dst[e]);
        }
      }
    }
}

}  // namespace svmx

// xchg_record.hpp -- packing of one exchange record of the solver into six self-stamped words.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

// A record carries 320 bits in five limbs: L0 = bits of v_up, L1 = bits of a_up, L2 = index
// word of up (low half) and of low (high half), L3 = bits of v_low, L4 = bits of a_low.  They
// travel as six 64-bit words; word w holds the 4-bit step stamp in bits 60..63 and bits
// [60w, 60w + 60) of the limb string in bits 0..59 (the last word only 20 of them).  A reader
// needs all six words to carry the stamp it waits for.  Each word is written and read as one
// 64-bit access, so a word is never seen half old and half new; a slot holds the stamp of two
// steps earlier or the current one, which differ modulo 16.
constexpr int REC_WORDS = 6;
constexpr unsigned long long REC_MASK60 = (1ull << 60) - 1ull;

__host__ __device__ inline unsigned long long rec_chunk(const unsigned long long (&L)[5], int w) {
  switch (w) {
    case 0: return L[0] & REC_MASK60;
    case 1: return ((L[0] >> 60) | (L[1] << 4)) & REC_MASK60;
    case 2: return ((L[1] >> 56) | (L[2] << 8)) & REC_MASK60;
    case 3: return ((L[2] >> 52) | (L[3] << 12)) & REC_MASK60;
    case 4: return ((L[3] >> 48) | (L[4] << 16)) & REC_MASK60;
    default: return L[4] >> 44;
  }
}

__host__ __device__ inline unsigned long long rec_word(const unsigned long long (&L)[5], int w, unsigned stamp) {
  return ((unsigned long long)(stamp & 15u) << 60) | rec_chunk(L, w);
}

__host__ __device__ inline bool rec_stamped(unsigned long long word, unsigned stamp) {
  return (unsigned)(word >> 60) == (stamp & 15u);
}

// Limbs from the six words (stamps ignored).
__host__ __device__ inline void rec_limbs(const unsigned long long (&c)[REC_WORDS], unsigned long long (&L)[5]) {
  const unsigned long long c0 = c[0] & REC_MASK60, c1 = c[1] & REC_MASK60, c2 = c[2] & REC_MASK60,
                           c3 = c[3] & REC_MASK60, c4 = c[4] & REC_MASK60, c5 = c[5] & REC_MASK60;
  L[0] = c0 | (c1 << 60);
  L[1] = (c1 >> 4) | (c2 << 56);
  L[2] = (c2 >> 8) | (c3 << 52);
  L[3] = (c3 >> 12) | (c4 << 48);
  L[4] = (c4 >> 16) | (c5 << 44);
}

}  // namespace svmx

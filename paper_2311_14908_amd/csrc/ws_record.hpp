// ws_record.hpp -- packing of one working-set candidate into three self-stamped words.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

// A candidate is a 64-bit sort key, a 32-bit aux word (local sample index, label sign in bit
// 31) and the 64 bits of its multiplier: 160 bits.  They travel as three 64-bit words; each
// word holds the 4-bit round stamp in bits 60..63 and 60 payload bits (the last word 40):
//   w0 = key[0, 60)
//   w1 = key[60, 64) | aux << 4 | a[0, 24) << 36
//   w2 = a[24, 64)
// A reader takes a candidate once all three words carry the stamp it waits for.
constexpr int CAND_WORDS = 3;
constexpr unsigned long long CAND_M60 = (1ull << 60) - 1ull;

__host__ __device__ inline void cand_words(unsigned long long key, unsigned aux, unsigned long long abits,
                                           unsigned stamp, unsigned long long (&w)[CAND_WORDS]) {
  const unsigned long long s = (unsigned long long)(stamp & 15u) << 60;
  w[0] = s | (key & CAND_M60);
  w[1] = s | (((key >> 60) | ((unsigned long long)aux << 4) | (abits << 36)) & CAND_M60);
  w[2] = s | (abits >> 24);
}

__host__ __device__ inline bool cand_stamped(unsigned long long w, unsigned stamp) {
  return (unsigned)(w >> 60) == (stamp & 15u);
}

__host__ __device__ inline void cand_fields(const unsigned long long (&w)[CAND_WORDS], unsigned long long &key,
                                            unsigned &aux, unsigned long long &abits) {
  key = (w[0] & CAND_M60) | ((w[1] & 15ull) << 60);
  aux = (unsigned)((w[1] >> 4) & 0xffffffffull);
  abits = ((w[1] >> 36) & 0xffffffull) | ((w[2] & CAND_M60) << 24);
}

// Order-preserving key of an fp64 value: a < b  <=>  key(a) < key(b) as unsigned integers, with
// -0 folded into +0 so that the two compare equal (NaN never occurs here).
__host__ __device__ inline unsigned long long f_key(double f) {
  if (f == 0.0) f = 0.0;
  union {
    double d;
    unsigned long long u;
  } c;
  c.d = f;
  return (c.u >> 63) ? ~c.u : (c.u | 0x8000000000000000ull);
}

__host__ __device__ inline double key_f(unsigned long long k) {
  union {
    double d;
    unsigned long long u;
  } c;
  c.u = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
  return c.d;
}

}  // namespace svmx

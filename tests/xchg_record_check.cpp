// Host check of the solver's six-word exchange record: every 320-bit limb string survives
// packing and unpacking, every word carries the stamp modulo 16, and a stamp two steps old is
// never taken for the current one.
#include "xchg_record.hpp"
#include <cstdio>
#include <random>
int main() {
  std::mt19937_64 g(12345);
  const unsigned long long special[] = {0ull, ~0ull, 1ull, 1ull << 63, 0x7ff0000000000000ull, 0x8000000000000000ull,
                                        0x3ff0000000000000ull, 0xfffffffffffffffeull};
  for (int it = 0; it < 200000; ++it) {
    unsigned long long L[5], back[5], c[svmx::REC_WORDS];
    for (int k = 0; k < 5; ++k) L[k] = (it < 64) ? special[(it + k) % 8] : g();
    const unsigned stamp = (unsigned)g();
    for (int w = 0; w < svmx::REC_WORDS; ++w) {
      c[w] = svmx::rec_word(L, w, stamp);
      if (!svmx::rec_stamped(c[w], stamp) || svmx::rec_stamped(c[w], stamp - 2) || svmx::rec_stamped(c[w], stamp + 2)) {
        printf("FAIL stamp\n");
        return 1;
      }
    }
    svmx::rec_limbs(c, back);
    for (int k = 0; k < 5; ++k)
      if (back[k] != L[k]) { printf("FAIL limb %d at %d\n", k, it); return 1; }
  }
  printf("ok: record round trip\n");
  return 0;
}

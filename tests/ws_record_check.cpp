// Host check of the working-set candidate words (csrc/ws_record.hpp): the order-preserving
// key of an fp64 value, its inverse, and the three-word packing with 4-bit stamps.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ws_record.hpp"

using namespace svmx;

static unsigned long long rnd64(unsigned long long &s) {
  s ^= s << 13;
  s ^= s >> 7;
  s ^= s << 17;
  return s;
}

static double bits_to_d(unsigned long long u) {
  double d;
  memcpy(&d, &u, 8);
  return d;
}

int main() {
  unsigned long long s = 0x9e3779b97f4a7c15ull;
  const double special[] = {0.0, -0.0, 1.0, -1.0, 1e-300, -1e-300, 4.9e-324, -4.9e-324, 1e300, -1e300, INFINITY,
                            -INFINITY, 0.5, -0.5, 2.0, -2.0};
  double v[4096];
  int nv = 0;
  for (double x : special) v[nv++] = x;
  while (nv < 4096) {
    double x = bits_to_d(rnd64(s));
    if (isnan(x)) continue;
    if (nv % 3 == 0) x = (double)((int)(rnd64(s) % 21) - 10) * 0.125;  // many exact ties
    v[nv++] = x;
  }
  for (int i = 0; i < nv; ++i) {
    const unsigned long long ki = f_key(v[i]);
    if (ki == ~0ull) { printf("sentinel key for %g\n", v[i]); return 1; }
    const double back = key_f(ki);
    if (!(back == v[i]) || (v[i] != 0.0 && memcmp(&back, &v[i], 8) != 0)) { printf("inverse of %g\n", v[i]); return 1; }
    for (int j = 0; j < nv; j += 7) {
      const unsigned long long kj = f_key(v[j]);
      const int want = v[i] < v[j] ? -1 : (v[i] > v[j] ? 1 : 0);
      const int got = ki < kj ? -1 : (ki > kj ? 1 : 0);
      if (want != got) { printf("order %g vs %g\n", v[i], v[j]); return 1; }
    }
  }
  for (int t = 0; t < 200000; ++t) {
    const unsigned long long key = t % 5 ? rnd64(s) : ~0ull;
    const unsigned aux = (unsigned)rnd64(s);
    const unsigned long long ab = rnd64(s);
    const unsigned stamp = (unsigned)(rnd64(s) & 63);
    unsigned long long w[CAND_WORDS];
    cand_words(key, aux, ab, stamp, w);
    for (int c = 0; c < CAND_WORDS; ++c)
      if (!cand_stamped(w[c], stamp) || cand_stamped(w[c], stamp + 1)) { printf("stamp\n"); return 1; }
    unsigned long long k2, ab2;
    unsigned aux2;
    cand_fields(w, k2, aux2, ab2);
    if (k2 != key || aux2 != aux || ab2 != ab) { printf("round trip %d\n", t); return 1; }
  }
  printf("ok\n");
  return 0;
}

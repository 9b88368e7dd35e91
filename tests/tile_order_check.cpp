// Host check that the upper-triangle tile order of the Gram kernels is a bijection.
#include "tile_order.hpp"
#include <cstdio>
#include <vector>
int main() {
  for (int64_t sup : {1, 8, 32}) {
    for (int64_t nt = 1; nt <= 300; ++nt) {
      const int64_t ntiles = nt * (nt + 1) / 2;
      std::vector<char> seen(nt * nt, 0);
      for (int64_t lin = 0; lin < ntiles; ++lin) {
        int64_t ti, tj;
        svmx::upper_tile_super(lin, nt, ti, tj, sup);
        if (ti < 0 || tj < ti || tj >= nt || seen[ti * nt + tj]) { printf("FAIL sup=%lld nt=%lld lin=%lld -> %lld %lld\n", (long long)sup, (long long)nt, (long long)lin, (long long)ti, (long long)tj); return 1; }
        seen[ti * nt + tj] = 1;
      }
    }
    // 782 (100000 rows)
    const int64_t nt = 782, ntiles = nt * (nt + 1) / 2;
    std::vector<char> seen(nt * nt, 0);
    for (int64_t lin = 0; lin < ntiles; ++lin) { int64_t ti, tj; svmx::upper_tile_super(lin, nt, ti, tj, sup); if (ti < 0 || tj < ti || tj >= nt || seen[ti*nt+tj]++) { printf("FAIL big sup=%lld\n", (long long)sup); return 1; } }
  }
  printf("ok: bijective for super-tiles of 1, 8 and 32, nt = 1..300 and 782\n");
  return 0;
}

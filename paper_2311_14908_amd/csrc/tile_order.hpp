// tile_order.hpp -- order of the upper-triangle tiles (ti <= tj) of a symmetric tile grid.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svmx {

// Linear index -> tile (ti, tj), ti <= tj < nt, in super-tile order: super-rows I of SUPER tile
// rows; in each, the diagonal super-tile (its upper triangle, row-major), then the super-tiles
// to its right (each row-major; the last one may be narrower).  A run of consecutive indices
// (what the workgroups of one XCD hold at once) therefore reads SUPER row slabs and SUPER column
// slabs, which stay in that XCD's L2, instead of one row slab and a different column slab per
// tile.  Bijective onto the upper triangle for every nt >= 1 and SUPER >= 1.  SUPER = 8 suits
// long rows, whose slabs are the traffic; short rows are bound by the tile stores, which a
// wider super-tile (32) keeps on fewer rows of the Gram at a time.
constexpr int64_t SUPER = 8;

__host__ __device__ inline void upper_tile_super(int64_t lin, int64_t nt, int64_t &ti, int64_t &tj,
                                                 const int64_t SUPER = svmx::SUPER) {
  int64_t I = 0, base = 0, r = 0, right = 0;
  for (;;) {
    r = nt - SUPER * I < SUPER ? nt - SUPER * I : SUPER;
    right = nt - SUPER * I - SUPER;
    if (right < 0) right = 0;
    const int64_t cnt = r * (r + 1) / 2 + r * right;
    if (lin < base + cnt) break;
    base += cnt;
    ++I;
  }
  int64_t off = lin - base;
  const int64_t r0 = SUPER * I;
  const int64_t dcnt = r * (r + 1) / 2;
  if (off < dcnt) {  // diagonal super-tile: row a holds r - a tiles
    int64_t a = 0;
    while (off >= r - a) {
      off -= r - a;
      ++a;
    }
    ti = r0 + a;
    tj = r0 + a + off;
    return;
  }
  off -= dcnt;
  const int64_t nfull = right / SUPER;  // full-width super-tiles to the right
  if (off < nfull * r * SUPER) {
    const int64_t J = off / (r * SUPER), o2 = off % (r * SUPER);
    ti = r0 + o2 / SUPER;
    tj = r0 + SUPER + J * SUPER + o2 % SUPER;
    return;
  }
  const int64_t o2 = off - nfull * r * SUPER;
  const int64_t c = right - nfull * SUPER;  // width of the last, narrower super-tile
  ti = r0 + o2 / c;
  tj = r0 + SUPER + nfull * SUPER + o2 % c;
}

}  // namespace svmx

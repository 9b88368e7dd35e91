// ws_smo.hip -- working-set SMO for gfx950: rounds of two-multiplier steps (paper, Section
// III.B) on a working set B of up to q samples, with the gradient of every sample updated once
// per round instead of once per step.
//
// One cooperative launch serves one problem.  Workgroups 0..nwg-1 own the samples
// [r*per_wg, (r+1)*per_wg) and keep their f, alpha and label in LDS; with more than one owner,
// one more workgroup runs the pair steps.  A round:
//   1. selection.  Every owner ranks its own members of I_up by (f, index) and of I_low by
//      (-f, index) with bitonic networks inside waves (a sorted list of 64 is one register per
//      lane) and publishes its 64 best of each side as candidates of three self-stamped words
//      (ws_record.hpp) -- the stamp-only protocol of the pair solver, so no fence is needed.
//      With more than 16 owners, group leaders merge their group's lists and publish those;
//      every workgroup then merges the (group) lists into the same two lists.  B = the first
//      q/2 of the I_up list, then those of the first q/2 of the I_low list that are not
//      already in B.
//   2. stop rule on the heads of the two lists, which are the maximal violating pair.
//   3. the owners fetch K_BB from the Gram between them and publish it; the solving workgroup
//      collects it into LDS, runs the pair steps on B in one wave until the gap on B is at most
//      max(tol, frac * gap of the round) or the round's step cap is reached, and publishes the
//      new multipliers of B; meanwhile every owner loads the Gram rows of B over its own
//      samples into LDS (over as many of them as 16,384 entries hold; the rest of the slice
//      reads them from the Gram in step 4);
//   4. every owner adds sum_p c_p K(B_p, j) to f_j of its own samples (c_p the change of a y
//      at B_p, in a fixed grouping of B's order) and stores the new multipliers of its
//      members of B.
#include "common.hpp"
#include "pair_step.hpp"
#include "ws_record.hpp"

#include <math.h>

namespace svmx {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int WS_BS = 256;
constexpr int WS_NW = WS_BS / 64;
constexpr int WS_QMAX = 128;        // working-set size limit (lists of 64 per side)
constexpr int WS_SLICE_MAX = 1024;  // samples per workgroup
constexpr int WS_LISTS_MAX = 16;    // lists merged by one workgroup at a level
constexpr int WS_LIST_WORDS = 2 * 64 * CAND_WORDS;  // one workgroup's (or group's) two lists
constexpr int WS_GATHER = 32;      // Gram loads a thread keeps in flight
constexpr int WS_QUARTERS = 4;     // fixed grouping of the f update's sum
constexpr int WS_MAXL = WS_LISTS_MAX / 2;     // lists one wave merges at a level
constexpr int WS_BCAST_PITCH = 2 * WS_QMAX + 8;  // steps word, then two words per multiplier
constexpr u64 KSENT = ~0ull;
constexpr unsigned VSENT = 0xffffffffu;

int ws_slice_max() { return WS_SLICE_MAX; }
int ws_q_max() { return WS_QMAX; }
int64_t ws_list_words() { return WS_LIST_WORDS; }
int64_t ws_bcast_words() { return 2LL * WS_BCAST_PITCH + 2LL * WS_QMAX * WS_QMAX; }
int ws_row_cap() { return WS_QMAX * WS_QMAX; }

// ---------------------------------------------------------------- sorted lists in a wave
// A list is 64 (key, value) pairs, one per lane, ascending in lexicographic order; value is a
// position that orders equal keys by sample index.  Empty entries are (KSENT, VSENT).

__device__ __forceinline__ bool kv_lt(u64 ka, unsigned va, u64 kb, unsigned vb) {
  return ka < kb || (ka == kb && va < vb);
}

// Value of lane (lane ^ d) for d = 1, 2, 4, 8, 16, 32 without LDS traffic: DPP quad
// permutes and a row rotation inside rows of 16; for d = 4 a left shift by 4 into the lanes
// 0-3 and 8-11 of each row and a right shift by 4 into the lanes 4-7 and 12-15 (two moves
// under complementary bank masks, no select); the gfx950 lane swaps across rows and halves
// (permlane16_swap with both operands x returns, in every lane, x of the pair's lane in the
// even row in its first result and of the lane in the odd row in its second; permlane32_swap
// likewise for the two halves).  The DPP moves take no old value (mov_dpp: every lane they
// write has a source), so x needs no copy.  d is a constant after unrolling.
__device__ __forceinline__ unsigned xor_lane(unsigned x, int d) {
  const int lane = threadIdx.x & 63;
  switch (d) {
    case 1: return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
    case 2: return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
    case 4: {
      const int t = __builtin_amdgcn_mov_dpp((int)x, 0x104, 0xF, 0x5, false);            // row_shl:4, banks 0, 2
      return (unsigned)__builtin_amdgcn_update_dpp(t, (int)x, 0x114, 0xF, 0xA, false);  // row_shr:4, banks 1, 3
    }
    case 8: return (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x128, 0xF, 0xF, false);  // row_ror:8
    case 16: {
      const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
      return (lane & 16) ? r[0] : r[1];
    }
    default: {
      const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
      return (lane & 32) ? r[0] : r[1];
    }
  }
}

__device__ __forceinline__ u64 xor_lane64(u64 x, int d) {
  return ((u64)xor_lane((unsigned)(x >> 32), d) << 32) | xor_lane((unsigned)x, d);
}

// Both entries of the pair (lane & ~d, lane | d), d = 16 or 32, in every lane: lo from the
// lane with bit d clear, hi from the one with it set (the two results of one lane swap).
__device__ __forceinline__ void pair_lanes(unsigned x, int d, unsigned &lo, unsigned &hi) {
  if (d == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    lo = r[0];
    hi = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    lo = r[0];
    hi = r[1];
  }
}

// Value of lane 63 - lane: the mirror inside each row of 16 (DPP row_mirror), then rows
// exchanged by xor 48.
__device__ __forceinline__ unsigned rev_lane(unsigned x) {
  const unsigned m = (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, false);  // row_mirror
  return xor_lane(xor_lane(m, 16), 32);
}

// Compare-exchange with the lane at distance d: in an ascending pair the lower lane keeps the
// smaller element, in a descending pair the larger one.  The entries of a list are distinct
// except empty ones, which are equal and interchangeable, so one comparison decides both lanes:
// a lane takes its partner's entry when "the partner's comes first" equals "keep the smaller".
// For d = 16 and 32 every lane holds both entries of its pair after the lane swaps, so it takes
// the pair's smaller or larger one directly: the same outcome without selecting the partner.
__device__ __forceinline__ void kv_cx(u64 &k, unsigned &v, int d, bool asc) {
  const int lane = threadIdx.x & 63;
  const bool keep_min = ((lane & d) == 0) == asc;
  if (d >= 16) {
    unsigned khl, khh, kll, klh, vl, vh;
    pair_lanes((unsigned)(k >> 32), d, khl, khh);
    pair_lanes((unsigned)k, d, kll, klh);
    pair_lanes(v, d, vl, vh);
    const u64 lo = ((u64)khl << 32) | kll, hi = ((u64)khh << 32) | klh;
    const bool take_hi = kv_lt(hi, vh, lo, vl) == keep_min;  // the pair's smaller entry, or its larger one
    k = take_hi ? hi : lo;
    v = take_hi ? vh : vl;
    return;
  }
  const u64 ok = xor_lane64(k, d);
  const unsigned ov = xor_lane(v, d);
  const bool take = kv_lt(ok, ov, k, v) == keep_min;  // selects, not a branch
  k = take ? ok : k;
  v = take ? ov : v;
}

__device__ __forceinline__ void wave_sort64(u64 &k, unsigned &v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int s = 2; s <= 64; s <<= 1)
#pragma unroll
    for (int d = s >> 1; d > 0; d >>= 1) kv_cx(k, v, d, (lane & s) == 0);
}

// (k, v) and (bk, bv) ascending -> the 64 smallest of both, ascending: the element-wise
// minimum of one list and the other reversed is bitonic and holds them; half-cleaners sort it.
__device__ __forceinline__ void wave_merge64(u64 &k, unsigned &v, u64 bk, unsigned bv) {
  const u64 rk = ((u64)rev_lane((unsigned)(bk >> 32)) << 32) | rev_lane((unsigned)bk);
  const unsigned rv = rev_lane(bv);
  const bool take = kv_lt(rk, rv, k, v);
  k = take ? rk : k;
  v = take ? rv : v;
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) kv_cx(k, v, d, true);
}

// Value of lane (lane ^ (M - 1)) for M = 16, 32, 64: the mirror inside groups of M lanes (DPP
// row_mirror, then the lane swaps across rows and halves).
template <int M>
__device__ __forceinline__ unsigned mirror_lane(unsigned x) {
  const unsigned m = (unsigned)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, false);  // row_mirror
  if (M == 16) return m;
  const unsigned m2 = xor_lane(m, 16);
  return M == 32 ? m2 : xor_lane(m2, 32);
}

template <int M>
__device__ __forceinline__ void kv_mirror(u64 k, unsigned v, u64 &ok, unsigned &ov) {
  ok = ((u64)mirror_lane<M>((unsigned)(k >> 32)) << 32) | mirror_lane<M>((unsigned)k);
  ov = mirror_lane<M>(v);
}

// Lists in segments.  A wave holds 64 / SEG lists of SEG entries, list s in lanes [s SEG,
// (s + 1) SEG), each ascending.  Merging keeps the SEG smallest of two lists: the element-wise
// minimum of one list and the other mirrored is bitonic and holds them, and the half-cleaners
// d = SEG/2 .. 1 sort it.  Lists of up to 16 entries thus merge four at a time in one register,
// with row-local DPP only.
template <int SEG>
__device__ __forceinline__ void seg_clean(u64 &k, unsigned &v) {
#pragma unroll
  for (int d = SEG / 2; d > 0; d >>= 1) kv_cx(k, v, d, true);
}

// One level inside a register: the partner of lane l is lane l ^ (M - 1), M = 2 SEG, 4 SEG, ...
// After the level with M = 2^j SEG every segment of a group of M lanes holds the same list (the
// merged list and its mirror image sort to the same entries), so the next level can again
// pair each segment with the mirror of the group of twice its size.
template <int SEG, int M>
__device__ __forceinline__ void seg_level(u64 &k, unsigned &v) {
  u64 ok;
  unsigned ov;
  kv_mirror<M>(k, v, ok, ov);
  const bool take = kv_lt(ok, ov, k, v);
  k = take ? ok : k;
  v = take ? ov : v;
  seg_clean<SEG>(k, v);
}

// All 64 / SEG lists of a register merged: afterwards every segment holds the SEG smallest.
template <int SEG>
__device__ __forceinline__ void seg_reduce(u64 &k, unsigned &v) {
  if (SEG <= 16) seg_level<SEG, 32>(k, v);
  if (SEG <= 32) seg_level<SEG, 64>(k, v);
}

// (k, v) and (bk, bv) hold the same layout of lists; (k, v) becomes the SEG smallest of both,
// segment by segment (SEG = 64: wave_merge64).
template <int SEG>
__device__ __forceinline__ void seg_merge(u64 &k, unsigned &v, u64 bk, unsigned bv) {
  u64 rk;
  unsigned rv;
  kv_mirror<SEG>(bk, bv, rk, rv);
  const bool take = kv_lt(rk, rv, k, v);
  k = take ? rk : k;
  v = take ? rv : v;
  seg_clean<SEG>(k, v);
}

__device__ __forceinline__ u64 readlane64(u64 x, int l) {
  return ((u64)(unsigned)__builtin_amdgcn_readlane((int)(x >> 32), l) << 32) |
         (unsigned)__builtin_amdgcn_readlane((int)x, l);
}

// s + c k, rounded as written (no contraction), so every placement sums to the same bits.
__device__ __forceinline__ double ws_acc(double s, double c, float k) {
#pragma clang fp contract(off)
  return s + c * (double)k;
}

__device__ __forceinline__ unsigned ws_aux(int64_t j, int y) { return (unsigned)j | (y < 0 ? 0x80000000u : 0u); }
__device__ __forceinline__ bool ws_in_up(int y, double a, double C) { return (y > 0 && a < C) || (y < 0 && a > 0.0); }
__device__ __forceinline__ bool ws_in_low(int y, double a, double C) { return (y > 0 && a > 0.0) || (y < 0 && a < C); }

// Local sample index -> global row: the two class ranges of a problem.
struct GMap {
  int64_t off0, len0, off1;
};
__device__ __forceinline__ int64_t ws_gmap(const GMap &P, int64_t j) {
  return j < P.len0 ? P.off0 + j : P.off1 + (j - P.len0);
}
__device__ __forceinline__ int64_t ws_gmap(const Prob &P, int64_t j) {
  return j < P.len0 ? P.off0 + j : P.off1 + (j - P.len0);
}
__device__ __forceinline__ int ws_label(const Prob &P, int64_t j) {
  return P.y ? gp(P.y)[ws_gmap(P, j)] : (j < P.len0 ? 1 : -1);
}

// A list entry: sort key and position (see the list comments above).
struct KV {
  u64 k;
  unsigned v;
};

// Lane `lane` of the calling wave publishes entry `lane` of a list: the three words of the
// candidate (key, aux, multiplier bits) or of an empty entry.
__device__ __forceinline__ void put_cand(u64 *list, int lane, u64 key, unsigned aux, u64 abits, unsigned stamp) {
  u64 w[CAND_WORDS];
  cand_words(key, aux, abits, stamp, w);
  u64 *dst = list + (size_t)lane * CAND_WORDS;
#pragma unroll
  for (int c = 0; c < CAND_WORDS; ++c) st_word(dst + c, w[c]);
}

// Wave-level: merge lists first, first + step, ... below last (side `side`, h <= SEG entries
// each; at most WS_MAXL lists) of the words at `words`: afterwards lanes 0 .. h - 1 of the
// result hold the h smallest, ascending (every segment of SEG lanes holds the same list).  A
// register takes 64 / SEG lists, list i of register r in segment i; v = (list - first0) * 64 +
// entry indexes the staging arrays, which receive each taken candidate's aux word and
// multiplier bits.  Every lane waits for its entries of all lists at once, so the round trips
// overlap.  Not inlined, and the result comes back by value: inside the kernel the compiler
// turned each compare-exchange into a branch with register copies (about twice the
// instructions of the selects it emits here).
template <int SEG>
__device__ __forceinline__ KV merge_lists(const u64 *words, int side, int first0, int first, int last,
                                                    int step, int h, unsigned stamp, unsigned *st_aux, u64 *st_ab,
                                                    uint64_t spin_limit, int32_t *err, int *abort_flag) {
  constexpr int R = 64 / SEG;         // lists per register
  constexpr int NR = WS_MAXL / R;     // registers
  const int lane = threadIdx.x & 63;
  const int seg = lane / SEG, e = lane % SEG;
  const int nl = first < last ? (last - first + step - 1) / step : 0;
  u64 w[NR][CAND_WORDS];
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int c = 0; c < CAND_WORDS; ++c) w[r][c] = 0;
  if (e < h) {
    unsigned pending = 0;
#pragma unroll
    for (int r = 0; r < NR; ++r)
      if (r * R + seg < nl) pending |= 1u << r;
    const uint64_t t0 = wall_clock64();
    while (pending) {
      // every load of the sweep first (no test between them, so they are in flight together)
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        const int i = r * R + seg;
        const u64 *src = words + ((size_t)(first + i * step) * 2 + side) * 64 * CAND_WORDS + (size_t)e * CAND_WORDS;
        if (pending & (1u << r)) {
#pragma unroll
          for (int c = 0; c < CAND_WORDS; ++c) w[r][c] = ld_word(src + c);
        }
      }
#pragma unroll
      for (int r = 0; r < NR; ++r) {
        bool ok = true;
#pragma unroll
        for (int c = 0; c < CAND_WORDS; ++c) ok = ok && cand_stamped(w[r][c], stamp);
        if (ok) pending &= ~(1u << r);
      }
      if (pending && wall_clock64() - t0 > spin_limit) {
        __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *abort_flag = 1;
        break;
      }
    }
  }
  u64 rk[NR];
  unsigned rv[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int i = r * R + seg;
    rk[r] = KSENT;
    rv[r] = VSENT;
    if (i < nl && e < h) {
      u64 key, ab;
      unsigned aux;
      cand_fields(w[r], key, aux, ab);
      if (key != KSENT) {
        rk[r] = key;
        rv[r] = (unsigned)((first + i * step - first0) * 64 + e);
        st_aux[rv[r]] = aux;
        st_ab[rv[r]] = ab;
      }
    }
  }
  // the lists of each register, then the registers pairwise
  const int nr = (nl + R - 1) / R;
#pragma unroll
  for (int r = 0; r < NR; ++r)
    if (r < nr && R > 1) seg_reduce<SEG>(rk[r], rv[r]);
#pragma unroll
  for (int span = 1; span < NR; span <<= 1)
#pragma unroll
    for (int r = 0; r + span < NR; r += 2 * span)
      if (r + span < nr) seg_merge<SEG>(rk[r], rv[r], rk[r + span], rv[r + span]);
  return KV{rk[0], rv[0]};
}

// Waits until words a and b both carry `stamp` (both loads in flight at once); returns their
// 60-bit payloads.
__device__ __forceinline__ void poll_word2(const u64 *a, const u64 *b, unsigned stamp, uint64_t spin_limit, int32_t *err,
                                          int *abort_flag, u64 &pa, u64 &pb) {
  const uint64_t t0 = wall_clock64();
  for (;;) {
    const u64 x = ld_word(a), y = ld_word(b);
    if (cand_stamped(x, stamp) && cand_stamped(y, stamp)) {
      pa = x & CAND_M60;
      pb = y & CAND_M60;
      return;
    }
    if (wall_clock64() - t0 > spin_limit) {
      __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *abort_flag = 1;
      pa = pb = 0;
      return;
    }
  }
}

// Waits until word `w` carries `stamp`; returns its 60-bit payload.
__device__ __forceinline__ u64 poll_word(const u64 *w, unsigned stamp, uint64_t spin_limit, int32_t *err,
                                         int *abort_flag) {
  const uint64_t t0 = wall_clock64();
  for (;;) {
    const u64 x = ld_word(w);
    if (cand_stamped(x, stamp)) return x & CAND_M60;
    if (wall_clock64() - t0 > spin_limit) {
      __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *abort_flag = 1;
      return 0;
    }
  }
}

// ---------------------------------------------------------------- the solver
struct WsLds {
  double f[WS_SLICE_MAX], a[WS_SLICE_MAX];
  signed char y[WS_SLICE_MAX];
  u64 key[2][WS_SLICE_MAX];  // sort keys of the I_up (by f) and I_low (by -f) sides, KSENT if not a member
  u64 lk[WS_NW][64];
  unsigned lv[WS_NW][64];
  u64 pk[WS_NW][64];  // own lists: each wave's members below its threshold, 64 at a time
  unsigned pv[WS_NW][64];
  union {
    struct {
      unsigned aux[2][WS_LISTS_MAX * 64];
      u64 ab[2][WS_LISTS_MAX * 64];
    } st;
    float K[WS_QMAX * WS_QMAX];  // solver: K_BB; owners: the Gram rows of B over the own samples
    struct {
      h8 b[2][8][WS_QMAX];  // row path, one block of samples: B rows, [hi, lo][k chunk][row]
      h8 s[2][8][128];      // and the samples, 64 features a stage
    } rs64;
  } u;
  union {
    double part[WS_QUARTERS][WS_SLICE_MAX];
    struct {
      h8 b[2][4][WS_QMAX];  // row path: B rows, [hi, lo][k chunk of 8][row]
      h8 s[2][4][128];      // and a block of own samples, [hi, lo][k chunk][column]
    } rs;
  } w;
  alignas(16) int bi[WS_QMAX];  // read four at a time
  signed char by[WS_QMAX];
  double bf[WS_QMAX], ba[WS_QMAX], bn[WS_QMAX];
  int nzp[WS_QMAX];
  int64_t roff[WS_QMAX];   // Gram row offset of B_p
  float bsc[WS_QMAX], bnr[WS_QMAX];  // row path: scale and squared norm of B_p
  int own[WS_QMAX];        // positions of B among this workgroup's samples
  int nown;
  int64_t nzoff[WS_QMAX];  // Gram row offset and change of the r-th nonzero change
  double nzc[WS_QMAX];
  int nu, nl, m, nnz, il, abort_flag;
  double bl;
  int64_t steps;
};

// Min of a over each half of the wave (lanes 0 .. 31 and 32 .. 63), left in lanes 31 and 63:
// the first five rounds of wave_minmax, the row-15 broadcast reaching rows 1 and 3 only.
__device__ __forceinline__ void halves_min(double &a) {
#define SVMX_HM_FULL(CTRL)                       \
  {                                              \
    const double oa = dpp_full_d<CTRL>(a);       \
    a = oa < a ? oa : a;                         \
  }
  SVMX_HM_FULL(0xB1)   // quad_perm [1,0,3,2]
  SVMX_HM_FULL(0x4E)   // quad_perm [2,3,0,1]
  SVMX_HM_FULL(0x124)  // row_ror:4
  SVMX_HM_FULL(0x128)  // row_ror:8
#undef SVMX_HM_FULL
  const double oa = dpp_mov_d<0x142, 0xA>(a);  // row_bcast:15 -> rows 1, 3
  a = oa < a ? oa : a;
}

// The pair steps on B (wave 0 only; K_BB in S.u.K): S.bn receives the new multipliers,
// S.steps the number of steps.  Lane l holds B positions l and l + 64.  The step is written
// without lane-divergent branches, and the two wave reductions are independent chains that
// the scheduler can interleave.  Not inlined: the loop gets registers of its own instead of
// reloading the kernel's spilled scalars every step.
// The parameters come as values: a reference to the kernel's parameter block would make the
// kernel keep a copy of it in scratch memory and reload fields from there inside the round.
// MAXM bounds m: up to 64 a lane holds one member of B (position lane), above two (lane and
// lane + 64).  Every bound gives the same steps (and local_solve_halves those for m <= 32).
template <int MAXM>
__device__ __attribute__((noinline)) void local_solve(WsLds &S, double C, double tol, double frac, int64_t max_inner_p,
                                                     int64_t max_iter, int m, double b_up, double b_low, int64_t t) {
  constexpr bool TWO = MAXM > 64;
  const int lane = threadIdx.x & 63;
  const int p0 = lane, p1 = lane + 64;
  const bool v0 = p0 < m, v1 = TWO && p1 < m;
  double f0 = v0 ? S.bf[p0] : 0.0, f1 = v1 ? S.bf[p1] : 0.0;
  double a0 = v0 ? S.ba[p0] : 0.0, a1 = v1 ? S.ba[p1] : 0.0;
  const int y0 = v0 ? S.by[p0] : 0, y1 = v1 ? S.by[p1] : 0;
  const int i0 = v0 ? S.bi[p0] : IBIG, i1 = v1 ? S.bi[p1] : IBIG;
  const double tl = fmax(tol, frac * (b_low - b_up));
  const int max_inner = (int)min<int64_t>(max_inner_p, max_iter - t);
  int inner = 0;
  for (; inner < max_inner; ++inner) {
    // this lane's best member of each side (positions l and l + 64)
    const bool u0 = ws_in_up(y0, a0, C), u1 = TWO && ws_in_up(y1, a1, C);
    const bool l0 = ws_in_low(y0, a0, C), l1 = TWO && ws_in_low(y1, a1, C);
    // position l + 64 wins a lane's side on a smaller (larger) f, or an equal f and a smaller
    // index (bitwise forms: no branches)
    const bool tie_i = (f1 == f0) & (i1 < i0);
    const bool up1 = TWO && (u1 & (!u0 | (f1 < f0) | tie_i));
    const bool lo1 = TWO && (l1 & (!l0 | (f1 > f0) | tie_i));
    const double cu_v = up1 ? f1 : (u0 ? f0 : INFINITY);
    const int cu_i = up1 ? i1 : (u0 ? i0 : IBIG);
    const int cu_p = up1 ? p1 : (u0 ? p0 : -1);
    const double cl_v = lo1 ? f1 : (l0 ? f0 : -INFINITY);
    const int cl_i = lo1 ? i1 : (l0 ? i0 : IBIG);
    const int cl_p = lo1 ? p1 : (l0 ? p0 : -1);
    // wave extremes of both sides, then the smallest index among the lanes holding each
    double ru = cu_v, rl = cl_v;
    wave_minmax(ru, rl);
    const unsigned long long tu = (unsigned long long)__ballot(cu_v == ru);
    const unsigned long long tw = (unsigned long long)__ballot(cl_v == rl);
    int lu = __ffsll(tu) - 1, ll = __ffsll(tw) - 1;
    if (__popcll(tu) > 1) {
      const int best = wave_min_int(cu_v == ru ? cu_i : IBIG);
      lu = __ffsll((unsigned long long)__ballot(cu_v == ru && cu_i == best)) - 1;
    }
    if (__popcll(tw) > 1) {
      const int best = wave_min_int(cl_v == rl ? cl_i : IBIG);
      ll = __ffsll((unsigned long long)__ballot(cl_v == rl && cl_i == best)) - 1;
    }
    lu &= 63;
    ll &= 63;
    const int pu = __builtin_amdgcn_readlane(cu_p, lu), pl = __builtin_amdgcn_readlane(cl_p, ll);
    if (pu < 0 || pl < 0) break;
    const double fu = readlane_d(cu_v, lu), fl = readlane_d(cl_v, ll);
    if (fl - fu <= tl) break;
    const bool hu1 = TWO && pu >= 64, hl1 = TWO && pl >= 64;  // which of its two positions the winner holds
    const double au = readlane_d(hu1 ? a1 : a0, lu), al = readlane_d(hl1 ? a1 : a0, ll);
    const double yu = (double)__builtin_amdgcn_readlane(hu1 ? y1 : y0, lu);
    const double yl = (double)__builtin_amdgcn_readlane(hl1 ? y1 : y0, ll);
    const float *Ku = S.u.K + pu * WS_QMAX, *Kl = S.u.K + pl * WS_QMAX;
    const double kul = (double)Ku[pl];
    const float ku0 = Ku[p0], kl0 = Kl[p0];
    const PairStep ps = solve_pair(C, fu, fl, au, al, yu, yl, kul);
    const double cu = (ps.au - au) * yu, cl = (ps.al - al) * yl;
    f0 = f_update(f0, cu, ku0, cl, kl0);
    a0 = p0 == pu ? ps.au : (p0 == pl ? ps.al : a0);
    if (TWO) {
      const float ku1 = Ku[p1], kl1 = Kl[p1];
      f1 = f_update(f1, cu, ku1, cl, kl1);
      a1 = p1 == pu ? ps.au : (p1 == pl ? ps.al : a1);
    }
  }
  if (v0) S.bn[p0] = a0;
  if (v1) S.bn[p1] = a1;
  if (lane == 0) S.steps = inner;
}

// The pair steps on B for m <= 32, as local_solve: member p sits in lanes p and p + 32, the
// lower half offering it to I_up by f, the upper half to I_low by -f, so one chain of wave
// reductions finds both extremes (the smallest f in I_up and the largest in I_low, ties to the
// smaller sample index: the choices of local_solve).  Both halves update their copy of every
// member with the same arithmetic, so the copies stay equal and the steps are those of
// local_solve.
__device__ __attribute__((noinline)) void local_solve_halves(WsLds &S, double C, double tol, double frac,
                                                            int64_t max_inner_p, int64_t max_iter, int m, double b_up,
                                                            double b_low, int64_t t) {
  const int lane = threadIdx.x & 63, p = lane & 31;
  const bool low = lane >= 32;
  const bool v = p < m;
  double f = v ? S.bf[p] : 0.0;
  double a = v ? S.ba[p] : 0.0;
  const int y = v ? S.by[p] : 0;
  const int i = v ? S.bi[p] : IBIG;
  const double tl = fmax(tol, frac * (b_low - b_up));
  const int max_inner = (int)min<int64_t>(max_inner_p, max_iter - t);
  // membership as in ws_in_up / ws_in_low: I_up takes y > 0 with a < C or y < 0 with a > 0,
  // I_low the reverse; which label goes with which test is fixed for the lane
  const bool with_below_c = low ? y < 0 : y > 0, with_above_0 = low ? y > 0 : y < 0;
  int inner = 0;
  for (; inner < max_inner; ++inner) {
    const bool mem = (with_below_c & (a < C)) | (with_above_0 & (a > 0.0));
    const double cv = mem ? (low ? -f : f) : INFINITY;
    double r = cv;
    halves_min(r);
    const double ru = readlane_d(r, 31), rl = readlane_d(r, 63);  // rl = -(largest f in I_low)
    const bool tie = low ? cv == rl : cv == ru;
    unsigned long long tu = (unsigned long long)__ballot(cv == ru) & 0xffffffffull;
    unsigned long long tw = (unsigned long long)__ballot(cv == rl) & ~0xffffffffull;
    if (__popcll(tu) > 1) {
      const int best = wave_min_int(!low && tie ? i : IBIG);
      tu = (unsigned long long)__ballot(!low && tie && i == best);
    }
    if (__popcll(tw) > 1) {
      const int best = wave_min_int(low && tie ? i : IBIG);
      tw = (unsigned long long)__ballot(low && tie && i == best);
    }
    const int lu = (__ffsll(tu) - 1) & 63, ll = (__ffsll(tw) - 1) & 63;
    const int cp = mem ? p : -1;
    const int pu = __builtin_amdgcn_readlane(cp, lu), pl = __builtin_amdgcn_readlane(cp, ll);
    if (pu < 0 || pl < 0) break;
    const double fu = readlane_d(f, lu), fl = readlane_d(f, ll);
    if (fl - fu <= tl) break;
    const double au = readlane_d(a, lu), al = readlane_d(a, ll);
    const double yu = (double)__builtin_amdgcn_readlane(y, lu);
    const double yl = (double)__builtin_amdgcn_readlane(y, ll);
    const float *Ku = S.u.K + pu * WS_QMAX, *Kl = S.u.K + pl * WS_QMAX;
    const double kul = (double)Ku[pl];
    const float ku = Ku[p], kl = Kl[p];
    const PairStep ps = solve_pair(C, fu, fl, au, al, yu, yl, kul);
    const double cu = (ps.au - au) * yu, cl = (ps.al - al) * yl;
    f = f_update(f, cu, ku, cl, kl);
    a = p == pu ? ps.au : (p == pl ? ps.al : a);
  }
  if (!low && v) S.bn[p] = a;
  if (lane == 0) S.steps = inner;
}

// Row path: K(x_{B_p}, x_j) for p < m and the workgroup's samples j < len into
// S.u.K[p * len + j] (m * len <= WS_QMAX^2).  The products run on v_mfma_f32_16x16x32_f16 with
// the split-fp16 rows (hi and lo halves, three products into one fp32 accumulator), the same
// arithmetic as the Gram kernel's: K = exp2(c max(0, n_p + n_j - 2 s_p s_j acc)), 1 between
// identical samples.  Samples go in blocks of 128 columns; both operands pass through LDS one
// chunk of 32 features at a time, with the global loads of the next two chunks in flight while
// a chunk is multiplied; wave w takes the 16 x 16 tiles w, w + 4, ...  Not inlined: its
// accumulators and load buffers get registers of their own.
struct RowLoad {
  h8 r[8];  // this thread's share of a chunk: [B hi x2, B lo x2, samples hi x2, samples lo x2]
};

__device__ __forceinline__ void row_chunk_load(RowLoad &L, const SplitX &X, int64_t gb, int64_t gs, int64_t k0,
                                               int lkq) {
#pragma unroll
  for (int sl = 0; sl < 2; ++sl) {
    const _Float16 *hb = sl ? X.lo : X.hi;
    if (gb >= 0) {
      const SVMX_GLOBAL h8 *q8 = gp(reinterpret_cast<const h8 *>(hb + gb * X.dp + k0)) + lkq;
      L.r[2 * sl] = q8[0];
      L.r[2 * sl + 1] = q8[1];
    } else {
      L.r[2 * sl] = (h8){};
      L.r[2 * sl + 1] = (h8){};
    }
    if (gs >= 0) {
      const SVMX_GLOBAL h8 *q8 = gp(reinterpret_cast<const h8 *>(hb + gs * X.dp + k0)) + lkq;
      L.r[4 + 2 * sl] = q8[0];
      L.r[4 + 2 * sl + 1] = q8[1];
    } else {
      L.r[4 + 2 * sl] = (h8){};
      L.r[4 + 2 * sl + 1] = (h8){};
    }
  }
}

__device__ __forceinline__ void row_chunk_store(WsLds &S, const RowLoad &L, int lrow, int lkq) {
#pragma unroll
  for (int sl = 0; sl < 2; ++sl) {
    S.w.rs.b[sl][lkq][lrow] = L.r[2 * sl];
    S.w.rs.b[sl][lkq + 1][lrow] = L.r[2 * sl + 1];
    S.w.rs.s[sl][lkq][lrow] = L.r[4 + 2 * sl];
    S.w.rs.s[sl][lkq + 1][lrow] = L.r[4 + 2 * sl + 1];
  }
}

__device__ __forceinline__ void row_chunk_mma(WsLds &S, v4f (&acc)[16], int ntile, int tj_n) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kq = lane >> 4, r16 = lane & 15;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int tile = wave + 4 * i;
    if (tile < ntile) {
      const int tp = tile / tj_n, tj = tile - tp * tj_n;
      const h8 ah = S.w.rs.b[0][kq][tp * 16 + r16], al = S.w.rs.b[1][kq][tp * 16 + r16];
      const h8 bh = S.w.rs.s[0][kq][tj * 16 + r16], bl = S.w.rs.s[1][kq][tj * 16 + r16];
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh, acc[i], 0, 0, 0);
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl, acc[i], 0, 0, 0);
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh, acc[i], 0, 0, 0);
    }
  }
}

// One block of at most 128 samples (the usual case): stages of 64 features staged in S.u (the
// destination of the results, free until the last stage), two stages in flight; every load
// instruction of a wave reads 8 whole 128-byte lines (16 bytes a lane: thread t takes chunk
// t % 8 of half (t / 8) % 2 of rows t / 16 + 16 i); wave w takes the row tiles w and w + 4 with
// every column tile, so each operand read from LDS feeds up to 8 (A) or 2 (B) tiles.
struct RowLoad64 {
  h8 b[8], s[8];  // rows t / 16 + 16 i of B and of the samples
};

__device__ __forceinline__ void row64_load(RowLoad64 &L, const SplitX &X, const int64_t (&gb)[8],
                                           const int64_t (&gs)[8], int64_t k0, bool full) {
  const int c = threadIdx.x & 7, half = (threadIdx.x >> 3) & 1;
  const _Float16 *hb = half ? X.lo : X.hi;
  const bool in = full || c < 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    L.b[i] = (gb[i] >= 0 && in) ? gp(reinterpret_cast<const h8 *>(hb + gb[i] * X.dp + k0))[c] : (h8){};
    L.s[i] = (gs[i] >= 0 && in) ? gp(reinterpret_cast<const h8 *>(hb + gs[i] * X.dp + k0))[c] : (h8){};
  }
}

__device__ __forceinline__ void row64_store(WsLds &S, const RowLoad64 &L) {
  const int c = threadIdx.x & 7, half = (threadIdx.x >> 3) & 1, r0 = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    S.u.rs64.b[half][c][r0 + 16 * i] = L.b[i];
    S.u.rs64.s[half][c][r0 + 16 * i] = L.s[i];
  }
}

__device__ __forceinline__ void row64_mma(WsLds &S, v4f (&acc)[2][8], int tp_n, int tj_n, int ksteps) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int kq = lane >> 4, r16 = lane & 15;
  for (int ks = 0; ks < ksteps; ++ks) {
    const int c = ks * 4 + kq;
    h8 ah[2], al[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int tp = wave + 4 * a;
      ah[a] = S.u.rs64.b[0][c][(tp & 7) * 16 + r16];
      al[a] = S.u.rs64.b[1][c][(tp & 7) * 16 + r16];
    }
#pragma unroll
    for (int tj = 0; tj < 8; ++tj) {
      if (tj < tj_n) {
        const h8 bh = S.u.rs64.s[0][c][tj * 16 + r16], bl = S.u.rs64.s[1][c][tj * 16 + r16];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
          if (wave + 4 * a < tp_n) {
            acc[a][tj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bh, acc[a][tj], 0, 0, 0);
            acc[a][tj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[a], bl, acc[a][tj], 0, 0, 0);
            acc[a][tj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[a], bh, acc[a][tj], 0, 0, 0);
          }
        }
      }
    }
  }
}

__device__ __attribute__((noinline)) void owner_rows_block(WsLds &S, SplitX X, float cexp, GMap P, int m,
                                                          int64_t base, int len) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kq = lane >> 4, r16 = lane & 15;
  const int nst = (int)((X.dp + 63) / 64);  // stages; the last one holds 32 features when dp % 64 == 32
  const int tp_n = (m + 15) / 16, tj_n = (len + 15) / 16;
  int64_t gb[8], gs[8];  // this thread's rows of B and of the samples (-1: past the end)
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = (tid >> 4) + 16 * i;
    gb[i] = r < m ? ws_gmap(P, S.bi[r]) : -1;
    gs[i] = r < len ? ws_gmap(P, base + r) : -1;
  }
  v4f acc[2][8];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int tj = 0; tj < 8; ++tj) acc[a][tj] = (v4f){0.f, 0.f, 0.f, 0.f};
  const auto full = [&](int st) { return (int64_t)st * 64 + 64 <= X.dp; };
  RowLoad64 la, lb;
  row64_load(la, X, gb, gs, 0, full(0));
  if (nst > 1) row64_load(lb, X, gb, gs, 64, full(1));
  for (int st = 0; st < nst; st += 2) {
    __syncthreads();  // the previous stage's operands have been read
    row64_store(S, la);
    __syncthreads();
    if (st + 2 < nst) row64_load(la, X, gb, gs, (int64_t)(st + 2) * 64, full(st + 2));
    row64_mma(S, acc, tp_n, tj_n, full(st) ? 2 : 1);
    if (st + 1 >= nst) break;
    __syncthreads();
    row64_store(S, lb);
    __syncthreads();
    if (st + 3 < nst) row64_load(lb, X, gb, gs, (int64_t)(st + 3) * 64, full(st + 3));
    row64_mma(S, acc, tp_n, tj_n, full(st + 1) ? 2 : 1);
  }
  __syncthreads();  // S.u now receives the results
  // lane l holds rows 4 (l / 16) + e and column l % 16 of each tile
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int tp = wave + 4 * a;
    if (tp < tp_n) {
#pragma unroll
      for (int tj = 0; tj < 8; ++tj) {
        const int j = tj * 16 + r16;
        if (tj < tj_n && j < len) {
          const int64_t gj = ws_gmap(P, base + j);
          const float sj = gp(X.scale)[gj], nj = gp(X.nrm)[gj];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int pr = tp * 16 + 4 * kq + e;
            if (pr < m) {
              const float dot = (acc[a][tj][e] * S.bsc[pr]) * sj;
              float t = S.bnr[pr] + nj - 2.0f * dot;
              t = t > 0.f ? t : 0.f;
              S.u.K[pr * len + j] = (S.bi[pr] == base + j) ? 1.0f : __builtin_amdgcn_exp2f(cexp * t);
            }
          }
        }
      }
    }
  }
  __syncthreads();
}

__device__ __attribute__((noinline)) void owner_rows(WsLds &S, SplitX X, float cexp, GMap P, int m, int64_t base,
                                                    int len) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kq = lane >> 4, r16 = lane & 15;
  const int stages = (int)(X.dp / 32);
  const int tp_n = (m + 15) / 16;
  const int lrow = tid >> 1, lkq = (tid & 1) * 2;  // this thread's share of a chunk
  const int64_t gb = lrow < m ? ws_gmap(P, S.bi[lrow]) : -1;
  for (int j0 = 0; j0 < len; j0 += 128) {
    const int cnt = min(128, len - j0);
    const int tj_n = (cnt + 15) / 16;
    const int ntile = tp_n * tj_n;
    const int64_t gs = lrow < cnt ? ws_gmap(P, base + j0 + lrow) : -1;
    v4f acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = (v4f){0.f, 0.f, 0.f, 0.f};
    RowLoad la, lb;
    row_chunk_load(la, X, gb, gs, 0, lkq);
    if (stages > 1) row_chunk_load(lb, X, gb, gs, 32, lkq);
    for (int st = 0; st < stages; st += 2) {
      __syncthreads();  // the previous chunk's operands have been read
      row_chunk_store(S, la, lrow, lkq);
      __syncthreads();
      if (st + 2 < stages) row_chunk_load(la, X, gb, gs, (int64_t)(st + 2) * 32, lkq);
      row_chunk_mma(S, acc, ntile, tj_n);
      if (st + 1 >= stages) break;
      __syncthreads();
      row_chunk_store(S, lb, lrow, lkq);
      __syncthreads();
      if (st + 3 < stages) row_chunk_load(lb, X, gb, gs, (int64_t)(st + 3) * 32, lkq);
      row_chunk_mma(S, acc, ntile, tj_n);
    }
    // lane l holds rows 4 (l / 16) + e and column l % 16 of each tile
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tile = wave + 4 * i;
      if (tile < ntile) {
        const int tp = tile / tj_n, tj = tile - tp * tj_n;
        const int j = j0 + tj * 16 + r16;
        if (j < len) {
          const int64_t gj = ws_gmap(P, base + j);
          const float sj = gp(X.scale)[gj], nj = gp(X.nrm)[gj];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int pr = tp * 16 + 4 * kq + e;
            if (pr < m) {
              const float dot = (acc[i][e] * S.bsc[pr]) * sj;
              float t = S.bnr[pr] + nj - 2.0f * dot;
              t = t > 0.f ? t : 0.f;
              S.u.K[pr * len + j] = (S.bi[pr] == base + j) ? 1.0f : __builtin_amdgcn_exp2f(cexp * t);
            }
          }
        }
      }
    }
    __syncthreads();  // the stage is rewritten by the next block
  }
}

// Keys of sample pos for both sides (0: I_up by f, 1: I_low by -f; KSENT where it is not a
// member), written wherever f or a of the sample is set, so that the lists read them ready-made.
__device__ __forceinline__ void put_keys(WsLds &S, int pos, double f, double a, int y, double C) {
  S.key[0][pos] = ws_in_up(y, a, C) ? f_key(f) : KSENT;
  S.key[1][pos] = ws_in_low(y, a, C) ? f_key(-f) : KSENT;
}

// Key of sample pos for a side, or KSENT if it is not a member or past the slice.
__device__ __forceinline__ u64 side_key(const WsLds &S, int side, int pos, int len) {
  return pos < len ? S.key[side][pos] : KSENT;
}

// Bitonic sort of the first S lanes (S = 16, 32, 64): lanes S .. 63 must hold empty entries,
// which stay there, so the 64 lanes read as one ascending list.
template <int S>
__device__ __forceinline__ void wave_sort_first(u64 &k, unsigned &v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int s = 2; s <= S; s <<= 1)
#pragma unroll
    for (int d = s >> 1; d > 0; d >>= 1) kv_cx(k, v, d, (lane & s) == 0);
}

// One wave's best members of one side among the chunks of 64 samples c = half, half + 2, ...:
// (k, v) ascending, lanes 0 .. h - 1 exact.  With one chunk it is sorted outright.  With more,
// every member's key stays in registers and each lane keeps its own best; the minima of groups
// of 64 / SEG lanes are at least SEG >= h members, so the largest of those minima is a threshold
// no member of the wave's best h exceeds.  Only the members at or below it are gathered in LDS
// and sorted (over 16, 32 or 64 lanes, as many as they need), 64 at a time, the threshold
// tightening to the list's h-th entry after each batch.

constexpr int WS_OWN_CHUNKS = WS_SLICE_MAX / 128;  // chunks of 64 samples one wave takes

template <int SEG>
__device__ __attribute__((noinline)) KV own_list(WsLds &S, int side, int half, int len, int h) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nch = (len + 63) / 64;
  u64 k = KSENT;
  unsigned v = VSENT;
  if (nch - half <= 2) {  // at most one chunk for this wave
    if (half < nch) {
      u64 ck = side_key(S, side, half * 64 + lane, len);
      unsigned cv = ck != KSENT ? (unsigned)(half * 64 + lane) : VSENT;
      if (__ballot(ck != KSENT) != 0) wave_sort64(ck, cv);
      k = ck;
      v = cv;
    }
    return KV{k, v};
  }
  u64 ck[WS_OWN_CHUNKS];
  u64 tk = KSENT;
  unsigned tv = VSENT;
#pragma unroll
  for (int i = 0; i < WS_OWN_CHUNKS; ++i) {  // every read first (addresses clamped into the slice)
    const int pos = (half + 2 * i) * 64 + lane;
    ck[i] = S.key[side][pos < len ? pos : 0];
  }
  __asm__ volatile("" ::: "memory");  // the reads are issued before the first is used
#pragma unroll
  for (int i = 0; i < WS_OWN_CHUNKS; ++i) {
    const int pos = (half + 2 * i) * 64 + lane;
    if (pos >= len) ck[i] = KSENT;  // empty past len
    const bool better = ck[i] != KSENT && kv_lt(ck[i], (unsigned)pos, tk, tv);
    tk = better ? ck[i] : tk;
    tv = better ? (unsigned)pos : tv;
  }
  // minimum over groups of G lanes, then the maximum over the 64 / G >= SEG >= h groups
  constexpr int G = 64 / SEG;
#pragma unroll
  for (int d = 1; d < G; d <<= 1) {
    const u64 ok = xor_lane64(tk, d);
    const unsigned ov = xor_lane(tv, d);
    if (kv_lt(ok, ov, tk, tv)) {
      tk = ok;
      tv = ov;
    }
  }
#pragma unroll
  for (int d = G; d < 64; d <<= 1) {
    const u64 ok = xor_lane64(tk, d);
    const unsigned ov = xor_lane(tv, d);
    if (kv_lt(tk, tv, ok, ov)) {
      tk = ok;
      tv = ov;
    }
  }
  bool have = false;
  int np = 0;
  u64 *pk = S.pk[wave];
  unsigned *pv = S.pv[wave];
  const u64 below = (1ull << lane) - 1ull;
  auto flush = [&]() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    u64 fk = lane < np ? pk[lane] : KSENT;
    unsigned fv = lane < np ? pv[lane] : VSENT;
    if (np <= 16)
      wave_sort_first<16>(fk, fv);
    else if (np <= 32)
      wave_sort_first<32>(fk, fv);
    else
      wave_sort_first<64>(fk, fv);
    if (!have) {
      k = fk;
      v = fv;
      have = true;
    } else {
      wave_merge64(k, v, fk, fv);
    }
    const u64 nk = readlane64(k, h - 1);
    const unsigned nv = (unsigned)__builtin_amdgcn_readlane((int)v, h - 1);
    if (kv_lt(nk, nv, tk, tv)) {
      tk = nk;
      tv = nv;
    }
    np = 0;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
#pragma unroll
  for (int i = 0; i < WS_OWN_CHUNKS; ++i) {
    const int pos = (half + 2 * i) * 64 + lane;
    bool q = ck[i] != KSENT && !kv_lt(tk, tv, ck[i], (unsigned)pos);
    u64 mask = __ballot(q);
    int nq = __popcll(mask);
    if (nq == 0) continue;
    if (np + nq > 64) {
      flush();
      q = q && !kv_lt(tk, tv, ck[i], (unsigned)pos);
      mask = __ballot(q);
      nq = __popcll(mask);
    }
    if (q) {
      const int at = np + __popcll(mask & below);
      pk[at] = ck[i];
      pv[at] = (unsigned)pos;
    }
    np += nq;
  }
  if (np > 0) flush();
  return KV{k, v};
}

template <bool GRAM, int SEG>
__global__ void __launch_bounds__(WS_BS) ws_solve(WsParams p) {
  __shared__ WsLds S;
  const SolveParams &sp = p.sp;
  const int32_t pid = sp.wg_prob[blockIdx.x];
  const Prob P = sp.probs[pid];
  const int rank = (int)blockIdx.x - P.wg0;
  Ctl *ctl = P.ctl;
  if (ctl->status != ST_RUNNING) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const double C = sp.C;
  const int h = p.q / 2;
  // Workgroups 0..nwg-1 own the samples; with more than one of them, workgroup nwg runs the
  // pair steps while the owners fetch the Gram rows of B they will need.
  const bool solo = P.nwg == 1;
  const bool solver = solo || rank == P.nwg;
  const bool owner = rank < P.nwg;
  const int64_t base = owner ? (int64_t)rank * P.per_wg : 0;
  const int len = owner ? (int)min<int64_t>(P.per_wg, P.n - base) : 0;
  u64 *bcast = P.slots2 + 2 * (size_t)P.ng * WS_LIST_WORDS;
  // K_BB as published by the owners, [2][WS_QMAX][WS_QMAX] words of (32-bit round stamp, fp32
  // bits) -- 32-bit stamps, so a word of an earlier round never passes for a current one,
  // whichever entries a round leaves untouched
  u64 *kbuf = bcast + 2 * WS_BCAST_PITCH;

  for (int j = tid; j < len; j += WS_BS) {
    const double fj = gp(P.f)[base + j], aj = gp(P.alpha)[base + j];
    const int yj = ws_label(P, base + j);
    S.f[j] = fj;
    S.a[j] = aj;
    S.y[j] = (signed char)yj;
    put_keys(S, j, fj, aj, yj, C);
  }
  if (tid == 0) S.abort_flag = 0;
  int64_t t = ctl->t;
  int64_t round = p.rounds[pid];
  const int64_t t_end = min(t + sp.steps, sp.max_iter);
  __syncthreads();

  int status = ST_RUNNING;
  double b_up = 0.0, b_low = 0.0;
  int iu = IBIG, il = IBIG;
  for (;;) {
    const unsigned stamp = (unsigned)(round + 1);
    const size_t par = (size_t)(round & 1);
    const int side = wave >> 1, half = wave & 1;
    // ---- 1a. this workgroup's two lists: waves 0, 1 take I_up, waves 2, 3 take I_low; each
    // wave takes every other chunk of 64 samples (own_list), then the two halves meet.
    u64 k = KSENT;
    unsigned v = VSENT;
    if (owner) {
      const KV r = own_list<SEG>(S, side, half, len, h);
      k = r.k;
      v = r.v;
    }
    if (half == 1) {
      S.lk[wave][lane] = k;
      S.lv[wave][lane] = v;
    }
    __syncthreads();
    if (half == 0) {
      wave_merge64(k, v, S.lk[wave + 1][lane], S.lv[wave + 1][lane]);
      if (owner && !solo && lane < h) {
        unsigned aux = 0;
        u64 ab = 0;
        if (k != KSENT) {
          aux = ws_aux(base + v, S.y[v]);
          ab = (u64)__double_as_longlong(S.a[v]);
        }
        put_cand(P.slots + (par * P.nwg + rank) * WS_LIST_WORDS + (size_t)side * 64 * CAND_WORDS, lane, k, aux, ab,
                 stamp);
      }
    }
    __syncthreads();  // lk/lv are rewritten below
    // ---- 1b. group lists (more than 16 owners): group leaders merge their group's lists
    if (owner && P.g1 > 0 && rank == group_leader(P, rank / P.g1)) {
      const int g = rank / P.g1;
      const int q0 = g * P.g1, q1 = min(P.nwg, q0 + P.g1);
      const KV r = merge_lists<SEG>(P.slots + par * P.nwg * WS_LIST_WORDS, side, q0, q0 + half, q1, 2, h, stamp,
                                    S.u.st.aux[side], S.u.st.ab[side], sp.spin_limit, sp.error, &S.abort_flag);
      k = r.k;
      v = r.v;
      if (half == 1) {
        S.lk[wave][lane] = k;
        S.lv[wave][lane] = v;
      }
      __syncthreads();
      if (half == 0) {
        seg_merge<SEG>(k, v, S.lk[wave + 1][lane], S.lv[wave + 1][lane]);
        if (lane < h) {
          const bool ok = k != KSENT;
          put_cand(P.slots2 + (par * P.ng + g) * WS_LIST_WORDS + (size_t)side * 64 * CAND_WORDS, lane, k,
                   ok ? S.u.st.aux[side][v] : 0u, ok ? S.u.st.ab[side][v] : 0ull, stamp);
        }
      }
      __syncthreads();
    }
    // ---- 1c. the problem's two lists, identical in every workgroup
    if (!solo) {
      const bool two = P.g1 > 0;
      const u64 *words = two ? P.slots2 + par * P.ng * WS_LIST_WORDS : P.slots + par * P.nwg * WS_LIST_WORDS;
      const int nls = two ? P.ng : P.nwg;
      const KV r = merge_lists<SEG>(words, side, 0, half, nls, 2, h, stamp, S.u.st.aux[side], S.u.st.ab[side],
                                    sp.spin_limit, sp.error, &S.abort_flag);
      k = r.k;
      v = r.v;
      if (half == 1) {
        S.lk[wave][lane] = k;
        S.lv[wave][lane] = v;
      }
      __syncthreads();
      if (half == 0) seg_merge<SEG>(k, v, S.lk[wave + 1][lane], S.lv[wave + 1][lane]);
    } else if (half == 0 && k != KSENT) {
      // one workgroup: its own lists are the problem's; stage them like merged candidates
      S.u.st.aux[side][v] = ws_aux(base + v, S.y[v]);
      S.u.st.ab[side][v] = (u64)__double_as_longlong(S.a[v]);
    }
    if (wave == 2) {  // the I_low list, for wave 0
      S.lk[2][lane] = k;
      S.lv[2][lane] = v;
    }
    __syncthreads();
    // ---- 1d. the working set (wave 0): the I_up list, then the I_low list without repeats
    if (wave == 0) {
      const bool ok = lane < h && k != KSENT;
      if (ok) {
        const unsigned aux = S.u.st.aux[0][v];
        S.bi[lane] = (int)(aux & 0x7fffffffu);
        S.by[lane] = (aux >> 31) ? -1 : 1;
        S.bf[lane] = key_f(k);
        S.ba[lane] = __longlong_as_double((long long)S.u.st.ab[0][v]);
      }
      const int nu = __popcll(__ballot(ok));
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      const u64 kl = S.lk[2][lane];
      const unsigned vl = S.lv[2][lane];
      const bool okl = lane < h && kl != KSENT;
      const unsigned aux = okl ? S.u.st.aux[1][vl] : 0u;
      const int idx = okl ? (int)(aux & 0x7fffffffu) : -1;
      // is idx among the first nu entries of the I_up list?  Broadcast LDS reads, four indices
      // a read, over a bound known at compile time (nu <= h <= SEG): no loop, no lane reads.
      bool dup = false;
#pragma unroll
      for (int r = 0; r < SEG; r += 4) {
        if (r < nu) {
          const int4 w = *reinterpret_cast<const int4 *>(&S.bi[r]);
          dup = dup || (w.x == idx) || (r + 1 < nu && w.y == idx) || (r + 2 < nu && w.z == idx) ||
                (r + 3 < nu && w.w == idx);
        }
      }
      const bool keep = okl && !dup;
      const u64 mk = __ballot(keep);
      const int nok = __popcll(__ballot(okl));
      const int pos = nu + __popcll(mk & ((1ull << lane) - 1ull));
      if (keep) {
        S.bi[pos] = idx;
        S.by[pos] = (aux >> 31) ? -1 : 1;
        S.bf[pos] = -key_f(kl);
        S.ba[pos] = __longlong_as_double((long long)S.u.st.ab[1][vl]);
      }
      if (lane == 0) {
        S.nu = nu;
        S.m = nu + __popcll(mk);
        S.nl = nok;
        S.il = okl ? idx : IBIG;
        S.bl = okl ? -key_f(kl) : -INFINITY;
      }
    }
    __syncthreads();
    // ---- 2. stop rule (every workgroup takes the same decision)
    const int nu = S.nu, m = S.m;
    iu = nu > 0 ? S.bi[0] : IBIG;
    b_up = nu > 0 ? S.bf[0] : INFINITY;
    il = S.nl > 0 ? S.il : IBIG;
    b_low = S.nl > 0 ? S.bl : -INFINITY;
    if (rank == 0 && tid == 0 && round < P.trace_len) {
      if (P.trace_ul) {
        P.trace_ul[2 * round] = iu;
        P.trace_ul[2 * round + 1] = il;
      }
      if (P.trace_b) {
        P.trace_b[2 * round] = b_up;
        P.trace_b[2 * round + 1] = b_low;
      }
    }
    if (S.abort_flag) status = ST_TIMEOUT;
    else if (nu == 0 || S.nl == 0 || b_low - b_up <= sp.tol) status = ST_CONVERGED;
    else if (t >= sp.max_iter) status = ST_MAXITER;
    if (status != ST_RUNNING) break;

    // ---- 3. the pair steps on B: K_BB into LDS, then one wave of the solving workgroup.
    // Gram path: the owners fetch K_BB from the Gram between them and publish it, then load the
    // Gram rows of B over their own samples while the pair steps run.  Row path: every owner
    // evaluates K(B, own samples) and publishes the columns of K_BB of its own members of B.
    // The solving workgroup collects K_BB.  On the Gram path the rows of B over the first lcap
    // own samples fit in LDS (over all of them while m len <= WS_QMAX^2); the f update reads the
    // rest of the slice from the Gram.
    const int lcap = !GRAM || m * len <= WS_QMAX * WS_QMAX ? len : (WS_QMAX * WS_QMAX) / m;
    const bool rows_in_lds = GRAM ? owner && !solo : owner;
    const size_t kpar = par * (size_t)(WS_QMAX * WS_QMAX);
    const unsigned kstamp = (unsigned)(round + 1);
    if (tid < m) {
      const int64_t gb = ws_gmap(P, S.bi[tid]);
      if (GRAM) {
        S.roff[tid] = gb * sp.ld;
      } else {
        S.bsc[tid] = gp(p.split.scale)[gb];
        S.bnr[tid] = gp(p.split.nrm)[gb];
      }
    }
    if (!GRAM && owner && wave == 0) {
      const int p0 = lane, p1 = lane + 64;
      const bool o0 = p0 < m && S.bi[p0] >= base && S.bi[p0] < base + len;
      const bool o1 = p1 < m && S.bi[p1] >= base && S.bi[p1] < base + len;
      const u64 m0 = __ballot(o0), m1 = __ballot(o1);
      const u64 below = (1ull << lane) - 1ull;
      if (o0) S.own[__popcll(m0 & below)] = p0;
      if (o1) S.own[__popcll(m0) + __popcll(m1 & below)] = p1;
      const int cnt = __popcll(m0) + __popcll(m1);
      if (lane == 0) S.nown = cnt;
    }
    __syncthreads();
    // Gram path with several owners: the owners fetch K_BB between them (owner r the entries
    // r, r + nwg, ...) and publish it as the row path does, since one workgroup alone can keep
    // only so many scattered reads in flight.
    const bool kdist = GRAM && !solo;
    if (kdist && owner) {
      const int mm = m * m;
      for (int e = rank + tid * P.nwg; e < mm; e += WS_BS * P.nwg) {
        const int ra = e / m, cb = e - ra * m;
        const float kv = gp(sp.gram)[S.roff[ra] + ws_gmap(P, S.bi[cb])];
        st_word(kbuf + kpar + (size_t)ra * WS_QMAX + cb, ((u64)kstamp << 32) | (u64)__float_as_uint(kv));
      }
    }
    if (solver && (!GRAM || kdist)) {
      // wait for every published entry of K_BB, WK_GATHER per thread at a time: each sweep
      // issues all its loads before testing any, so they are in flight together
      constexpr int WK_GATHER = 16;
      const int mm = m * m;
      const int dra = WS_BS / m, dcb = WS_BS - dra * m;  // slot e -> e + WS_BS in (row, column)
      for (int e0 = 0; e0 < mm; e0 += WS_BS * WK_GATHER) {
        int off[WK_GATHER];
        unsigned pending = 0;
        {
          int ra = (e0 + tid) / m, cb = (e0 + tid) - ra * m;
#pragma unroll
          for (int b = 0; b < WK_GATHER; ++b) {
            off[b] = ra * WS_QMAX + cb;
            if (e0 + b * WS_BS + tid < mm) pending |= 1u << b;
            ra += dra;
            cb += dcb;
            if (cb >= m) {
              cb -= m;
              ++ra;
            }
          }
        }
        const uint64_t t0 = wall_clock64();
        while (pending) {
          u64 w[WK_GATHER];
#pragma unroll
          for (int b = 0; b < WK_GATHER; ++b) w[b] = (pending & (1u << b)) ? ld_word(kbuf + kpar + off[b]) : 0ull;
#pragma unroll
          for (int b = 0; b < WK_GATHER; ++b) {
            if ((pending & (1u << b)) && (unsigned)(w[b] >> 32) == kstamp) {
              S.u.K[off[b]] = __uint_as_float((unsigned)w[b]);
              pending &= ~(1u << b);
            }
          }
          if (pending && wall_clock64() - t0 > sp.spin_limit) {
            __hip_atomic_store(sp.error, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            S.abort_flag = 1;
            break;
          }
        }
      }
    }
    if (solver) {
      if (GRAM && !kdist) {
        // one workgroup: K_BB from the Gram; flat indices clamped to the last element, so the
        // loads of a batch issue back to back; only the stores are guarded
        const int mm = m * m;
        for (int e0 = 0; e0 < mm; e0 += WS_BS * WS_GATHER) {
          float kv[WS_GATHER];
#pragma unroll
          for (int b = 0; b < WS_GATHER; ++b) {
            const int e = min(e0 + b * WS_BS + tid, mm - 1);
            const int ra = e / m, cb = e - ra * m;
            kv[b] = gp(sp.gram)[S.roff[ra] + ws_gmap(P, S.bi[cb])];
          }
#pragma unroll
          for (int b = 0; b < WS_GATHER; ++b) {
            const int e = e0 + b * WS_BS + tid;
            if (e < mm) {
              const int ra = e / m, cb = e - ra * m;
              S.u.K[ra * WS_QMAX + cb] = kv[b];
            }
          }
        }
      }
      __syncthreads();
      if (wave == 0) {
        if (m <= 32)
          local_solve_halves(S, sp.C, sp.tol, p.frac, p.max_inner, sp.max_iter, m, b_up, b_low, t);
        else if (m <= 64)
          local_solve<64>(S, sp.C, sp.tol, p.frac, p.max_inner, sp.max_iter, m, b_up, b_low, t);
        else
          local_solve<WS_QMAX>(S, sp.C, sp.tol, p.frac, p.max_inner, sp.max_iter, m, b_up, b_low, t);
      }
      __syncthreads();
      if (!solo) {
        // publish the new multipliers (two words each) and the step count
        // every entry is rewritten each round (zero past m): a word left from 16 rounds earlier
        // would carry the same 4-bit stamp
        u64 *bw = bcast + par * WS_BCAST_PITCH;
        const u64 sw = (u64)(stamp & 15u) << 60;
        if (tid < WS_QMAX) {
          const u64 b = tid < m ? (u64)__double_as_longlong(S.bn[tid]) : 0ull;
          st_word(bw + 1 + 2 * tid, sw | (b & 0xffffffffull));
          st_word(bw + 2 + 2 * tid, sw | (b >> 32));
        }
        if (tid == WS_BS - 1) st_word(bw, sw | (u64)S.steps);
      }
    } else {
      if (!GRAM) {
        // row path: K(B, own samples) into LDS, then the columns of K_BB of the own members
        if (len <= 128)
          owner_rows_block(S, p.split, p.cexp, GMap{P.off0, P.len0, P.off1}, m, base, len);
        else
          owner_rows(S, p.split, p.cexp, GMap{P.off0, P.len0, P.off1}, m, base, len);
        const int nk = S.nown * m;
        for (int e = tid; e < nk; e += WS_BS) {
          const int kk = e / m, a = e - kk * m;
          const int pb = S.own[kk];
          const float kv = S.u.K[a * len + (int)(S.bi[pb] - base)];
          st_word(kbuf + kpar + (size_t)a * WS_QMAX + pb, ((u64)kstamp << 32) | (u64)__float_as_uint(kv));
        }
      }
      // owners: the Gram rows of B over the own samples into LDS while the pair steps run
      if (GRAM && rows_in_lds) {
        const int ml = m * lcap;
        for (int e0 = 0; e0 < ml; e0 += WS_BS * WS_GATHER) {
          float kv[WS_GATHER];
#pragma unroll
          for (int b = 0; b < WS_GATHER; ++b) {
            const int e = min(e0 + b * WS_BS + tid, ml - 1);
            const int ra = e / lcap, pos = e - ra * lcap;
            kv[b] = gp(sp.gram)[S.roff[ra] + ws_gmap(P, base + pos)];
          }
#pragma unroll
          for (int b = 0; b < WS_GATHER; ++b) {
            const int e = e0 + b * WS_BS + tid;
            if (e < ml) S.u.K[e] = kv[b];
          }
        }
      }
      const u64 *bw = bcast + par * WS_BCAST_PITCH;
      if (tid < m) {
        u64 lo, hi;
        poll_word2(bw + 1 + 2 * tid, bw + 2 + 2 * tid, stamp, sp.spin_limit, sp.error, &S.abort_flag, lo, hi);
        S.bn[tid] = __longlong_as_double((long long)((hi << 32) | lo));
      }
      if (tid == WS_BS - 1) S.steps = (int64_t)poll_word(bw, stamp, sp.spin_limit, sp.error, &S.abort_flag);
      __syncthreads();
    }
    t += S.steps;
    // ---- 4. owners: changes of a y in B's order, new multipliers of the own members of B,
    // and f_j += ((s0 + s1) + s2) + s3, s_g the sum over the g-th quarter of the changes: a
    // fixed grouping, so the bits do not depend on how many workgroups share the samples.
    if (owner) {
      if (wave == 0) {
        const int p0 = lane, p1 = lane + 64;
        const bool v0 = p0 < m, v1 = p1 < m;
        const double c0 = v0 ? (S.bn[p0] - S.ba[p0]) * (double)S.by[p0] : 0.0;
        const double c1 = v1 ? (S.bn[p1] - S.ba[p1]) * (double)S.by[p1] : 0.0;
        const u64 m0 = __ballot(v0 && c0 != 0.0), m1 = __ballot(v1 && c1 != 0.0);
        const u64 below = (1ull << lane) - 1ull;
        if (v0 && c0 != 0.0) {
          const int r = __popcll(m0 & below);
          S.nzp[r] = p0;
          S.nzoff[r] = S.roff[p0];
          S.nzc[r] = c0;
        }
        if (v1 && c1 != 0.0) {
          const int r = __popcll(m0) + __popcll(m1 & below);
          S.nzp[r] = p1;
          S.nzoff[r] = S.roff[p1];
          S.nzc[r] = c1;
        }
        const int nnz = __popcll(m0) + __popcll(m1);
        if (lane == 0) S.nnz = nnz;
      }
      // the new multipliers of the own members of B, before the barrier: the keys written with
      // the new f below read them
      for (int q = tid; q < m; q += WS_BS) {
        const int64_t j = S.bi[q] - base;
        if (j >= 0 && j < len) S.a[j] = S.bn[q];
      }
      __syncthreads();
      // threads as (sample, quarters): span samples by 256 / span thread groups, span a power
      // of two that divides the workgroup, so every thread's group is below ngrp
      const int nnz = S.nnz;
      const int span = len <= 64 ? 64 : (len <= 128 ? 128 : WS_BS);
      const int ngrp = WS_BS / span;  // 4, 2 or 1 thread groups
      const int grp = tid / span;
      const int g0 = grp * (WS_QUARTERS / ngrp), g1 = g0 + WS_QUARTERS / ngrp;
      const int qlen = nnz - (WS_QUARTERS - 1) * nnz / WS_QUARTERS;  // the longest quarter (the last)
      // The terms of the quarter chains as lane registers of every wave: term i of quarter g
      // (change c and row offset in S.u.K) in lane (g QL + i) mod 64 of register (g QL) / 64,
      // QL = SEG / 2 >= the longest quarter (m <= 2 SEG).  A term past its quarter's end is
      // (0, row 0): it adds 0 * K = +0, which leaves the sum unchanged (a sum that starts at +0
      // and adds products never becomes -0).  The loops read the terms with lane reads, so only
      // the rows come from LDS and no row read waits on another LDS read.
      constexpr int QL = SEG / 2, NSR = (WS_QUARTERS * QL + 63) / 64;
      double tc[NSR];
      int to[NSR];
#pragma unroll
      for (int r = 0; r < NSR; ++r) {
        const int sl = r * 64 + lane, g = sl / QL, i = sl - g * QL;
        const int idx = g * nnz / WS_QUARTERS + i;
        const bool in = g < WS_QUARTERS && idx < (g + 1) * nnz / WS_QUARTERS;
        const int ic = in ? idx : 0;
        tc[r] = in ? S.nzc[ic] : 0.0;
        to[r] = in ? S.nzp[ic] * lcap : 0;
      }
      if (ngrp == 1 && rows_in_lds) {
        // every thread sums all four quarters of two of its samples in registers: the eight
        // chains advance together, each in its own order, so the sums are those written
        for (int pa = tid; pa < lcap; pa += 2 * WS_BS) {
          const int pb = pa + WS_BS;
          const bool hb = pb < lcap;
          double qa[WS_QUARTERS], qb[WS_QUARTERS];
#pragma unroll
          for (int g = 0; g < WS_QUARTERS; ++g) qa[g] = qb[g] = 0.0;
          // no branch inside, so the row reads of the four quarters are issued together
          const int pbx = hb ? pb : pa;
          // two terms of each chain a batch (QL is even and at least qlen, so a batch stays inside
          // the quarters' slots; terms past a quarter's end are (0, row 0))
          for (int i0 = 0; i0 < qlen; i0 += 2) {
            double c[2][WS_QUARTERS];
            float ka[2][WS_QUARTERS], kb[2][WS_QUARTERS];
#pragma unroll
            for (int d = 0; d < 2; ++d)
#pragma unroll
              for (int g = 0; g < WS_QUARTERS; ++g) {
                const int sl = (g * QL) % 64 + i0 + d;
                c[d][g] = readlane_d(tc[(g * QL) / 64], sl);
                const float *row = S.u.K + __builtin_amdgcn_readlane(to[(g * QL) / 64], sl);
                ka[d][g] = row[pa];
                kb[d][g] = row[pbx];
              }
            // compiler barrier: the reads of the batch are issued before the first is used (left
            // to itself the scheduler waits for each read before issuing the next)
            __asm__ volatile("" ::: "memory");
#pragma unroll
            for (int d = 0; d < 2; ++d)
#pragma unroll
              for (int g = 0; g < WS_QUARTERS; ++g) {
                qa[g] = ws_acc(qa[g], c[d][g], ka[d][g]);
                qb[g] = ws_acc(qb[g], c[d][g], kb[d][g]);
              }
          }
          const double fa = S.f[pa] + (((qa[0] + qa[1]) + qa[2]) + qa[3]);
          S.f[pa] = fa;
          put_keys(S, pa, fa, S.a[pa], S.y[pa], C);
          if (hb) {
            const double fb = S.f[pb] + (((qb[0] + qb[1]) + qb[2]) + qb[3]);
            S.f[pb] = fb;
            put_keys(S, pb, fb, S.a[pb], S.y[pb], C);
          }
        }
        // the samples past lcap: the same four chains with the rows read from the Gram (term
        // slots as above, with the Gram row offset; 0, the first row, past a quarter's end),
        // eight terms of each a batch, all 32 reads issued before the first is used (QL is a
        // multiple of eight and at least qlen, so a batch stays inside the quarters' slots)
        if (lcap < len) {
          int64_t tg[NSR];
#pragma unroll
          for (int r = 0; r < NSR; ++r) {
            const int sl = r * 64 + lane, g = sl / QL, i = sl - g * QL;
            const int idx = g * nnz / WS_QUARTERS + i;
            const bool in = g < WS_QUARTERS && idx < (g + 1) * nnz / WS_QUARTERS;
            tg[r] = in ? S.nzoff[in ? idx : 0] : 0;
          }
          for (int pos = lcap + tid; pos < len; pos += WS_BS) {
            const int64_t gj = ws_gmap(P, base + pos);
            double qs[WS_QUARTERS];
#pragma unroll
            for (int g = 0; g < WS_QUARTERS; ++g) qs[g] = 0.0;
            for (int i0 = 0; i0 < qlen; i0 += 8) {
              double c[8][WS_QUARTERS];
              float kk[8][WS_QUARTERS];
#pragma unroll
              for (int d = 0; d < 8; ++d)
#pragma unroll
                for (int g = 0; g < WS_QUARTERS; ++g) {
                  const int sl = (g * QL) % 64 + i0 + d;
                  c[d][g] = readlane_d(tc[(g * QL) / 64], sl);
                  const int64_t ro = (int64_t)readlane64((u64)tg[(g * QL) / 64], sl);
                  kk[d][g] = gp(sp.gram)[ro + gj];
                }
              __asm__ volatile("" ::: "memory");
#pragma unroll
              for (int d = 0; d < 8; ++d)
#pragma unroll
                for (int g = 0; g < WS_QUARTERS; ++g) qs[g] = ws_acc(qs[g], c[d][g], kk[d][g]);
            }
            const double fp = S.f[pos] + (((qs[0] + qs[1]) + qs[2]) + qs[3]);
            S.f[pos] = fp;
            put_keys(S, pos, fp, S.a[pos], S.y[pos], C);
          }
        }
      } else if (rows_in_lds) {
        // each thread its one or two quarters (g0, g0 + 1) of one sample, the chains together
        // g0 is the same in the whole wave (span >= 64); quarter g0 + 1 only with two of them
        const int la = (g0 + 1) * nnz / WS_QUARTERS - g0 * nnz / WS_QUARTERS;
        const int lb = g1 - g0 == 2 ? (g0 + 2) * nnz / WS_QUARTERS - (g0 + 1) * nnz / WS_QUARTERS : 0;
        const int lm = max(la, lb);
        const int la0 = __builtin_amdgcn_readfirstlane(g0 * QL), lb0 = la0 + QL;
        auto term = [&](int sl, double &c, int &o) {  // slot sl < 4 QL, the same in the wave
          if (NSR == 1 || sl < 64) {
            c = readlane_d(tc[0], sl & 63);
            o = __builtin_amdgcn_readlane(to[0], sl & 63);
          } else {
            c = readlane_d(tc[NSR - 1], sl & 63);
            o = __builtin_amdgcn_readlane(to[NSR - 1], sl & 63);
          }
        };
        for (int pos = tid - grp * span; pos < len; pos += WS_BS) {
          double sa = 0.0, sb = 0.0;
          // four terms of each chain a batch (QL is a multiple of four, so a batch stays inside
          // its quarter's slots; terms past the quarter's end are (0, row 0))
          for (int i0 = 0; i0 < lm; i0 += 4) {
            double ca[4], cb[4];
            float ka[4], kb[4];
#pragma unroll
            for (int d = 0; d < 4; ++d) {
              int oa, ob = 0;
              term(la0 + i0 + d, ca[d], oa);
              cb[d] = 0.0;
              if (lb > 0) term(lb0 + i0 + d, cb[d], ob);
              ka[d] = S.u.K[oa + pos];
              kb[d] = S.u.K[ob + pos];
            }
            __asm__ volatile("" ::: "memory");  // the reads of the batch are issued together
#pragma unroll
            for (int d = 0; d < 4; ++d) {
              sa = ws_acc(sa, ca[d], ka[d]);
              sb = ws_acc(sb, cb[d], kb[d]);
            }
          }
          S.w.part[g0][pos] = sa;
          if (g1 - g0 == 2) S.w.part[g0 + 1][pos] = sb;
        }
        __syncthreads();
        for (int pos = tid; pos < len; pos += WS_BS) {
          const double s = ((S.w.part[0][pos] + S.w.part[1][pos]) + S.w.part[2][pos]) + S.w.part[3][pos];
          const double fp = S.f[pos] + s;
          S.f[pos] = fp;
          put_keys(S, pos, fp, S.a[pos], S.y[pos], C);
        }
      } else {
      // one workgroup alone (LDS holds K_BB): the rows of B read from the Gram
      for (int pos = tid - grp * span; pos < len; pos += WS_BS) {
        const int64_t gj = ws_gmap(P, base + pos);
        for (int g = g0; g < g1; ++g) {
          const int r0 = g * nnz / WS_QUARTERS, r1 = (g + 1) * nnz / WS_QUARTERS;
          double s = 0.0;
          for (int r = r0; r < r1; r += WS_GATHER) {
            float kk[WS_GATHER];
#pragma unroll
            for (int e = 0; e < WS_GATHER; ++e) kk[e] = gp(sp.gram)[S.nzoff[min(r + e, r1 - 1)] + gj];
#pragma unroll
            for (int e = 0; e < WS_GATHER; ++e)
              if (r + e < r1) s = ws_acc(s, S.nzc[r + e], kk[e]);
          }
          S.w.part[g][pos] = s;
        }
      }
      __syncthreads();
      for (int pos = tid; pos < len; pos += WS_BS) {
        const double s = ((S.w.part[0][pos] + S.w.part[1][pos]) + S.w.part[2][pos]) + S.w.part[3][pos];
        const double fp = S.f[pos] + s;
        S.f[pos] = fp;
        put_keys(S, pos, fp, S.a[pos], S.y[pos], C);
      }
      }
    }
    ++round;
    __syncthreads();
    if (S.abort_flag) {
      status = ST_TIMEOUT;
      break;
    }
    if (t >= t_end || round >= p.round_end) break;  // launch budget spent: the state is whole at a round boundary
  }

  for (int j = tid; j < len; j += WS_BS) {
    gp(P.f)[base + j] = S.f[j];
    gp(P.alpha)[base + j] = S.a[j];
  }
  if (rank == 0 && tid == 0) {
    ctl->t = t;
    ctl->status = status;
    ctl->b_up = b_up;
    ctl->b_low = b_low;
    ctl->u = iu;
    ctl->l = il;
    p.rounds[pid] = round;
  }
}

hipError_t launch_ws_solver(const WsParams &p, int32_t total_wg, hipStream_t s, int32_t *max_coresident) {
  // lists merge in segments of 16, 32 or 64 entries (the smallest that holds q / 2)
  const int h = p.q / 2;
  const void *fn;
  if (h <= 16)
    fn = p.sp.gram ? reinterpret_cast<const void *>(&ws_solve<true, 16>)
                   : reinterpret_cast<const void *>(&ws_solve<false, 16>);
  else if (h <= 32)
    fn = p.sp.gram ? reinterpret_cast<const void *>(&ws_solve<true, 32>)
                   : reinterpret_cast<const void *>(&ws_solve<false, 32>);
  else
    fn = p.sp.gram ? reinterpret_cast<const void *>(&ws_solve<true, 64>)
                   : reinterpret_cast<const void *>(&ws_solve<false, 64>);
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, WS_BS, 0);
  if (e != hipSuccess) return e;
  if (max_coresident) *max_coresident = per_cu * cus;
  if (total_wg <= 0) return hipSuccess;
  if ((int64_t)total_wg > (int64_t)per_cu * cus) return hipErrorCooperativeLaunchTooLarge;
  WsParams pp = p;
  void *args[] = {&pp};
  return hipLaunchCooperativeKernel(fn, dim3((unsigned)total_wg), dim3(WS_BS), args, 0, s);
}

}  // namespace svmx

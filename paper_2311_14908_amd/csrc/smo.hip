// smo.hip -- persistent SMO solver for gfx950 (paper, Section III.B: SMO with two Lagrange
// multipliers per step; the data-parallel work runs one thread per training sample).
//
// One cooperative launch advances every running problem by up to `steps` SMO steps.  A
// problem is served by nwg workgroups; workgroup r owns local samples [r*per_wg,
// (r+1)*per_wg) and keeps their f, alpha and label in registers for the whole launch.
// Each step:
//   1. every workgroup selects its own candidates  u_r = argmin_{I_up} f,  l_r = argmax_{I_low} f
//      (ties to the smaller index) with DPP wave reductions and one LDS hand-off;
//   2. the nwg partial results are exchanged through global memory as records of six
//      self-stamped 64-bit words (step stamp | payload, xchg_record.hpp), so no fence or cache
//      flush is needed: a reader simply waits until every word it needs carries the current
//      stamp.  With one level every
//      workgroup polls all records, one record per lane over as many waves as needed; with
//      two levels (the default above 128 workgroups) group leaders reduce about sqrt(nwg)
//      records each and publish a group record, and every workgroup then reads the group
//      records;
//   3. every workgroup reduces the same nwg records to the same pair (u, l), tests the stop
//      rule, and solves the 2x2 sub-problem redundantly (identical fp64 arithmetic);
//   4. every workgroup fetches K(u, j) and K(l, j) for its own samples -- from the Gram, or
//      computed from X as a GEMV against x_u and x_l with the squared row norms, the first
//      rows of its slice of X held in LDS for the whole launch -- and applies
//      f_j += da_u y_u K_uj + da_l y_l K_lj.
// Every wait is bounded by a wall-clock limit; on expiry the kernel records an error and
// all waits end, so a launch always drains.
#include "common.hpp"
#include "rbf_rows.hpp"
#include "pair_step.hpp"
#include "xchg_record.hpp"

#include <math.h>

namespace svmx {

// Gram path: 256-thread workgroups, up to 16 samples per thread.  Row path: 512-thread
// workgroups, one per CU (8 waves, each with a batch of samples x the lane's loads in flight,
// keep the streaming of X busy without spilling), up to 8 samples per thread.
constexpr int BS_GRAM = 256, MAXP_GRAM = 16;
constexpr int BS_ROWS = 512, MAXP_ROWS = 8;
constexpr int ROW_BATCH = 2;   // samples per lane group and batch of rows read from LDS
constexpr int ROW_SBATCH = 2;  // samples per lane group and batch of rows streamed from HBM
constexpr int ROW_MAXM = ROW_POSITIONS;  // feature positions per lane whose loads are issued together

int solver_block_size(bool gram) { return gram ? BS_GRAM : BS_ROWS; }
int max_per_thread(bool gram) { return gram ? MAXP_GRAM : MAXP_ROWS; }


// Candidates of one selection: min f over I_up (vu at index iu) and max f over I_low (vl at
// il), each with the multiplier and label of its sample.
struct Sel {
  double vu, au, vl, al;
  int iu, yu, il, yl;
};

__device__ __forceinline__ void sel_init(Sel &s) {
  s.vu = INFINITY; s.au = 0.0; s.iu = IBIG; s.yu = 0;
  s.vl = -INFINITY; s.al = 0.0; s.il = IBIG; s.yl = 0;
}

__device__ __forceinline__ void sel_merge(Sel &s, const Sel &o) {
  if (lt_min(o.vu, o.iu, s.vu, s.iu)) { s.vu = o.vu; s.iu = o.iu; s.au = o.au; s.yu = o.yu; }
  if (gt_max(o.vl, o.il, s.vl, s.il)) { s.vl = o.vl; s.il = o.il; s.al = o.al; s.yl = o.yl; }
}

// Wave-wide selection, returned to every lane.  Must be called by all 64 lanes of the wave.
// Each side's winner: its extreme value, then the smallest index among the lanes holding it
// (the (value, index) lexicographic order; -0 and +0 compare equal), with value, index,
// multiplier and label read from that lane.  The two sides' reductions run interleaved.
__device__ __forceinline__ Sel sel_wave(const Sel &mine) {
  double ru = mine.vu, rl = mine.vl;
  wave_minmax(ru, rl);
  const int lu = tie_lane(mine.vu == ru, mine.iu), ll = tie_lane(mine.vl == rl, mine.il);
  Sel r;
  r.vu = readlane_d(mine.vu, lu);  // the winner's own value (its sign of zero included)
  r.iu = __builtin_amdgcn_readlane(mine.iu, lu);
  r.au = readlane_d(mine.au, lu);
  r.yu = __builtin_amdgcn_readlane(mine.yu, lu);
  r.vl = readlane_d(mine.vl, ll);
  r.il = __builtin_amdgcn_readlane(mine.il, ll);
  r.al = readlane_d(mine.al, ll);
  r.yl = __builtin_amdgcn_readlane(mine.yl, ll);
  return r;
}

// Candidate of the second-order choice of l (used with p.second_order): the largest gain
// g = (f_t - b_up)^2 / a_ut over the members t of I_low above b_up (ties to the smaller index),
// with f, multiplier, label and K(u, t) of that sample.
struct Sel2 {
  double g, fl, al, kul;
  int il, yl;
};

__device__ __forceinline__ void rec_init(Sel &s) { sel_init(s); }
__device__ __forceinline__ void rec_init(Sel2 &s) {
  s.g = -INFINITY; s.fl = 0.0; s.al = 0.0; s.kul = 0.0; s.il = IBIG; s.yl = 0;
}
__device__ __forceinline__ void rec_merge(Sel &s, const Sel &o) { sel_merge(s, o); }
__device__ __forceinline__ void rec_merge(Sel2 &s, const Sel2 &o) {
  if (gt_max(o.g, o.il, s.g, s.il)) s = o;
}
__device__ __forceinline__ Sel rec_wave(const Sel &mine) { return sel_wave(mine); }
__device__ __forceinline__ Sel2 rec_wave(const Sel2 &mine) {
  const int lane = winner_lane<true>(mine.g, mine.il);
  Sel2 r;
  r.g = readlane_d(mine.g, lane);
  r.fl = readlane_d(mine.fl, lane);
  r.al = readlane_d(mine.al, lane);
  r.kul = readlane_d(mine.kul, lane);
  r.il = __builtin_amdgcn_readlane(mine.il, lane);
  r.yl = __builtin_amdgcn_readlane(mine.yl, lane);
  return r;
}

// LDS hand-off between the waves of a workgroup.  Two buffers used alternately, so one
// barrier per hand-off suffices: a buffer is rewritten only after another hand-off's barrier.
template <class R, int NW>
struct RecLds {
  R slot[2][NW];
};

// Combine the wave results of all waves; every thread returns the same workgroup result.
template <class R, int NW>
__device__ __forceinline__ R rec_block(const R &wave_res, RecLds<R, NW> &L, int &buf) {
  if ((threadIdx.x & 63) == 0) L.slot[buf][threadIdx.x >> 6] = wave_res;
  __syncthreads();
  R r = L.slot[buf][0];
#pragma unroll
  for (int q = 1; q < NW; ++q) rec_merge(r, L.slot[buf][q]);
  buf ^= 1;
  return r;
}

__device__ __forceinline__ unsigned pack_index(int i, int y) { return (unsigned)i | (y < 0 ? 0x80000000u : 0u); }
__device__ __forceinline__ void unpack_index(unsigned w, int &i, int &y) {
  i = (int)(w & 0x7fffffffu);
  y = (w >> 31) ? -1 : 1;
}

// Limbs of a record (xchg_record.hpp): v_up, a_up, index words, v_low, a_low; the label travels
// in bit 31 of the index word.
__device__ __forceinline__ void rec_limbs_of(const Sel &s, u64 (&L)[5]) {
  L[0] = (u64)__double_as_longlong(s.vu);
  L[1] = (u64)__double_as_longlong(s.au);
  L[2] = (u64)pack_index(s.iu, s.yu) | ((u64)pack_index(s.il, s.yl) << 32);
  L[3] = (u64)__double_as_longlong(s.vl);
  L[4] = (u64)__double_as_longlong(s.al);
}
__device__ __forceinline__ void rec_from_limbs(const u64 (&L)[5], Sel &o) {
  o.vu = __longlong_as_double((long long)L[0]);
  o.au = __longlong_as_double((long long)L[1]);
  unpack_index((unsigned)L[2], o.iu, o.yu);
  unpack_index((unsigned)(L[2] >> 32), o.il, o.yl);
  o.vl = __longlong_as_double((long long)L[3]);
  o.al = __longlong_as_double((long long)L[4]);
}
// Second-order record: gain, f_l, index word, a_l, K(u, l).
__device__ __forceinline__ void rec_limbs_of(const Sel2 &s, u64 (&L)[5]) {
  L[0] = (u64)__double_as_longlong(s.g);
  L[1] = (u64)__double_as_longlong(s.fl);
  L[2] = (u64)pack_index(s.il, s.yl);
  L[3] = (u64)__double_as_longlong(s.al);
  L[4] = (u64)__double_as_longlong(s.kul);
}
__device__ __forceinline__ void rec_from_limbs(const u64 (&L)[5], Sel2 &o) {
  o.g = __longlong_as_double((long long)L[0]);
  o.fl = __longlong_as_double((long long)L[1]);
  unpack_index((unsigned)L[2], o.il, o.yl);
  o.al = __longlong_as_double((long long)L[3]);
  o.kul = __longlong_as_double((long long)L[4]);
}

// Lanes 0..REC_WORDS-1 of the calling wave each write one word of the record.
template <class R>
__device__ __forceinline__ void put_record(u64 *rec, unsigned stamp, const R &s) {
  const int t = threadIdx.x & 63;
  if (t < REC_WORDS) {
    u64 L[5];
    rec_limbs_of(s, L);
    st_word(rec + t, rec_word(L, t, stamp));
  }
}

// Wave-level: wait for records q0 + lane, q0 + lane + stride, ... below q1 of `words` to carry
// `stamp`, reduce them, and return the result to every lane of the wave (all 64 lanes must
// call).
template <class R>
__device__ R poll_reduce(const u64 *words, int q0, int q1, int stride, unsigned stamp, uint64_t spin_limit,
                         int32_t *err, int *abort_flag) {
  R s;
  rec_init(s);
  for (int q = q0 + (int)(threadIdx.x & 63); q < q1; q += stride) {
    const u64 *rec = words + (size_t)q * SLOT_WORDS;
    u64 w[REC_WORDS];
    const uint64_t t0 = wall_clock64();
    for (;;) {
      bool ok = true;
#pragma unroll
      for (int k = 0; k < REC_WORDS; ++k) {
        w[k] = ld_word(rec + k);
        ok = ok && rec_stamped(w[k], stamp);
      }
      if (ok) break;
      if (wall_clock64() - t0 > spin_limit) {
        __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *abort_flag = 1;
        break;
      }
    }
    u64 L[5];
    rec_limbs(w, L);
    R o;
    rec_from_limbs(L, o);
    rec_merge(s, o);
  }
  return rec_wave(s);
}

// Exchange of the workgroup results of one problem (see file comment, item 2).  Wave 0
// publishes the record.  With one level, the records are polled by as many waves as needed
// for one record per lane (wave w takes records w*64 + lane, then every 64*pollers-th), each
// wave reduces its share, and the shares meet in LDS.  With two levels, wave 0 does the
// global-memory work of both levels.  The stamp's parity selects the buffer.
template <class R, int NW>
__device__ R exchange(const Prob &P, int rank, unsigned stamp, const R &mine, RecLds<R, NW> &L, int &buf,
                      uint64_t spin_limit, int32_t *err, int *abort_flag) {
  const size_t par = stamp & 1u;
  u64 *lv1 = P.slots + par * (size_t)P.nwg * SLOT_WORDS;
  const int wave = threadIdx.x >> 6;
  int pollers = 1;
  if (wave == 0) put_record(lv1 + (size_t)rank * SLOT_WORDS, stamp, mine);
  if (P.g1 > 0) {
    if (wave == 0) {
      u64 *lv2 = P.slots2 + par * (size_t)P.ng * SLOT_WORDS;
      const int g = rank / P.g1;
      if (rank == group_leader(P, g)) {
        const int q0 = g * P.g1, q1 = min(P.nwg, q0 + P.g1);
        const R gs = poll_reduce<R>(lv1, q0, q1, 64, stamp, spin_limit, err, abort_flag);
        put_record(lv2 + (size_t)g * SLOT_WORDS, stamp, gs);
      }
      const R s = poll_reduce<R>(lv2, 0, P.ng, 64, stamp, spin_limit, err, abort_flag);
      if (threadIdx.x == 0) L.slot[buf][0] = s;
    }
  } else {
    pollers = min(NW, (P.nwg + 63) >> 6);
    if (wave < pollers) {
      const R s = poll_reduce<R>(lv1, wave * 64, P.nwg, 64 * pollers, stamp, spin_limit, err, abort_flag);
      if ((threadIdx.x & 63) == 0) L.slot[buf][wave] = s;
    }
  }
  __syncthreads();
  R r = L.slot[buf][0];
  for (int q = 1; q < pollers; ++q) rec_merge(r, L.slot[buf][q]);
  buf ^= 1;
  return r;
}

__device__ __forceinline__ int64_t gmap(const Prob &P, int64_t j) { return j < P.len0 ? P.off0 + j : P.off1 + (j - P.len0); }
__device__ __forceinline__ int label_of(const Prob &P, int64_t j) {
  return P.y ? gp(P.y)[gmap(P, j)] : (j < P.len0 ? 1 : -1);
}

// Gain of the second-order rule for a member t of I_low above b_up: (f_t - b_up)^2 / a_ut with
// a_ut = K_uu + K_tt - 2 K_ut, K_uu = K_tt = 1 for the RBF kernel, 1e-12 when not positive.
// Rounded as written (no contraction).
__device__ __forceinline__ double so_gain(double ft, double bup, float kut) {
#pragma clang fp contract(off)
  const double bt = ft - bup;
  double at = (1.0 + 1.0) - 2.0 * (double)kut;
  if (at <= 0.0) at = 1e-12;
  return bt * bt / at;
}

// Offer sample j (value f, multiplier a, label y) to this thread's candidates.
__device__ __forceinline__ void consider(Sel &s, double f, double a, int y, int j, double C) {
  const bool up = (y > 0 && a < C) || (y < 0 && a > 0.0);
  const bool lo = (y > 0 && a > 0.0) || (y < 0 && a < C);
  if (up && lt_min(f, j, s.vu, s.iu)) { s.vu = f; s.iu = j; s.au = a; s.yu = y; }
  if (lo && gt_max(f, j, s.vl, s.il)) { s.vl = f; s.il = j; s.al = a; s.yl = y; }
}

// ---------------------------------------------------------------------------------------
// SO (Gram path): the second index of the pair by the second-order rule (p.second_order).
template <int BS, int PER, bool GRAM, bool VEC4, bool ONE = false, bool SO = false>
__global__ void __launch_bounds__(BS) smo_solve(SolveParams p) {
  constexpr int NW = BS / 64;
  // Samples per lane group and batch (a sample's arithmetic does not depend on them): scalar
  // lanes hold a quarter of the registers per sample, so they take twice as many; ONE: one at
  // a time (row_batch_one).
  constexpr int SB = ONE ? 1 : VEC4 ? ROW_BATCH : 2 * ROW_BATCH;
  // Row path, dynamic LDS: dot products against x_u and x_l [2][per_wg] (fp64), cache tags
  // [cap], then the rows of X this workgroup keeps resident [res][d] (16-byte aligned).
  extern __shared__ float4 dyn4[];
  __shared__ RecLds<Sel, NW> sh;
  __shared__ RecLds<Sel2, NW> sh2;
  __shared__ int s_abort;
  __shared__ double s_kul;
  int buf = 0, buf2 = 0;

  const int32_t pid = p.wg_prob[blockIdx.x];
  const Prob P = p.probs[pid];
  const int rank = (int)blockIdx.x - P.wg0;
  Ctl *ctl = P.ctl;
  if (ctl->status != ST_RUNNING) return;
  int64_t t = ctl->t;
  if (threadIdx.x == 0) s_abort = 0;

  const int64_t base = (int64_t)rank * P.per_wg;
  const int64_t lim = min(base + (int64_t)P.per_wg, P.n);
  double f[PER], a[PER];
  int yv[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int64_t j = base + threadIdx.x + (int64_t)k * BS;
    if (j < lim) {
      f[k] = gp(P.f)[j];
      a[k] = gp(P.alpha)[j];
      yv[k] = label_of(P, j);
    } else {
      f[k] = 0.0;
      a[k] = 0.0;
      yv[k] = 0;
    }
  }

  double *dotu = reinterpret_cast<double *>(dyn4), *dotl = dotu + P.per_wg;
  int *tags = reinterpret_cast<int *>(dotl + P.per_wg);
  float *xres = reinterpret_cast<float *>(dyn4 + ((16 * (int64_t)P.per_wg + 4 * (int64_t)p.cache_cap + 15) >> 4));
  const bool use_cache = !GRAM && p.cache != nullptr && p.cache_cap > 0;
  // Resident rows: the first `res` samples of the slice, copied once per launch; every step
  // reads them from LDS instead of HBM.
  const int64_t res = GRAM ? 0 : min<int64_t>(p.res_rows, max<int64_t>(0, lim - base));
  double sq[PER];  // squared norms of the own samples (row path)
  if (!GRAM) {
    if (use_cache) {
      for (int s = threadIdx.x; s < p.cache_cap; s += BS) tags[s] = gp(p.cache_tags)[(size_t)blockIdx.x * p.cache_cap + s];
    }
    typedef typename Lane<VEC4>::T T;
    const int64_t units = VEC4 ? (p.d >> 2) : p.d;
    T *xr = reinterpret_cast<T *>(xres);
    for (int64_t e = threadIdx.x; e < res * units; e += BS) {
      const int64_t r = e / units, k = e - r * units;
      xr[e] = gp(reinterpret_cast<const T *>(p.X + gmap(P, base + r) * p.d))[k];
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int64_t j = base + threadIdx.x + (int64_t)k * BS;
      sq[k] = j < lim ? gp(p.sqn)[gmap(P, j)] : 0.0;
    }
  }
  __syncthreads();

  const double C = p.C;
  const int64_t t_end = min(t + p.steps, p.max_iter);
  // Candidates of this thread's samples; after the first scan they are gathered in the same
  // pass as the f update of the previous step.
  Sel s;
  sel_init(s);
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int64_t j = base + threadIdx.x + (int64_t)k * BS;
    if (j < lim) consider(s, f[k], a[k], yv[k], (int)j, C);
  }
  for (;;) {
    // 1. workgroup candidates
    s = rec_block<Sel, NW>(rec_wave(s), sh, buf);
    // 2. exchange across the problem's workgroups (with the second-order rule every step has two
    // exchanges, stamped 2t + 1 and 2t + 2)
    const unsigned stamp1 = SO ? (unsigned)(2 * t + 1) : (unsigned)(t + 1);
    if (P.nwg > 1) s = exchange<Sel, NW>(P, rank, stamp1, s, sh, buf, p.spin_limit, p.error, &s_abort);
    const bool aborted = s_abort != 0;
    // 3. stop rule
    if (rank == 0 && threadIdx.x == 0 && t < P.trace_len) {
      if (P.trace_ul) { P.trace_ul[2 * t] = s.iu; P.trace_ul[2 * t + 1] = s.il; }
      if (P.trace_b) { P.trace_b[2 * t] = s.vu; P.trace_b[2 * t + 1] = s.vl; }
    }
    int status = ST_RUNNING;
    if (aborted) status = ST_TIMEOUT;
    else if (s.iu == IBIG || s.il == IBIG || s.vl - s.vu <= p.tol) status = ST_CONVERGED;
    else if (t >= p.max_iter) status = ST_MAXITER;
    if (status != ST_RUNNING || t >= t_end) {
      if (rank == 0 && threadIdx.x == 0) {
        ctl->t = t;
        ctl->status = status;
        ctl->b_up = s.vu;
        ctl->b_low = s.vl;
        ctl->u = s.iu;
        ctl->l = s.il;
      }
      break;
    }
    const int64_t u = s.iu;
    int64_t l = s.il;
    const int64_t gu = gmap(P, u);
    double yl = (double)s.yl, fl = s.vl, al = s.al;
    const double yu = (double)s.yu;

    // 4. kernel rows of u and l for the own samples, K_ul, 2x2 solve, f update
    float ku[PER], kl[PER];
    double kul;
    if (GRAM && SO) {
      // Second-order rule: row u first, the gains of the own members of I_low above b_up, a
      // second exchange for l (its record carries f_l, a_l, y_l and K(u, l)), then row l.
      const SVMX_GLOBAL float *Ru = gp(p.gram) + gu * p.ld;
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int64_t j = base + threadIdx.x + (int64_t)k * BS;
        if (j < lim) ku[k] = Ru[gmap(P, j)];
      }
      Sel2 c;
      rec_init(c);
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int64_t j = base + threadIdx.x + (int64_t)k * BS;
        const bool lo = (yv[k] > 0 && a[k] > 0.0) || (yv[k] < 0 && a[k] < C);
        if (j < lim && lo && f[k] > s.vu) {
          const double g = so_gain(f[k], s.vu, ku[k]);
          if (gt_max(g, (int)j, c.g, c.il)) {
            c.g = g; c.fl = f[k]; c.al = a[k]; c.kul = (double)ku[k]; c.il = (int)j; c.yl = yv[k];
          }
        }
      }
      c = rec_block<Sel2, NW>(rec_wave(c), sh2, buf2);
      if (P.nwg > 1)
        c = exchange<Sel2, NW>(P, rank, (unsigned)(2 * t + 2), c, sh2, buf2, p.spin_limit, p.error, &s_abort);
      if (s_abort != 0) {
        if (rank == 0 && threadIdx.x == 0) {
          ctl->t = t;
          ctl->status = ST_TIMEOUT;
        }
        break;
      }
      // A member of I_low above b_up exists whenever the stop rule fails (b_low > b_up + tol);
      // the maximal violating pair's l stands in should none have been found.
      if (c.il != IBIG) {
        l = c.il;
        yl = (double)c.yl;
        fl = c.fl;
        al = c.al;
      }
      if (rank == 0 && threadIdx.x == 0 && t < P.trace_len && P.trace_ul) P.trace_ul[2 * t + 1] = (int)l;
      const int64_t gl = gmap(P, l);
      const SVMX_GLOBAL float *Rl = gp(p.gram) + gl * p.ld;
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int64_t j = base + threadIdx.x + (int64_t)k * BS;
        if (j < lim) kl[k] = Rl[gmap(P, j)];
      }
      kul = c.il != IBIG ? c.kul : (double)Ru[gl];
    } else if (GRAM) {
      const int64_t gl = gmap(P, l);
      const SVMX_GLOBAL float *Ru = gp(p.gram) + gu * p.ld;
      const SVMX_GLOBAL float *Rl = gp(p.gram) + gl * p.ld;
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int64_t j = base + threadIdx.x + (int64_t)k * BS;
        if (j < lim) {
          const int64_t g = gmap(P, j);
          ku[k] = Ru[g];
          kl[k] = Rl[g];
        }
      }
      kul = (double)Ru[gl];
    } else {
      const int64_t gl = gmap(P, l);
      const int64_t d = p.d;
      const int gs = group_size_for(d, VEC4);
      const int lig = threadIdx.x & (gs - 1);
      const int ngroups = BS / gs;
      const int grp = threadIdx.x / gs;
      // Block 0 of x_u and x_l is held in registers for the whole step; the samples stream
      // past it in batches of SB.
      const float *xu = p.X + gu * d, *xl = p.X + gl * d;
      const double nu = gp(p.sqn)[gu], nl = gp(p.sqn)[gl];
      RowPair<VEC4, ROW_MAXM> rp;
      load_pair(rp, xu, xl, d, lig, gs);
      int su = -1, sl = -1;
      bool hit_u = false, hit_l = false;
      if (use_cache) {
        su = (int)(gu % p.cache_cap);
        sl = (int)(gl % p.cache_cap);
        hit_u = tags[su] == (int)gu;
        hit_l = tags[sl] == (int)gl;
      }
      // K_ul: x_l as the sample against x_u, exactly as the row of u evaluates sample l
      if (grp == 0) {
        const float *xs1[1] = {xl};
        double pu1[1], pl1[1];
        dot_batch<VEC4, 1, ROW_MAXM>(xs1, 1, xu, xl, d, lig, gs, rp, pu1, pl1);
        if (lig == 0) s_kul = (double)rbf_from_dot(nu, nl, pu1[0], p.gamma);
      }
      if (!(hit_u && hit_l)) {
        typedef typename Lane<VEC4>::T T;
        const int64_t cnt = lim - base;
        // Streamed samples [res, cnt) go in batches of SBS per group; the first batch of each
        // group is loaded before the resident samples are computed, so its HBM latency
        // overlaps that work.
        constexpr int SBS = ONE ? 1 : VEC4 ? ROW_SBATCH : 2 * ROW_SBATCH;
        const int64_t sstride = (int64_t)ngroups * SBS;
        int64_t qs = res + (int64_t)grp * SBS;
        int nbs = 0;
        const float *xs[SBS];
        T vs[SBS][ROW_MAXM];
        if (qs < cnt) {
          nbs = (int)min<int64_t>(SBS, cnt - qs);
#pragma unroll
          for (int b = 0; b < SBS; ++b) xs[b] = p.X + gmap(P, base + qs + min(b, nbs - 1)) * d;
          load_block0<VEC4, SBS, ROW_MAXM>(vs, xs, nbs, d, lig, gs);
        }
        for (int64_t q0 = (int64_t)grp * SB; q0 < res; q0 += (int64_t)ngroups * SB) {
          const int nb = (int)min<int64_t>(SB, res - q0);
          const float *xr[SB];
#pragma unroll
          for (int b = 0; b < SB; ++b) xr[b] = xres + (q0 + min(b, nb - 1)) * d;
          T vr[SB][ROW_MAXM];
          load_block0<VEC4, SB, ROW_MAXM, true>(vr, xr, nb, d, lig, gs);
          float fu[SB], fl[SB];
          dot_partials<VEC4, SB, ROW_MAXM, true>(vr, xr, nb, xu, xl, d, lig, gs, rp, fu, fl);
          group_sums_store<SB>(fu, fl, nb, gs, lig, dotu + q0, dotl + q0);
        }
        while (qs < cnt) {
          float fu[SBS], fl[SBS];
          dot_partials<VEC4, SBS, ROW_MAXM>(vs, xs, nbs, xu, xl, d, lig, gs, rp, fu, fl);
          group_sums_store<SBS>(fu, fl, nbs, gs, lig, dotu + qs, dotl + qs);
          qs += sstride;
          if (qs < cnt) {
            nbs = (int)min<int64_t>(SBS, cnt - qs);
#pragma unroll
            for (int b = 0; b < SBS; ++b) xs[b] = p.X + gmap(P, base + qs + min(b, nbs - 1)) * d;
            load_block0<VEC4, SBS, ROW_MAXM>(vs, xs, nbs, d, lig, gs);
          }
        }
      }
      __syncthreads();
      kul = s_kul;
      const bool store_u = use_cache && !hit_u;
      const bool store_l = use_cache && !hit_l && !(sl == su && store_u);
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int64_t j = base + threadIdx.x + (int64_t)k * BS;
        if (j < lim) {
          const int64_t q = j - base;
          ku[k] = hit_u ? gp(p.cache)[(size_t)su * p.ld + j] : rbf_from_dot(nu, sq[k], dotu[q], p.gamma);
          kl[k] = hit_l ? gp(p.cache)[(size_t)sl * p.ld + j] : rbf_from_dot(nl, sq[k], dotl[q], p.gamma);
          if (store_u) gp(p.cache)[(size_t)su * p.ld + j] = ku[k];
          if (store_l) gp(p.cache)[(size_t)sl * p.ld + j] = kl[k];
        }
      }
      if (use_cache) {
        __syncthreads();
        if (threadIdx.x == 0) {
          if (store_u) tags[su] = (int)gu;
          if (store_l) tags[sl] = (int)gl;
        }
      }
    }
    const PairStep ps = solve_pair(C, s.vu, fl, s.au, al, yu, yl, kul);
    const double au_new = ps.au, al_new = ps.al;
    const double cu = (au_new - s.au) * yu, cl = (al_new - al) * yl;
    sel_init(s);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int64_t j = base + threadIdx.x + (int64_t)k * BS;
      if (j < lim) {
        f[k] = f_update(f[k], cu, ku[k], cl, kl[k]);
        if (j == u) a[k] = au_new;
        if (j == l) a[k] = al_new;
        consider(s, f[k], a[k], yv[k], (int)j, C);
      }
    }
    ++t;
  }

#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int64_t j = base + threadIdx.x + (int64_t)k * BS;
    if (j < lim) {
      gp(P.f)[j] = f[k];
      gp(P.alpha)[j] = a[k];
    }
  }
  if (use_cache) {
    __syncthreads();
    for (int s2 = threadIdx.x; s2 < p.cache_cap; s2 += BS) gp(p.cache_tags)[(size_t)blockIdx.x * p.cache_cap + s2] = tags[s2];
  }
}

// a = 0, f = -y for every problem; exchange words and control blocks cleared.
__global__ void smo_init(const Prob *probs, int32_t nprob) {
  const int32_t pid = blockIdx.y;
  const Prob P = probs[pid];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  for (int64_t j = i0; j < P.n; j += stride) {
    P.alpha[j] = 0.0;
    P.f[j] = -(double)label_of(P, j);
  }
  for (int64_t q = i0; q < 2 * (int64_t)P.nwg * SLOT_WORDS; q += stride) P.slots[q] = 0ull;
  if (P.slots2)
    for (int64_t q = i0; q < 2 * (int64_t)P.ng * SLOT_WORDS; q += stride) P.slots2[q] = 0ull;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    P.ctl->t = 0;
    P.ctl->status = ST_RUNNING;
    P.ctl->b_up = 0.0;
    P.ctl->b_low = 0.0;
    P.ctl->u = -1;
    P.ctl->l = -1;
  }
}

constexpr int FBS = 256;

// Per problem: out[4p+0] = sum a, out[4p+1] = sum a y f, out[4p+2] = #(a>0), out[4p+3] = #(a>=C).
__global__ void __launch_bounds__(FBS) smo_finalize(const Prob *probs, double C, double *out) {
  const Prob P = probs[blockIdx.x];
  double sa = 0.0, saf = 0.0, nsv = 0.0, nb = 0.0;
  for (int64_t j = threadIdx.x; j < P.n; j += FBS) {
    const double aj = P.alpha[j];
    sa += aj;
    saf += aj * (double)label_of(P, j) * P.f[j];
    nsv += aj > 0.0 ? 1.0 : 0.0;
    nb += aj >= C ? 1.0 : 0.0;
  }
  __shared__ double red[4][FBS / 64];
  for (int o = 32; o > 0; o >>= 1) {
    sa += __shfl_xor(sa, o);
    saf += __shfl_xor(saf, o);
    nsv += __shfl_xor(nsv, o);
    nb += __shfl_xor(nb, o);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { red[0][w] = sa; red[1][w] = saf; red[2][w] = nsv; red[3][w] = nb; }
  __syncthreads();
  if (threadIdx.x < 4) {
    double v = 0.0;
    for (int q = 0; q < FBS / 64; ++q) v += red[threadIdx.x][q];
    out[4 * (int64_t)blockIdx.x + threadIdx.x] = v;
  }
}

hipError_t launch_solver_init(const Prob *probs, int32_t nprob, int64_t max_n, hipStream_t s) {
  int64_t bx = (max_n + 255) / 256;
  if (bx < 1) bx = 1;
  if (bx > 4096) bx = 4096;
  hipLaunchKernelGGL(smo_init, dim3((unsigned)bx, (unsigned)nprob), dim3(256), 0, s, probs, nprob);
  return hipGetLastError();
}

hipError_t launch_finalize(const Prob *probs, int32_t nprob, double C, double *out, hipStream_t s) {
  hipLaunchKernelGGL(smo_finalize, dim3((unsigned)nprob), dim3(FBS), 0, s, probs, C, out);
  return hipGetLastError();
}

// Dynamic LDS of the row path: the fp64 dot products [2][per_wg], the cache tags, then `res`
// resident rows of d floats from a 16-byte boundary.
static size_t row_path_lds(const SolveParams &p, int64_t res) {
  const int64_t head = (16 * (int64_t)p.max_per_wg + 4 * (int64_t)p.cache_cap + 15) & ~(int64_t)15;
  return (size_t)(head + 4 * res * p.d);
}

static bool row_vec4(const SolveParams &p) {
  return (p.d % 4 == 0) && ((reinterpret_cast<uintptr_t>(p.X) & 15) == 0);
}

// Row path, float4 lanes with 8 samples a thread: there batches of two samples spill registers.
// For lane groups of up to 8 lanes (rows of up to 128 features) batches of one are faster
// (1,000,000 x 16: 25.8 -> 17.5 us a step; 1,000,000 x 64: 55.0 -> 46.0; 600,000 x 128: 55.2 ->
// 49.1); for wider groups the loads one batch keeps in flight matter more than the spill
// (batches of one: 600,000 x 256 115 -> 120 us, x 512 214 -> 238, x 784 326 -> 362).
static bool row_batch_one(const SolveParams &p, int32_t per_thread) {
  return per_thread == 8 && row_vec4(p) && group_size_for(p.d, true) <= 8;
}

template <int BS, int PER, bool GRAM, bool VEC4, bool ONE = false, bool SO = false>
static const void *kernel_of() {
  return reinterpret_cast<const void *>(&smo_solve<BS, PER, GRAM, VEC4, ONE, SO>);
}

// The solver variant for a path, samples per thread, (row path) float4 lanes and batches of
// one, (Gram path) the second-order rule; NULL if none.
static const void *solver_kernel(bool gram, int32_t per_thread, bool vec4, bool one = false, bool so = false) {
  if (gram && so) {
    switch (per_thread) {
      case 1: return kernel_of<BS_GRAM, 1, true, false, false, true>();
      case 2: return kernel_of<BS_GRAM, 2, true, false, false, true>();
      case 4: return kernel_of<BS_GRAM, 4, true, false, false, true>();
      case 8: return kernel_of<BS_GRAM, 8, true, false, false, true>();
      case 16: return kernel_of<BS_GRAM, 16, true, false, false, true>();
      default: return nullptr;
    }
  }
  if (gram) {
    switch (per_thread) {
      case 1: return kernel_of<BS_GRAM, 1, true, false>();
      case 2: return kernel_of<BS_GRAM, 2, true, false>();
      case 4: return kernel_of<BS_GRAM, 4, true, false>();
      case 8: return kernel_of<BS_GRAM, 8, true, false>();
      case 16: return kernel_of<BS_GRAM, 16, true, false>();
      default: return nullptr;
    }
  }
  switch (per_thread * 2 + (vec4 ? 1 : 0)) {
    case 2: return kernel_of<BS_ROWS, 1, false, false>();
    case 3: return kernel_of<BS_ROWS, 1, false, true>();
    case 4: return kernel_of<BS_ROWS, 2, false, false>();
    case 5: return kernel_of<BS_ROWS, 2, false, true>();
    case 8: return kernel_of<BS_ROWS, 4, false, false>();
    case 9: return kernel_of<BS_ROWS, 4, false, true>();
    case 16: return kernel_of<BS_ROWS, 8, false, false>();
    case 17: return one ? kernel_of<BS_ROWS, 8, false, true, true>() : kernel_of<BS_ROWS, 8, false, true>();
    default: return nullptr;
  }
}

hipError_t launch_solver(const SolveParams &p, int32_t total_wg, int32_t per_thread, bool gram, hipStream_t s,
                         int32_t *max_coresident) {
  if (p.second_order && !gram) return hipErrorInvalidValue;
  const void *fn = solver_kernel(gram, per_thread, !gram && row_vec4(p), !gram && row_batch_one(p, per_thread),
                                 p.second_order != 0);
  if (!fn) return hipErrorInvalidValue;
  const int bs = gram ? BS_GRAM : BS_ROWS;
  const size_t shmem = gram ? 0 : row_path_lds(p, p.res_rows);
  if (shmem > 48 * 1024) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return e;
  }
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, bs, shmem);
  if (e != hipSuccess) return e;
  if (max_coresident) *max_coresident = per_cu * cus;
  if (total_wg <= 0) return hipSuccess;  // capacity query only
  if ((int64_t)total_wg > (int64_t)per_cu * cus) return hipErrorCooperativeLaunchTooLarge;
  SolveParams pp = p;
  void *args[] = {&pp};
  return hipLaunchCooperativeKernel(fn, dim3((unsigned)total_wg), dim3(bs), args, (unsigned)shmem, s);
}

int64_t solver_res_rows_max(const SolveParams &p, int32_t per_thread) {
  int dev = 0, max_lds = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return -1;
  const void *fn = solver_kernel(false, per_thread, row_vec4(p), row_batch_one(p, per_thread));
  if (!fn) return -1;
  hipFuncAttributes attr;
  if (hipFuncGetAttributes(&attr, fn) != hipSuccess) return -1;
  const int64_t avail = (int64_t)max_lds - (int64_t)attr.sharedSizeBytes - (int64_t)row_path_lds(p, 0);
  return avail > 0 ? avail / (4 * p.d) : 0;
}

}  // namespace svmx

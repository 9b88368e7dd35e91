// api.cpp -- the C ABI of libsvmx.so (declared in include/svmx.h): argument checks, workspace
// planning, the host-side convergence loop and the one-vs-one orchestration.
//
// The paper runs the SMO iterations on the device and checks convergence on the host after
// every set of iterations (Section III.B).  Here each solver launch advances every running
// problem by up to check_every steps on the device; the host then reads the per-problem
// control blocks and launches again while any problem is still running.  Because the device
// stops a problem by itself once the stop rule holds, results do not depend on check_every.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"
#include "warm.hpp"
#include "svmx.h"

using namespace svmx;

namespace {

thread_local std::string g_err;

svm_status fail(svm_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIPCHK(expr)                                                                      \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess) return fail(SVM_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr int64_t DEFAULT_GRAM_BUDGET = 200LL << 30;  // bytes of HBM the Gram may take by default
constexpr int32_t DEFAULT_CHECK_EVERY = 65536;
constexpr int64_t ALIGN = 256;
constexpr int32_t CACHE_CAP_MAX = 4096;               // row-cache slots (tags live in LDS)
constexpr double SPIN_SECONDS = 2.0;                  // longest a device-side wait may last
constexpr int64_t LDS_BYTES = 160 * 1024;
constexpr int32_t MAX_CLASSES = 64;
constexpr double WS_FRAC = 0.5;           // working-set rounds stop at max(tol, 0.5 x the round's gap)
constexpr int32_t WS_INNER_PER_Q = 100;   // and take at most 100 q pair steps
// working_set = SVM_WORKING_SET_AUTO: for rows of 256 features or more q = 64 with a Gram (47.0
// ms against 49.4 with q = 128 at 20,000 x 784) and 128 without (88.5 ms against 109.5 with
// q = 64), else 32; the first WS_AUTO_PROBE_ROUNDS rounds decide.  The rounds go on when they took at least as many
// pair steps per round as a round costs in pair steps (measured on MI355X: a round of q = 32
// costs 4.4 to 6.2 pair steps on the Gram path -- 23.0 us against 5.22 at 100,000 x 32, 20.4
// against 4.61 at 50,000 x 128, 25.1 against 4.05 at 20,000 x 784 -- and 4.7 on the row path
// -- 38.7 us against 8.25 at 100,000 x 32; one of q = 128 9.9 to 18.1 on the Gram path -- 45.8
// us against 4.61 at 50,000 x 128, 65.1 against 5.22 at 100,000 x 32, 73.4 against 4.05 at
// 20,000 x 784 -- and about 11.4 on the row path, 135 us against 11.8 at 20,000 x 784), else
// the pair solver takes over from the state the rounds reached.  Steps a round rise over a
// training (at 100,000 x 32 from 6.5 in the first 128 rounds to 8.6 over all; on the
// 50,000 x 128 mixture from 4.3 to 4.8), so the q = 32 thresholds sit a little under the
// break-even of the problems that q is chosen for (rows of fewer than 256 features: 4.4 on the
// Gram path, 4.7 on the row path); q = 128 keeps a margin above its 18.1.
constexpr int64_t WS_AUTO_PROBE_ROUNDS = 128;
double ws_auto_min_steps(int32_t q, bool gram) {
  if (q >= 128) return gram ? 20.0 : 12.5;
  if (q >= 64) return gram ? 10.0 : 8.0;  // break-evens 9.75 (39.5 us against 4.05 at 20,000 x 784), 7.8
  return gram ? 4.25 : 4.5;
}

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

bool finite_pos(double v) { return std::isfinite(v) && v > 0.0; }

struct Opts {
  int32_t gram;
  int64_t gram_budget;
  int64_t row_cache_bytes;
  int64_t max_iter;
  int32_t check_every;
  int32_t trace_len;
  int32_t *trace_ws;
  double *trace_b;
  double *f_out;
  hipStream_t stream;
  int32_t workgroups;
  int32_t levels;
  int32_t gram_mfma;
  int32_t working_set;
  int32_t resident_rows;
  int32_t selection;
  const double *alpha_init;
  const double *f_init;
};

bool resolve(const svm_options *o, int64_t n, Opts *r) {
  svm_options d;
  svm_default_options(&d);
  if (!o) o = &d;
  if (o->struct_size != (int32_t)sizeof(svm_options)) return false;
  r->gram = o->gram;
  r->gram_budget = o->gram_budget_bytes > 0 ? o->gram_budget_bytes : DEFAULT_GRAM_BUDGET;
  r->row_cache_bytes = std::max<int64_t>(0, o->row_cache_bytes);
  r->max_iter = o->max_iter > 0 ? o->max_iter : std::max<int64_t>(10000000, 100 * n);
  r->check_every = o->check_every > 0 ? o->check_every : DEFAULT_CHECK_EVERY;
  r->trace_len = std::max<int32_t>(0, o->trace_len);
  r->trace_ws = o->trace_ws;
  r->trace_b = o->trace_b;
  r->f_out = o->f_out;
  r->stream = reinterpret_cast<hipStream_t>(o->stream);
  r->workgroups = std::max<int32_t>(0, o->workgroups);
  r->levels = o->exchange_levels;
  r->gram_mfma = o->gram_mfma;
  r->working_set = o->working_set;
  r->resident_rows = o->resident_rows;
  r->selection = o->selection;
  r->alpha_init = o->alpha_init;
  r->f_init = o->f_init;
  if (o->reserved != 0 || (r->selection != SVM_SELECT_MVP && r->selection != SVM_SELECT_SECOND_ORDER)) return false;
  if (r->selection == SVM_SELECT_SECOND_ORDER && r->working_set > 0) return false;
  const bool ws_ok = r->working_set == 0 || r->working_set == SVM_WORKING_SET_AUTO ||
                     (r->working_set >= 2 && r->working_set <= ws_q_max() && r->working_set % 2 == 0);
  return r->gram >= SVM_GRAM_AUTO && r->gram <= SVM_GRAM_OFF && r->levels >= 0 && r->levels <= 2 &&
         (r->gram_mfma == SVM_MFMA_SPLIT_F16 || r->gram_mfma == SVM_MFMA_F32) && ws_ok && r->resident_rows >= -1;
}

// How a problem of n samples is spread over workgroups.
struct Shape {
  int32_t nwg, per_wg, per_thread, g1, ng;
};

constexpr int32_t TWO_LEVEL_ABOVE = 128;  // workgroups per problem above which the exchange has two levels


// Gram path: one workgroup up to 4096 samples (no exchange at all), else about sqrt(n)/3.5
// workgroups, at most 64 -- the measured optimum between per-workgroup work and exchange
// cost on MI355X (40 at n = 20,000, 64 at 50,000 and 100,000).  Row path: up to 256 workgroups of 512
// threads (at least 64 samples each), so that the streaming of X keeps every CU busy.  `cap` bounds the count
// (one-vs-one runs all pairs in one launch, so their workgroups must fit together).
bool choose_shape(int64_t n, bool gram, int32_t requested, int32_t levels, Shape *s, int64_t cap = 256) {
  const int64_t BS = solver_block_size(gram), MAXP = max_per_thread(gram);
  int64_t nwg;
  if (requested > 0)
    nwg = requested;
  else if (gram)
    nwg = n <= 4096 ? 1
                    : std::min<int64_t>(std::min<int64_t>(cap, 64),
                                        std::max<int64_t>(8, (int64_t)std::ceil(std::sqrt((double)n) / 3.5)));
  else
    nwg = std::min<int64_t>(cap, std::max<int64_t>(1, (n + 63) / 64));
  nwg = std::max<int64_t>(1, std::min<int64_t>(nwg, n));
  if ((n + nwg - 1) / nwg > BS * MAXP) nwg = (n + BS * MAXP - 1) / (BS * MAXP);
  int64_t per_wg = (n + nwg - 1) / nwg;
  nwg = (n + per_wg - 1) / per_wg;  // no empty workgroups
  int64_t per = (per_wg + BS - 1) / BS, p = 1;
  while (p < per) p <<= 1;
  if (p > MAXP || nwg > 65536) return false;
  s->nwg = (int32_t)nwg;
  s->per_wg = (int32_t)per_wg;
  s->per_thread = (int32_t)p;
  // One level up to 128 workgroups; beyond that, every workgroup polling every record costs
  // more (the polls of all workgroups crowd the same lines) than a second round trip.
  if (nwg > 1 && (levels == 2 || (levels == 0 && nwg > TWO_LEVEL_ABOVE))) {
    s->g1 = (int32_t)std::ceil(std::sqrt((double)nwg));
    s->ng = (int32_t)((nwg + s->g1 - 1) / s->g1);
  } else {
    s->g1 = 0;
    s->ng = 0;
  }
  return true;
}

// Working-set solver: 64 samples or more per owning workgroup (at most ws_slice_max()), at
// most 255 owners (plus the solving workgroup), so that every list merge takes at most 16
// lists: one level up to 16 owners, else groups of ceil(sqrt(nwg)).
constexpr int32_t WS_MAX_WG = 255;

bool choose_ws_shape(int64_t n, int32_t requested, int32_t q, bool gram, Shape *s) {
  int64_t nwg = requested > 0 ? requested : std::min<int64_t>(WS_MAX_WG, (n + 63) / 64);
  nwg = std::max<int64_t>(1, std::min<int64_t>(nwg, n));
  // row path: at least two owners (the solving workgroup holds K_BB while the owners hold
  // K(B, own samples)), and q x samples per owner within the LDS row buffer
  const int64_t smax = gram ? ws_slice_max() : std::min<int64_t>(ws_slice_max(), ws_row_cap() / q);
  if (!gram) nwg = std::max<int64_t>(nwg, 2);
  if ((n + nwg - 1) / nwg > smax) nwg = (n + smax - 1) / smax;
  if (nwg > WS_MAX_WG) return false;
  const int64_t per_wg = (n + nwg - 1) / nwg;
  nwg = (n + per_wg - 1) / per_wg;
  s->nwg = (int32_t)nwg;
  s->per_wg = (int32_t)per_wg;
  s->per_thread = 0;
  if (nwg > 16) {
    s->g1 = (int32_t)std::ceil(std::sqrt((double)nwg));
    s->ng = (int32_t)((nwg + s->g1 - 1) / s->g1);
  } else {
    s->g1 = 0;
    s->ng = 0;
  }
  return true;
}

struct Layout {
  int64_t total = 0;
  int64_t add(int64_t bytes) {
    int64_t off = round_up(total, ALIGN);
    total = off + std::max<int64_t>(bytes, 0);
    return off;
  }
};

// ---------------------------------------------------------------------------- static scratch
// The device workspace of svm_train_static: one array per device, alive until the process ends.
// Its name is a host-side stand-in in host code; the device address comes from
// hipGetSymbolAddress, taken once per device (with that device current) and kept.
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

svm_status static_scratch(void **out);

// ---------------------------------------------------------------------------- binary plan
struct TrainPlan {
  bool gram;
  int64_t ld;
  Shape shape;
  int32_t working_set;   // q of the working-set rounds (0: pair steps only)
  int32_t auto_q;        // working_set = AUTO chose rounds of q: probe them, maybe switch
  double auto_min_steps; // pair steps per round the probe must reach to keep the rounds
  Shape pair_shape;      // the pair solver's shape, for a switch
  int32_t cache_cap;
  int64_t off_f, off_gram, off_split, off_sqn, off_cache, off_tags, off_ctl, off_prob, off_wgp, off_slots, off_slots2,
      off_tul, off_tb, off_fin, off_err, off_rounds, off_warm;
  int64_t slot_words, slot2_words;
  int64_t total;
};

svm_status plan_train(int64_t n, int64_t d, const Opts &o_in, TrainPlan *p) {
  Opts o = o_in;
  if (n < 2 || d < 1) return fail(SVM_EINVAL, "need n >= 2 and d >= 1 (got n=%lld, d=%lld)", (long long)n, (long long)d);
  if (n > 0x7ffffffeLL) return fail(SVM_ENOMEM, "n=%lld exceeds the 32-bit sample index", (long long)n);
  if (d > (INT64_MAX / 8) / n) return fail(SVM_EINVAL, "n*d overflows 64-bit byte counts");
  p->ld = round_up(n, 64);
  const double gram_bytes = 4.0 * (double)n * (double)p->ld;
  if (o.gram == SVM_GRAM_ON)
    p->gram = true;
  else if (o.gram == SVM_GRAM_OFF)
    p->gram = false;
  else
    p->gram = gram_bytes <= (double)o.gram_budget;
  if (p->gram && gram_bytes > 9.0e18) return fail(SVM_EINVAL, "the Gram's n^2 size overflows 64-bit byte counts");
  if (o.selection == SVM_SELECT_SECOND_ORDER && !p->gram)
    return fail(SVM_EINVAL, "second-order selection needs the Gram path (the Gram does not fit gram_budget_bytes, "
                            "or gram = SVM_GRAM_OFF)");
  p->auto_q = 0;
  p->auto_min_steps = 0.0;
  if (o.working_set == SVM_WORKING_SET_AUTO) {
    // rounds only where a problem spreads over several workgroups, with the first-order rule,
    // no trace (a trace records pair steps) and the automatic workgroup count
    o.working_set = 0;
    const int32_t q = d >= 256 ? (p->gram ? 64 : 128) : 32;
    Shape ws;
    if (o.selection == SVM_SELECT_MVP && o.trace_len == 0 && o.workgroups == 0 && n > 4096 &&
        choose_ws_shape(n, 0, q, p->gram, &ws) && ws.nwg > 1) {
      o.working_set = q;
      p->auto_q = q;
      p->auto_min_steps = ws_auto_min_steps(q, p->gram);
      if (!choose_shape(n, p->gram, 0, o.levels, &p->pair_shape)) return fail(SVM_ENOMEM, "problem too large to place");
    }
  }
  p->working_set = o.working_set;
  if (o.working_set > 0) {
    if (!choose_ws_shape(n, o.workgroups, o.working_set, p->gram, &p->shape))
      return fail(SVM_ENOMEM, "n=%lld exceeds the working-set solver's %d workgroups of %d samples", (long long)n,
                  WS_MAX_WG, p->gram ? ws_slice_max() : std::min(ws_slice_max(), ws_row_cap() / o.working_set));
  } else if (!choose_shape(n, p->gram, o.workgroups, o.levels, &p->shape)) {
    return fail(SVM_ENOMEM, "problem too large to place");
  }
  p->cache_cap = 0;
  if (!p->gram) {
    if (o.row_cache_bytes > 0)
      p->cache_cap = (int32_t)std::min<int64_t>(CACHE_CAP_MAX, std::min<int64_t>(n, o.row_cache_bytes / (4 * p->ld)));
    const int64_t lds = 16LL * p->shape.per_wg + 4LL * p->cache_cap + 8192;
    if (lds > LDS_BYTES) return fail(SVM_EINVAL, "row path: dot products and cache tags do not fit the LDS");
  }
  Layout L;
  p->off_f = L.add(8 * n);
  p->off_gram = p->gram ? L.add((int64_t)gram_bytes) : -1;
  // split rows: the split-fp16 Gram, or the working-set row path (which evaluates its rows with them)
  const bool split = (p->gram && o.gram_mfma == SVM_MFMA_SPLIT_F16) || (!p->gram && o.working_set > 0);
  p->off_split = split ? L.add(gram_split_scratch_bytes(n, d)) : -1;
  p->off_sqn = p->gram ? -1 : L.add(8 * n);
  p->off_cache = p->cache_cap ? L.add(4LL * p->cache_cap * p->ld) : -1;
  p->off_tags = p->cache_cap ? L.add(4LL * p->cache_cap * p->shape.nwg) : -1;
  p->off_ctl = L.add(sizeof(Ctl));
  p->off_prob = L.add(sizeof(Prob));
  p->off_wgp = L.add(4LL * std::max(p->shape.nwg + 1, p->auto_q ? p->pair_shape.nwg : 0));
  const int64_t per_rec = o.working_set > 0 ? ws_list_words() : SLOT_WORDS;
  p->slot_words = 2LL * p->shape.nwg * per_rec;
  p->slot2_words = 2LL * std::max(1, p->shape.ng) * per_rec + (o.working_set > 0 ? ws_bcast_words() : 0);
  p->off_slots = L.add(8LL * p->slot_words);
  p->off_slots2 = L.add(8LL * p->slot2_words);
  p->off_tul = L.add(4LL * 2 * o.trace_len);
  p->off_tb = L.add(8LL * 2 * o.trace_len);
  p->off_fin = L.add(8 * 4);
  p->off_err = L.add(16);
  p->off_rounds = L.add(8);
  p->off_warm = o.alpha_init ? L.add(12LL * n) : -1;  // warm start: support-vector list (coefs, indices)
  p->total = round_up(L.total, ALIGN);
  return SVM_OK;
}

uint64_t spin_ticks() {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      khz <= 0)
    khz = 100000;
  return (uint64_t)(SPIN_SECONDS * 1000.0 * (double)khz);
}

// A pair of HIP events on the launch stream; init(false) leaves it off (no events are created,
// every record is a no-op and seconds() is 0), for the entry point that creates no resources.
struct Timer {
  hipEvent_t a = nullptr, b = nullptr;
  ~Timer() {
    if (a) (void)hipEventDestroy(a);
    if (b) (void)hipEventDestroy(b);
  }
  hipError_t init(bool on = true) {
    if (!on) return hipSuccess;
    hipError_t e = hipEventCreate(&a);
    if (e != hipSuccess) return e;
    return hipEventCreate(&b);
  }
  hipError_t start(hipStream_t s) { return a ? hipEventRecord(a, s) : hipSuccess; }
  hipError_t stop(hipStream_t s) { return b ? hipEventRecord(b, s) : hipSuccess; }
  double seconds() {
    float ms = 0.f;
    if (!a || !b || hipEventElapsedTime(&ms, a, b) != hipSuccess) return 0.0;
    return ms * 1e-3;
  }
};

struct NeverStop {
  bool operator()() const { return false; }
};

// Launch a solver (launch(&max_coresident) enqueues one launch) until no problem is running,
// or until stop() says so after a launch.  Returns SVM_OK or a negative status.
template <class Launch, class Stop = NeverStop>
svm_status run_launches(Launch launch, int32_t *error, int32_t nprob, int32_t total_wg, Ctl *d_ctl, hipStream_t stream,
                        int32_t *launches, std::vector<Ctl> &h, double *t_kernel, bool timed = true,
                        Stop stop = Stop()) {
  int32_t herr = 0;
  Timer tk;
  HIPCHK(tk.init(timed));
  h.assign(nprob, Ctl{});
  std::vector<int64_t> prev(nprob, -1);
  for (;;) {
    int32_t maxres = 0;
    HIPCHK(tk.start(stream));
    hipError_t e = launch(&maxres);
    if (e == hipErrorCooperativeLaunchTooLarge)
      return fail(SVM_ENOMEM, "%d solver workgroups do not fit on the device at once (at most %d)", total_wg, maxres);
    if (e != hipSuccess) return fail(SVM_EDEVICE, "solver launch: %s", hipGetErrorString(e));
    ++*launches;
    HIPCHK(tk.stop(stream));
    HIPCHK(hipMemcpyAsync(h.data(), d_ctl, sizeof(Ctl) * nprob, hipMemcpyDeviceToHost, stream));
    HIPCHK(hipMemcpyAsync(&herr, error, sizeof(herr), hipMemcpyDeviceToHost, stream));
    HIPCHK(hipStreamSynchronize(stream));
    if (herr) return fail(SVM_EDEVICE, "a device-side wait exceeded its %.1f s limit", SPIN_SECONDS);
    *t_kernel += tk.seconds();
    bool running = false, progress = false;
    for (int32_t q = 0; q < nprob; ++q) {
      if (h[q].status == ST_TIMEOUT)
        return fail(SVM_EDEVICE, "a device-side wait exceeded its %.1f s limit (problem %d, step %lld)", SPIN_SECONDS, q,
                    (long long)h[q].t);
      if (h[q].status == ST_RUNNING) running = true;
      if (h[q].t != prev[q]) progress = true;
      prev[q] = h[q].t;
    }
    if (!running) return SVM_OK;
    if (!progress) return fail(SVM_EDEVICE, "solver made no progress");
    if (stop()) return SVM_OK;
  }
}

// (*t_kernel accumulates over the calls of one training.)
svm_status run_solver(SolveParams sp, int32_t nprob, int32_t total_wg, int32_t per_thread, bool gram, Ctl *d_ctl,
                      hipStream_t stream, int32_t *launches, std::vector<Ctl> &h, double *t_kernel,
                      bool timed = true) {
  return run_launches([&](int32_t *maxres) { return launch_solver(sp, total_wg, per_thread, gram, stream, maxres); },
                      sp.error, nprob, total_wg, d_ctl, stream, launches, h, t_kernel, timed);
}

// EINVAL unless every value of X[0 .. count) is finite (a NaN or an infinity would leave no
// stop test true, and the solver would run to max_iter).  flag: a cleared device word.
svm_status check_finite(const float *X, int64_t count, int32_t *flag, hipStream_t stream) {
  HIPCHK(launch_check_finite(X, count, flag, stream));
  int32_t bad = 0;
  HIPCHK(hipMemcpyAsync(&bad, flag, sizeof(bad), hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  if (bad) return fail(SVM_EINVAL, "X holds a value that is not finite");
  return SVM_OK;
}

svm_status check_labels_pm1(const int32_t *y, int64_t n, hipStream_t stream) {
  std::vector<int32_t> h(n);
  HIPCHK(hipMemcpyAsync(h.data(), y, 4 * n, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  int64_t pos = 0, neg = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (h[i] == 1)
      ++pos;
    else if (h[i] == -1)
      ++neg;
    else
      return fail(SVM_EINVAL, "label y[%lld] = %d is not +1 or -1", (long long)i, h[i]);
  }
  if (!pos || !neg) return fail(SVM_EINVAL, "both classes must be present (%lld positive, %lld negative)", (long long)pos,
                                (long long)neg);
  return SVM_OK;
}

// ---------------------------------------------------------------------------- one-vs-one
struct OvoPlan {
  bool gram;
  int64_t ld;
  int32_t P;
  int64_t off_perm, off_xs, off_f, off_gram, off_split, off_sqn, off_ctl, off_prob, off_wgp, off_slots, off_slots2,
      off_fin, off_err;
  int64_t total;
};

constexpr int32_t OVO_MAX_WG_PER_PAIR = 256;
constexpr int32_t OVO_MAX_GROUPS = 16;  // second-level groups of a pair: ceil(256 / ceil(sqrt(256)))
constexpr int64_t OVO_TOTAL_WG = 512;  // default workgroup budget shared by all pairs of one launch

svm_status plan_ovo(int64_t n, int64_t d, int32_t k, const Opts &o, OvoPlan *p) {
  if (n < 2 || d < 1) return fail(SVM_EINVAL, "need n >= 2 and d >= 1");
  if (k < 2 || k > MAX_CLASSES) return fail(SVM_EINVAL, "k=%d must be in [2, %d]", k, MAX_CLASSES);
  if (n > 0x7ffffffeLL) return fail(SVM_ENOMEM, "n too large");
  if (d > (INT64_MAX / 8) / n) return fail(SVM_EINVAL, "n*d overflows 64-bit byte counts");
  p->P = k * (k - 1) / 2;
  p->ld = round_up(n, 64);
  const double gram_bytes = 4.0 * (double)n * (double)p->ld;
  p->gram = o.gram == SVM_GRAM_ON || (o.gram == SVM_GRAM_AUTO && gram_bytes <= (double)o.gram_budget);
  if (o.selection == SVM_SELECT_SECOND_ORDER && !p->gram)
    return fail(SVM_EINVAL, "second-order selection needs the Gram path");
  Layout L;
  p->off_perm = L.add(4 * n);
  p->off_xs = L.add(4 * n * d);
  p->off_f = L.add(8 * (int64_t)(k - 1) * n);
  p->off_gram = p->gram ? L.add((int64_t)gram_bytes) : -1;
  p->off_split = (p->gram && o.gram_mfma == SVM_MFMA_SPLIT_F16) ? L.add(gram_split_scratch_bytes(n, d)) : -1;
  p->off_sqn = p->gram ? -1 : L.add(8 * n);
  p->off_ctl = L.add((int64_t)sizeof(Ctl) * p->P);
  p->off_prob = L.add((int64_t)sizeof(Prob) * p->P);
  p->off_wgp = L.add(4LL * p->P * OVO_MAX_WG_PER_PAIR);
  p->off_slots = L.add(8LL * 2 * SLOT_WORDS * p->P * OVO_MAX_WG_PER_PAIR);
  p->off_slots2 = L.add(8LL * 2 * SLOT_WORDS * p->P * OVO_MAX_GROUPS);
  p->off_fin = L.add(8LL * 4 * p->P);
  p->off_err = L.add(16);
  p->total = round_up(L.total, ALIGN);
  return SVM_OK;
}

// Class counts and the stable class-sorted order of the labels (host copy).
svm_status class_sort(const int32_t *label, int64_t n, int32_t k, hipStream_t stream, std::vector<int32_t> &perm,
                      std::vector<int64_t> &start, std::vector<int64_t> &cnt) {
  std::vector<int32_t> h(n);
  HIPCHK(hipMemcpyAsync(h.data(), label, 4 * n, hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  cnt.assign(k, 0);
  for (int64_t i = 0; i < n; ++i) {
    if (h[i] < 0 || h[i] >= k) return fail(SVM_EINVAL, "label[%lld] = %d is outside 0..%d", (long long)i, h[i], k - 1);
    cnt[h[i]]++;
  }
  for (int32_t c = 0; c < k; ++c)
    if (!cnt[c]) return fail(SVM_EINVAL, "class %d has no samples", c);
  start.assign(k, 0);
  for (int32_t c = 1; c < k; ++c) start[c] = start[c - 1] + cnt[c - 1];
  perm.assign(n, 0);
  std::vector<int64_t> pos(start);
  for (int64_t i = 0; i < n; ++i) perm[pos[h[i]]++] = (int32_t)i;
  return SVM_OK;
}

// Layout of the prediction scratch: for up to `pairs` problems of one launch with up to ntr
// training samples each (n rows of X in all) and m test samples of d features, the compacted
// support vectors, the partial sums, the problems' descriptions, and the split-fp16 rows of
// both sets.
struct PredictWs {
  PredictScratch ps;
  SplitX train, test;
};

constexpr int32_t PREDICT_PAIRS_MAX = 64;  // problems per prediction launch (bounds the partial sums)

int64_t predict_scratch_bytes(int64_t n, int64_t ntr, int64_t pairs, int64_t m, int64_t d) {
  Layout L;
  L.add(4 * ntr * pairs);
  L.add(8 * ntr * pairs);
  L.add(8 * pairs);
  L.add(8LL * predict_splits(m, ntr) * std::max<int64_t>(m, 1) * pairs);
  L.add((int64_t)sizeof(PredPair) * pairs);
  L.add(gram_split_scratch_bytes(n, d));
  L.add(gram_split_scratch_bytes(std::max<int64_t>(m, 1), d));
  return round_up(L.total, ALIGN);
}

PredictWs predict_scratch(void *base, int64_t n, int64_t ntr, int64_t pairs, int64_t m, int64_t d) {
  Layout L;
  char *b = static_cast<char *>(base);
  PredictWs w;
  w.ps.sv_row = reinterpret_cast<int32_t *>(b + L.add(4 * ntr * pairs));
  w.ps.sv_coef = reinterpret_cast<double *>(b + L.add(8 * ntr * pairs));
  w.ps.count = reinterpret_cast<int64_t *>(b + L.add(8 * pairs));
  w.ps.part = reinterpret_cast<double *>(b + L.add(8LL * predict_splits(m, ntr) * std::max<int64_t>(m, 1) * pairs));
  w.ps.pairs = reinterpret_cast<PredPair *>(b + L.add((int64_t)sizeof(PredPair) * pairs));
  w.train = split_views(b + L.add(gram_split_scratch_bytes(n, d)), n, d);
  w.test = split_views(b + L.add(gram_split_scratch_bytes(std::max<int64_t>(m, 1), d)), std::max<int64_t>(m, 1), d);
  return w;
}

// Split rows of the training and test sets for the split-fp16 predict kernel (default), or
// leave the fp32 kernel selected.
hipError_t predict_prepare(PredictWs &w, const Opts &r, const float *Xtr, int64_t ntr, const float *T, int64_t m,
                           int64_t d) {
  if (r.gram_mfma != SVM_MFMA_SPLIT_F16) return hipSuccess;
  hipError_t e = launch_split_rows(Xtr, ntr, d, w.train, r.stream);
  if (e != hipSuccess) return e;
  e = launch_split_rows(T, m, d, w.test, r.stream);
  if (e != hipSuccess) return e;
  w.ps.split_train = &w.train;
  w.ps.split_test = &w.test;
  return hipSuccess;
}

}  // namespace

static __device__ __align__(256) unsigned char scratch[SVM_STATIC_SCRATCH_BYTES];

namespace {
svm_status static_scratch(void **out) {
  int dev = 0;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(SVM_EDEVICE, "device %d outside the scratch table", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SVM_EDEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SVM_OK;
}
}  // namespace

// ============================================================================ C ABI
extern "C" {

void svm_default_options(svm_options *o) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->struct_size = (int32_t)sizeof(svm_options);
  o->gram = SVM_GRAM_AUTO;
  o->check_every = DEFAULT_CHECK_EVERY;
}

const char *svm_last_error(void) { return g_err.c_str(); }

int64_t svm_train_workspace_bytes(int64_t n, int64_t d, const svm_options *o) {
  Opts r;
  if (!resolve(o, n, &r)) return -1;
  TrainPlan p;
  if (plan_train(n, d, r, &p) != SVM_OK) return -1;
  return p.total;
}

// Binary training.  static_ws: the workspace is the library's static device scratch (the
// caller passes none); the plan must fit it, and no HIP events or other resources are created.
static svm_status train_impl(const float *X, const int32_t *y, int64_t n, int64_t d, double C, double gamma,
                             double tol, double *alpha, double *b, void *workspace, int64_t workspace_bytes,
                             const svm_options *o, svm_stats *st, bool static_ws) {
  const auto t_start = std::chrono::steady_clock::now();
  g_err.clear();
  if (!X || !y || !alpha || !b) return fail(SVM_EINVAL, "NULL pointer argument");
  if (!finite_pos(C) || !finite_pos(gamma) || !finite_pos(tol))
    return fail(SVM_EINVAL, "C, gamma and tol must be finite and > 0");
  Opts r;
  if (!resolve(o, n, &r)) return fail(SVM_EINVAL, "bad options (struct_size or gram mode)");
  if (r.trace_len > 0 && (int64_t)r.trace_len > r.max_iter + 1) r.trace_len = (int32_t)(r.max_iter + 1);
  TrainPlan p;
  svm_status s0;
  if (static_ws) {
    // AUTO takes the Gram only when the whole plan fits the scratch, else the row path
    Opts rs = r;
    if (rs.gram == SVM_GRAM_AUTO) rs.gram_budget = std::min<int64_t>(rs.gram_budget, SVM_STATIC_SCRATCH_BYTES);
    s0 = plan_train(n, d, rs, &p);
    if (s0 == SVM_OK && r.gram == SVM_GRAM_AUTO && p.gram && p.total > SVM_STATIC_SCRATCH_BYTES) {
      rs.gram = SVM_GRAM_OFF;
      s0 = plan_train(n, d, rs, &p);
    }
    if (s0 != SVM_OK) return s0;
    if (p.total > SVM_STATIC_SCRATCH_BYTES)
      return fail(SVM_EWORKSPACE, "n=%lld, d=%lld needs %lld bytes of device scratch; svm_train_static has %lld",
                  (long long)n, (long long)d, (long long)p.total, (long long)SVM_STATIC_SCRATCH_BYTES);
    s0 = static_scratch(&workspace);
    if (s0 != SVM_OK) return s0;
    workspace_bytes = SVM_STATIC_SCRATCH_BYTES;
  } else {
    s0 = plan_train(n, d, r, &p);
    if (s0 != SVM_OK) return s0;
    if (!workspace || workspace_bytes < p.total)
      return fail(SVM_EWORKSPACE, "workspace of %lld bytes needed, %lld given", (long long)p.total,
                  (long long)workspace_bytes);
  }
  const bool timed = !static_ws;
  hipStream_t stream = r.stream;
  s0 = check_labels_pm1(y, n, stream);
  if (s0 != SVM_OK) return s0;
  // warm start: the given multipliers (and f) read to the host before anything writes alpha,
  // checked, and their support vectors listed for the device
  std::vector<double> warm_a, warm_f, warm_coef;
  std::vector<int32_t> warm_y, warm_sv;
  if (r.f_init && !r.alpha_init) return fail(SVM_EINVAL, "f_init needs alpha_init");
  if (r.alpha_init) {
    warm_a.resize(n);
    warm_y.resize(n);
    HIPCHK(hipMemcpyAsync(warm_a.data(), r.alpha_init, 8 * n, hipMemcpyDeviceToHost, stream));
    HIPCHK(hipMemcpyAsync(warm_y.data(), y, 4 * n, hipMemcpyDeviceToHost, stream));
    if (r.f_init) {
      warm_f.resize(n);
      HIPCHK(hipMemcpyAsync(warm_f.data(), r.f_init, 8 * n, hipMemcpyDeviceToHost, stream));
    }
    HIPCHK(hipStreamSynchronize(stream));
    double sum_ay = 0.0;
    for (int64_t i = 0; i < n; ++i) {
      const double a = warm_a[i];
      if (!(std::isfinite(a) && a >= 0.0 && a <= C))
        return fail(SVM_EINVAL, "alpha_init[%lld] = %g is outside [0, C]", (long long)i, a);
      sum_ay += a * (double)warm_y[i];
      if (a > 0.0) {
        warm_sv.push_back((int32_t)i);
        warm_coef.push_back(a * (double)warm_y[i]);
      }
    }
    if (!(std::fabs(sum_ay) <= 1e-9 * C * (double)n))
      return fail(SVM_EINVAL, "alpha_init breaks the equality constraint: sum a_i y_i = %g", sum_ay);
    for (int64_t i = 0; i < (int64_t)warm_f.size(); ++i)
      if (!std::isfinite(warm_f[i])) return fail(SVM_EINVAL, "f_init[%lld] is not finite", (long long)i);
  }

  char *ws = static_cast<char *>(workspace);
  double *f = reinterpret_cast<double *>(ws + p.off_f);
  float *G = p.gram ? reinterpret_cast<float *>(ws + p.off_gram) : nullptr;
  Ctl *ctl = reinterpret_cast<Ctl *>(ws + p.off_ctl);
  Prob *dprob = reinterpret_cast<Prob *>(ws + p.off_prob);
  int32_t *wgp = reinterpret_cast<int32_t *>(ws + p.off_wgp);
  u64 *slots = reinterpret_cast<u64 *>(ws + p.off_slots);
  int32_t *tul = reinterpret_cast<int32_t *>(ws + p.off_tul);
  double *tb = reinterpret_cast<double *>(ws + p.off_tb);
  double *fin = reinterpret_cast<double *>(ws + p.off_fin);
  int32_t *err = reinterpret_cast<int32_t *>(ws + p.off_err);

  Prob hp{};
  hp.n = n;
  hp.off0 = 0;
  hp.len0 = n;
  hp.off1 = n;
  hp.y = y;
  hp.alpha = alpha;
  hp.f = f;
  hp.ctl = ctl;
  hp.slots = slots;
  hp.trace_ul = r.trace_len ? tul : nullptr;
  hp.trace_b = r.trace_len ? tb : nullptr;
  hp.trace_len = r.trace_len;
  hp.wg0 = 0;
  hp.nwg = p.shape.nwg;
  hp.per_wg = p.shape.per_wg;
  hp.g1 = p.shape.g1;
  hp.ng = p.shape.ng;
  hp.slots2 = (p.shape.g1 || p.working_set > 0) ? reinterpret_cast<u64 *>(ws + p.off_slots2) : nullptr;
  std::vector<int32_t> hwgp(std::max(p.shape.nwg + 1, p.auto_q ? p.pair_shape.nwg : 0), 0);
  HIPCHK(hipMemcpyAsync(dprob, &hp, sizeof(Prob), hipMemcpyHostToDevice, stream));
  HIPCHK(hipMemcpyAsync(wgp, hwgp.data(), 4 * hwgp.size(), hipMemcpyHostToDevice, stream));
  HIPCHK(hipMemsetAsync(err, 0, 16, stream));
  s0 = check_finite(X, n * d, err + 2, stream);
  if (s0 != SVM_OK) return s0;
  if (p.cache_cap)
    HIPCHK(hipMemsetAsync(ws + p.off_tags, 0xff, 4LL * p.cache_cap * p.shape.nwg, stream));
  const double t_upload = std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();

  Timer tg, ts, tf;
  HIPCHK(tg.init(timed));
  HIPCHK(ts.init(timed));
  HIPCHK(tf.init(timed));
  HIPCHK(tg.start(stream));
  double *sqn = p.gram ? nullptr : reinterpret_cast<double *>(ws + p.off_sqn);
  if (p.gram && p.off_split >= 0)
    HIPCHK(launch_gram_split(X, n, d, (float)gamma, G, p.ld, ws + p.off_split, stream));
  else if (p.gram)
    HIPCHK(launch_gram(X, n, d, (float)gamma, G, p.ld, stream));
  else if (p.working_set > 0)
    HIPCHK(launch_split_rows(X, n, d, split_views(ws + p.off_split, n, d), stream));
  else
    HIPCHK(launch_row_norms(X, n, d, sqn, stream));
  HIPCHK(tg.stop(stream));

  HIPCHK(ts.start(stream));
  HIPCHK(launch_solver_init(dprob, 1, n, stream));
  if (r.alpha_init) {
    HIPCHK(hipMemcpyAsync(alpha, warm_a.data(), 8 * n, hipMemcpyHostToDevice, stream));
    if (r.f_init) {
      HIPCHK(hipMemcpyAsync(f, warm_f.data(), 8 * n, hipMemcpyHostToDevice, stream));
    } else {
      const int64_t nsv = (int64_t)warm_sv.size();
      double *dcoef = reinterpret_cast<double *>(ws + p.off_warm);
      int32_t *dsv = reinterpret_cast<int32_t *>(ws + p.off_warm + 8 * n);
      if (nsv > 0) {
        HIPCHK(hipMemcpyAsync(dcoef, warm_coef.data(), 8 * nsv, hipMemcpyHostToDevice, stream));
        HIPCHK(hipMemcpyAsync(dsv, warm_sv.data(), 4 * nsv, hipMemcpyHostToDevice, stream));
      }
      HIPCHK(launch_f_from_alpha(dsv, dcoef, nsv, y, n, G, p.ld, X, d, gamma, f, stream));
    }
  }
  SolveParams sp{};
  sp.probs = dprob;
  sp.wg_prob = wgp;
  sp.C = C;
  sp.tol = tol;
  sp.gamma = gamma;
  sp.max_iter = r.max_iter;
  sp.steps = r.check_every;
  sp.gram = G;
  sp.ld = p.ld;
  sp.X = X;
  sp.sqn = sqn;
  sp.d = d;
  sp.cache = p.cache_cap ? reinterpret_cast<float *>(ws + p.off_cache) : nullptr;
  sp.cache_tags = p.cache_cap ? reinterpret_cast<int32_t *>(ws + p.off_tags) : nullptr;
  sp.cache_cap = p.cache_cap;
  sp.max_per_wg = p.shape.per_wg;
  sp.second_order = r.selection == SVM_SELECT_SECOND_ORDER ? 1 : 0;
  sp.res_rows = 0;
  // row path of the pair solver: rows of X each workgroup keeps in LDS
  auto resident = [&](SolveParams &q, const Shape &sh) -> svm_status {
    q.res_rows = 0;
    if (!p.gram && r.resident_rows >= 0) {
      const int64_t fit = solver_res_rows_max(q, sh.per_thread);
      if (fit < 0) return fail(SVM_EDEVICE, "row path: LDS capacity query failed");
      int64_t res = std::min<int64_t>(fit, sh.per_wg);
      if (r.resident_rows > 0) res = std::min<int64_t>(res, r.resident_rows);
      q.res_rows = (int32_t)res;
    }
    return SVM_OK;
  };
  if (p.working_set == 0) {
    s0 = resident(sp, p.shape);
    if (s0 != SVM_OK) return s0;
  }
  sp.spin_limit = spin_ticks();
  sp.error = err;
  int32_t launches = 0;
  std::vector<Ctl> hc;
  double t_kernel = 0.0;
  int64_t *d_rounds = reinterpret_cast<int64_t *>(ws + p.off_rounds);
  svm_status s1;
  int32_t schedule = p.working_set > 0 ? 1 : 0;  // svm_stats.schedule
  int64_t h_rounds = 0;
  if (p.working_set > 0) {
    HIPCHK(hipMemsetAsync(slots, 0, 8 * p.slot_words, stream));
    HIPCHK(hipMemsetAsync(ws + p.off_slots2, 0, 8 * p.slot2_words, stream));
    HIPCHK(hipMemsetAsync(d_rounds, 0, 8, stream));
    WsParams wp{};
    wp.sp = sp;
    wp.rounds = d_rounds;
    wp.frac = WS_FRAC;
    wp.q = p.working_set;
    wp.max_inner = WS_INNER_PER_Q * p.working_set;
    wp.round_end = INT64_MAX;
    if (!p.gram) {
      wp.split = split_views(ws + p.off_split, n, d);
      wp.cexp = (float)(-gamma * 1.4426950408889634);
    }
    const int32_t nwg = p.shape.nwg + (p.shape.nwg > 1 ? 1 : 0);  // owners and the solving workgroup
    auto ws_launch = [&](int32_t *maxres) { return launch_ws_solver(wp, nwg, stream, maxres); };
    bool go_on = true;
    if (p.auto_q) {
      // the probe: the first WS_AUTO_PROBE_ROUNDS rounds (in as many launches as the host check
      // cadence makes), then the rule
      wp.round_end = WS_AUTO_PROBE_ROUNDS;
      auto probed = [&]() {
        if (hipMemcpy(&h_rounds, d_rounds, 8, hipMemcpyDeviceToHost) != hipSuccess) return true;
        return h_rounds >= WS_AUTO_PROBE_ROUNDS;
      };
      s1 = run_launches(ws_launch, err, 1, nwg, ctl, stream, &launches, hc, &t_kernel, timed, probed);
      if (s1 != SVM_OK) return s1;
      if (hc[0].status == ST_RUNNING) {
        HIPCHK(hipMemcpy(&h_rounds, d_rounds, 8, hipMemcpyDeviceToHost));
        go_on = (double)hc[0].t >= p.auto_min_steps * (double)h_rounds;
      } else {
        go_on = false;  // solved within the probe
      }
      wp.round_end = INT64_MAX;
    }
    if (go_on) {
      s1 = run_launches(ws_launch, err, 1, nwg, ctl, stream, &launches, hc, &t_kernel, timed);
    } else if (hc[0].status == ST_RUNNING) {
      // the pair solver takes over from the state the rounds left: f and alpha in the workspace
      // and the caller's alpha, the step count in the control block.  Its exchange words are
      // stamped so that no current stamp matches them (the next two steps read stamps t + 1
      // and t + 2); the row path gets its squared row norms.
      schedule = 2;
      const Shape &sh = p.pair_shape;
      hp.nwg = sh.nwg;
      hp.per_wg = sh.per_wg;
      hp.g1 = sh.g1;
      hp.ng = sh.ng;
      hp.slots2 = reinterpret_cast<u64 *>(ws + p.off_slots2);
      HIPCHK(hipMemcpyAsync(dprob, &hp, sizeof(Prob), hipMemcpyHostToDevice, stream));
      const uint32_t stale = (uint32_t)((hc[0].t + 9) & 15) << 28;
      HIPCHK(hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(slots), stale, 2 * p.slot_words, stream));
      HIPCHK(hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(ws + p.off_slots2), stale, 2 * p.slot2_words, stream));
      if (!p.gram) HIPCHK(launch_row_norms(X, n, d, sqn, stream));
      sp.max_per_wg = sh.per_wg;
      s0 = resident(sp, sh);
      if (s0 != SVM_OK) return s0;
      s1 = run_solver(sp, 1, sh.nwg, sh.per_thread, p.gram, ctl, stream, &launches, hc, &t_kernel, timed);
    } else {
      s1 = SVM_OK;
    }
  } else {
    s1 = run_solver(sp, 1, p.shape.nwg, p.shape.per_thread, p.gram, ctl, stream, &launches, hc, &t_kernel, timed);
  }
  if (s1 != SVM_OK) return s1;
  if (p.working_set > 0) HIPCHK(hipMemcpyAsync(&h_rounds, d_rounds, 8, hipMemcpyDeviceToHost, stream));
  HIPCHK(ts.stop(stream));

  HIPCHK(tf.start(stream));
  HIPCHK(launch_finalize(dprob, 1, C, fin, stream));
  double hfin[4];
  HIPCHK(hipMemcpyAsync(hfin, fin, sizeof(hfin), hipMemcpyDeviceToHost, stream));
  HIPCHK(hipStreamSynchronize(stream));
  if (r.trace_len) {
    const int64_t steps = std::min<int64_t>(r.trace_len, (p.working_set > 0 ? h_rounds : hc[0].t) + 1);
    if (r.trace_ws) HIPCHK(hipMemcpyAsync(r.trace_ws, tul, 4 * 2 * steps, hipMemcpyDeviceToHost, stream));
    if (r.trace_b) HIPCHK(hipMemcpyAsync(r.trace_b, tb, 8 * 2 * steps, hipMemcpyDeviceToHost, stream));
  }
  if (r.f_out) HIPCHK(hipMemcpyAsync(r.f_out, f, 8 * n, hipMemcpyDeviceToDevice, stream));
  HIPCHK(tf.stop(stream));
  HIPCHK(hipStreamSynchronize(stream));

  const Ctl &c = hc[0];
  *b = 0.5 * (c.b_up + c.b_low);
  if (st) {
    st->iterations = c.t;
    st->n_sv = (int64_t)hfin[2];
    st->n_bound_sv = (int64_t)hfin[3];
    st->b_up = c.b_up;
    st->b_low = c.b_low;
    st->dual_obj = 0.5 * hfin[0] - 0.5 * hfin[1];
    st->gram_used = p.gram ? 1 : 0;
    st->launches = launches;
    st->t_gram = tg.seconds();
    st->t_solve = ts.seconds();
    st->t_finalize = tf.seconds();
    st->t_total = std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();
    st->t_kernel = t_kernel;
    st->rounds = p.working_set > 0 ? h_rounds : 0;
    st->resident_rows = sp.res_rows;
    st->schedule = schedule;
    st->t_upload = t_upload;
  }
  return c.status == ST_MAXITER ? SVM_NOT_CONVERGED : SVM_OK;
}

svm_status svm_train(const float *X, const int32_t *y, int64_t n, int64_t d, double C, double gamma, double tol,
                     double *alpha, double *b, void *workspace, int64_t workspace_bytes, const svm_options *o,
                     svm_stats *st) {
  return train_impl(X, y, n, d, C, gamma, tol, alpha, b, workspace, workspace_bytes, o, st, false);
}

svm_status svm_train_static(const float *X, const int32_t *y, int64_t n, int64_t d, double C, double gamma,
                            double tol, double *alpha, double *b, const svm_options *o, svm_stats *st) {
  return train_impl(X, y, n, d, C, gamma, tol, alpha, b, nullptr, 0, o, st, true);
}

int64_t svm_predict_workspace_bytes(int64_t n, int64_t d, int64_t m) {
  if (n < 1 || d < 1 || m < 0 || n > 0x7ffffffeLL || m > (INT64_MAX / 8) / 64 / std::max<int64_t>(n, 1)) return -1;
  return predict_scratch_bytes(n, n, 1, m, d);
}

svm_status svm_predict(const float *X_train, const int32_t *y, const double *alpha, double b, int64_t n, int64_t d,
                       double gamma, const float *X_test, int64_t m, double *dec, void *workspace,
                       int64_t workspace_bytes, const svm_options *o) {
  g_err.clear();
  if (n < 1 || d < 1 || m < 0) return fail(SVM_EINVAL, "need n >= 1, d >= 1, m >= 0");
  if (!X_train || !y || !alpha || (m > 0 && (!X_test || !dec))) return fail(SVM_EINVAL, "NULL pointer argument");
  if (!finite_pos(gamma) || !std::isfinite(b)) return fail(SVM_EINVAL, "gamma must be finite and > 0, b finite");
  if (n > 0x7ffffffeLL) return fail(SVM_ENOMEM, "n=%lld exceeds the 32-bit sample index", (long long)n);
  if (d > (INT64_MAX / 8) / std::max<int64_t>(n, m)) return fail(SVM_EINVAL, "sizes overflow 64-bit byte counts");
  Opts r;
  if (!resolve(o, n, &r)) return fail(SVM_EINVAL, "bad options");
  if (m == 0) return SVM_OK;
  const int64_t need = svm_predict_workspace_bytes(n, d, m);
  if (need < 0) return fail(SVM_EINVAL, "sizes overflow 64-bit byte counts");
  if (!workspace || workspace_bytes < need)
    return fail(SVM_EWORKSPACE, "workspace of %lld bytes needed, %lld given", (long long)need, (long long)workspace_bytes);
  PredictWs pw = predict_scratch(workspace, n, n, 1, m, d);
  HIPCHK(predict_prepare(pw, r, X_train, n, X_test, m, d));
  PredPair pp{};
  pp.off0 = 0;
  pp.len0 = n;
  pp.off1 = n;
  pp.y = y;
  pp.perm = nullptr;
  pp.alpha_off = 0;
  pp.ntr = n;
  pp.sv_off = 0;
  pp.part_off = 0;
  pp.b = b;
  pp.nsplit = predict_splits(m, n);
  HIPCHK(hipMemcpyAsync(pw.ps.pairs, &pp, sizeof(pp), hipMemcpyHostToDevice, r.stream));
  HIPCHK(launch_predict_pairs(X_train, d, 1, pp.nsplit, alpha, gamma, X_test, m, dec, 1, pw.ps, r.stream));
  HIPCHK(hipStreamSynchronize(r.stream));
  return SVM_OK;
}

int64_t svm_train_ovo_workspace_bytes(int64_t n, int64_t d, int32_t k, const svm_options *o) {
  Opts r;
  if (!resolve(o, n, &r)) return -1;
  OvoPlan p;
  if (plan_ovo(n, d, k, r, &p) != SVM_OK) return -1;
  return p.total;
}

svm_status svm_train_ovo(const float *X, const int32_t *label, int64_t n, int64_t d, int32_t k, double C,
                         double gamma, double tol, double *alpha, double *b, void *workspace,
                         int64_t workspace_bytes, const svm_options *o, svm_stats *st) {
  const auto t_start = std::chrono::steady_clock::now();
  g_err.clear();
  if (!X || !label || !alpha || !b) return fail(SVM_EINVAL, "NULL pointer argument");
  if (!finite_pos(C) || !finite_pos(gamma) || !finite_pos(tol))
    return fail(SVM_EINVAL, "C, gamma and tol must be finite and > 0");
  Opts r;
  if (!resolve(o, n, &r)) return fail(SVM_EINVAL, "bad options");
  if (r.alpha_init || r.f_init) return fail(SVM_EINVAL, "alpha_init / f_init: binary training only");
  OvoPlan p;
  svm_status s0 = plan_ovo(n, d, k, r, &p);
  if (s0 != SVM_OK) return s0;
  if (!workspace || workspace_bytes < p.total)
    return fail(SVM_EWORKSPACE, "workspace of %lld bytes needed, %lld given", (long long)p.total,
                (long long)workspace_bytes);
  hipStream_t stream = r.stream;
  std::vector<int32_t> perm;
  std::vector<int64_t> start, cnt;
  s0 = class_sort(label, n, k, stream, perm, start, cnt);
  if (s0 != SVM_OK) return s0;

  char *ws = static_cast<char *>(workspace);
  int32_t *dperm = reinterpret_cast<int32_t *>(ws + p.off_perm);
  float *Xs = reinterpret_cast<float *>(ws + p.off_xs);
  double *f = reinterpret_cast<double *>(ws + p.off_f);
  float *G = p.gram ? reinterpret_cast<float *>(ws + p.off_gram) : nullptr;
  Ctl *ctl = reinterpret_cast<Ctl *>(ws + p.off_ctl);
  Prob *dprob = reinterpret_cast<Prob *>(ws + p.off_prob);
  int32_t *wgp = reinterpret_cast<int32_t *>(ws + p.off_wgp);
  u64 *slots = reinterpret_cast<u64 *>(ws + p.off_slots);
  u64 *slots2 = reinterpret_cast<u64 *>(ws + p.off_slots2);
  double *fin = reinterpret_cast<double *>(ws + p.off_fin);
  int32_t *err = reinterpret_cast<int32_t *>(ws + p.off_err);

  std::vector<Prob> hp(p.P);
  std::vector<int32_t> hwgp;
  int64_t max_n = 0;
  int32_t per_thread = 1, wg = 0, max_per_wg = 1;
  // Spread a workgroup budget over the pairs; all pairs run in one cooperative launch.
  auto assign = [&](int64_t budget) -> svm_status {
    hwgp.clear();
    int64_t pack = 0;
    max_n = 0;
    per_thread = 1;
    max_per_wg = 1;
    wg = 0;
    int32_t q = 0;
    for (int32_t a = 0; a < k; ++a)
      for (int32_t bb = a + 1; bb < k; ++bb, ++q) {
        Prob &P = hp[q];
        P = Prob{};
        P.n = cnt[a] + cnt[bb];
        P.off0 = start[a];
        P.len0 = cnt[a];
        P.off1 = start[bb];
        P.y = nullptr;
        P.alpha = alpha + pack;
        P.f = f + pack;
        P.ctl = ctl + q;
        Shape sh;
        const int64_t cap = std::max<int64_t>(1, budget / p.P);
        if (!choose_shape(P.n, p.gram, r.workgroups, r.levels, &sh, cap) || sh.nwg > OVO_MAX_WG_PER_PAIR)
          return fail(SVM_ENOMEM, "pair (%d,%d) too large to place", a, bb);
        P.slots = slots + (size_t)q * 2 * OVO_MAX_WG_PER_PAIR * SLOT_WORDS;
        P.g1 = sh.g1;
        P.ng = sh.ng;
        P.slots2 = sh.g1 ? slots2 + (size_t)q * 2 * OVO_MAX_GROUPS * SLOT_WORDS : nullptr;
        P.wg0 = wg;
        P.nwg = sh.nwg;
        P.per_wg = sh.per_wg;
        per_thread = std::max(per_thread, sh.per_thread);
        max_per_wg = std::max(max_per_wg, sh.per_wg);
        for (int32_t w = 0; w < sh.nwg; ++w) hwgp.push_back(q);
        wg += sh.nwg;
        pack += P.n;
        max_n = std::max(max_n, P.n);
      }
    return SVM_OK;
  };
  // Shrink the budget until the variant the shapes need fits on the device at once; with more
  // pairs than that even at one workgroup each, the pairs run in consecutive batches (one
  // cooperative launch sequence per batch).
  int64_t budget = OVO_TOTAL_WG;
  int32_t capacity = 0;
  for (;;) {
    s0 = assign(budget);
    if (s0 != SVM_OK) return s0;
    SolveParams probe{};
    probe.X = Xs;
    probe.d = d;
    probe.max_per_wg = max_per_wg;
    HIPCHK(launch_solver(probe, 0, per_thread, p.gram, stream, &capacity));
    if (capacity <= 0) return fail(SVM_ENOMEM, "the solver does not fit on the device");
    if (wg <= capacity || budget <= p.P) break;
    budget = std::max<int64_t>(p.P, std::min<int64_t>(budget - 1, capacity));
  }
  std::vector<int32_t> bstart{0}, bwg;  // batch boundaries over the pairs, workgroups per batch
  {
    int32_t acc = 0;
    for (int32_t q = 0; q < p.P; ++q) {
      if (hp[q].nwg > capacity)
        return fail(SVM_ENOMEM, "pair %d needs %d workgroups, the device holds %d at once", q, hp[q].nwg, capacity);
      if (acc + hp[q].nwg > capacity) {
        bwg.push_back(acc);
        bstart.push_back(q);
        acc = 0;
      }
      hp[q].wg0 = acc;  // relative to its batch's launch
      acc += hp[q].nwg;
    }
    bwg.push_back(acc);
    bstart.push_back(p.P);
    hwgp.clear();  // workgroup -> pair index within its batch
    for (size_t bi = 0; bi + 1 < bstart.size(); ++bi)
      for (int32_t q = bstart[bi]; q < bstart[bi + 1]; ++q)
        for (int32_t w = 0; w < hp[q].nwg; ++w) hwgp.push_back(q - bstart[bi]);
  }
  HIPCHK(hipMemcpyAsync(dperm, perm.data(), 4 * n, hipMemcpyHostToDevice, stream));
  HIPCHK(hipMemcpyAsync(dprob, hp.data(), sizeof(Prob) * hp.size(), hipMemcpyHostToDevice, stream));
  HIPCHK(hipMemcpyAsync(wgp, hwgp.data(), 4 * hwgp.size(), hipMemcpyHostToDevice, stream));
  HIPCHK(hipMemsetAsync(err, 0, 16, stream));
  HIPCHK(launch_gather_rows(X, d, dperm, n, Xs, stream));
  s0 = check_finite(X, n * d, err + 2, stream);  // its synchronisation also ends the class-sorted copy
  if (s0 != SVM_OK) return s0;
  const double t_upload = std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();

  Timer tg, ts, tf;
  HIPCHK(tg.init());
  HIPCHK(ts.init());
  HIPCHK(tf.init());
  HIPCHK(tg.start(stream));
  double *sqn = p.gram ? nullptr : reinterpret_cast<double *>(ws + p.off_sqn);
  if (p.gram && p.off_split >= 0)
    HIPCHK(launch_gram_split(Xs, n, d, (float)gamma, G, p.ld, ws + p.off_split, stream));
  else if (p.gram)
    HIPCHK(launch_gram(Xs, n, d, (float)gamma, G, p.ld, stream));
  else
    HIPCHK(launch_row_norms(Xs, n, d, sqn, stream));
  HIPCHK(tg.stop(stream));
  HIPCHK(ts.start(stream));
  HIPCHK(launch_solver_init(dprob, p.P, max_n, stream));
  SolveParams sp{};
  sp.probs = dprob;
  sp.wg_prob = wgp;
  sp.C = C;
  sp.tol = tol;
  sp.gamma = gamma;
  sp.max_iter = r.max_iter;
  sp.steps = r.check_every;
  sp.gram = G;
  sp.ld = p.ld;
  sp.X = Xs;
  sp.sqn = sqn;
  sp.d = d;
  sp.max_per_wg = max_per_wg;
  sp.second_order = r.selection == SVM_SELECT_SECOND_ORDER ? 1 : 0;
  sp.spin_limit = spin_ticks();
  sp.error = err;
  int32_t launches = 0;
  std::vector<Ctl> hc;
  double t_kernel = 0.0;
  int32_t woff = 0;
  for (size_t bi = 0; bi + 1 < bstart.size(); ++bi) {
    SolveParams sb = sp;
    sb.probs = dprob + bstart[bi];
    sb.wg_prob = wgp + woff;
    std::vector<Ctl> hb;
    int32_t lb = 0;
    double tb = 0.0;
    svm_status s1 = run_solver(sb, bstart[bi + 1] - bstart[bi], bwg[bi], per_thread, p.gram, ctl + bstart[bi], stream,
                               &lb, hb, &tb);
    if (s1 != SVM_OK) return s1;
    launches += lb;
    t_kernel += tb;
    hc.insert(hc.end(), hb.begin(), hb.end());
    woff += bwg[bi];
  }
  HIPCHK(ts.stop(stream));
  HIPCHK(tf.start(stream));
  HIPCHK(launch_finalize(dprob, p.P, C, fin, stream));
  std::vector<double> hfin(4 * (size_t)p.P);
  HIPCHK(hipMemcpyAsync(hfin.data(), fin, 8 * hfin.size(), hipMemcpyDeviceToHost, stream));
  HIPCHK(tf.stop(stream));
  HIPCHK(hipStreamSynchronize(stream));
  bool maxed = false;
  const double t_total = std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();
  for (int32_t q2 = 0; q2 < p.P; ++q2) {
    b[q2] = 0.5 * (hc[q2].b_up + hc[q2].b_low);
    maxed = maxed || hc[q2].status == ST_MAXITER;
    if (st) {
      svm_stats &S = st[q2];
      S.iterations = hc[q2].t;
      S.n_sv = (int64_t)hfin[4 * q2 + 2];
      S.n_bound_sv = (int64_t)hfin[4 * q2 + 3];
      S.b_up = hc[q2].b_up;
      S.b_low = hc[q2].b_low;
      S.dual_obj = 0.5 * hfin[4 * q2] - 0.5 * hfin[4 * q2 + 1];
      S.gram_used = p.gram ? 1 : 0;
      S.launches = launches;
      S.t_gram = tg.seconds();
      S.t_solve = ts.seconds();
      S.t_finalize = tf.seconds();
      S.t_total = t_total;
      S.t_kernel = t_kernel;
      S.rounds = 0;
      S.resident_rows = 0;
      S.schedule = 0;
      S.t_upload = t_upload;
    }
  }
  return maxed ? SVM_NOT_CONVERGED : SVM_OK;
}

int64_t svm_predict_ovo_workspace_bytes(int64_t n, int64_t d, int32_t k, int64_t m) {
  if (n < 2 || d < 1 || k < 2 || k > MAX_CLASSES || m < 0 || n > 0x7ffffffeLL) return -1;
  const int64_t P = (int64_t)k * (k - 1) / 2;
  return round_up(4 * n, ALIGN) + predict_scratch_bytes(n, n, std::min<int64_t>(P, PREDICT_PAIRS_MAX), m, d);
}

svm_status svm_predict_ovo(const float *X, const int32_t *label, int64_t n, int64_t d, int32_t k,
                           const double *alpha, const double *b, double gamma, const float *X_test, int64_t m,
                           double *dec, int32_t *pred, void *workspace, int64_t workspace_bytes,
                           const svm_options *o) {
  g_err.clear();
  if (n < 2 || d < 1 || m < 0) return fail(SVM_EINVAL, "need n >= 2, d >= 1, m >= 0");
  if (k < 2 || k > MAX_CLASSES) return fail(SVM_EINVAL, "k=%d must be in [2, %d]", k, MAX_CLASSES);
  if (!X || !label || !alpha || !b || (m > 0 && (!X_test || !dec || !pred))) return fail(SVM_EINVAL, "NULL pointer");
  if (!finite_pos(gamma)) return fail(SVM_EINVAL, "gamma must be finite and > 0");
  Opts r;
  if (!resolve(o, n, &r)) return fail(SVM_EINVAL, "bad options");
  const int64_t need = svm_predict_ovo_workspace_bytes(n, d, k, m);
  if (!workspace || workspace_bytes < need) return fail(SVM_EWORKSPACE, "workspace of %lld bytes needed", (long long)need);
  const int32_t P = k * (k - 1) / 2;
  for (int32_t q = 0; q < P; ++q)
    if (!std::isfinite(b[q])) return fail(SVM_EINVAL, "b[%d] is not finite", q);
  std::vector<int32_t> perm;
  std::vector<int64_t> start, cnt;
  svm_status s0 = class_sort(label, n, k, r.stream, perm, start, cnt);
  if (s0 != SVM_OK) return s0;
  if (m == 0) return SVM_OK;
  int32_t *dperm = static_cast<int32_t *>(workspace);
  const int32_t chunk = std::min<int32_t>(P, PREDICT_PAIRS_MAX);
  PredictWs pw = predict_scratch(static_cast<char *>(workspace) + round_up(4 * n, ALIGN), n, n, chunk, m, d);
  HIPCHK(predict_prepare(pw, r, X, n, X_test, m, d));
  HIPCHK(hipMemcpyAsync(dperm, perm.data(), 4 * n, hipMemcpyHostToDevice, r.stream));
  // the pairs in chunks of up to PREDICT_PAIRS_MAX, each chunk one launch per stage
  std::vector<PredPair> pp;
  pp.reserve(P);
  int64_t pack = 0;
  for (int32_t a = 0; a < k; ++a)
    for (int32_t bb = a + 1; bb < k; ++bb) {
      PredPair e{};
      e.off0 = start[a];
      e.len0 = cnt[a];
      e.off1 = start[bb];
      e.y = nullptr;
      e.perm = dperm;
      e.alpha_off = pack;
      e.ntr = cnt[a] + cnt[bb];
      e.b = b[pp.size()];
      e.nsplit = predict_splits(m, e.ntr);
      pp.push_back(e);
      pack += e.ntr;
    }
  for (int32_t c0 = 0; c0 < P; c0 += chunk) {
    const int32_t np = std::min<int32_t>(chunk, P - c0);
    int nsplit_max = 1;
    int64_t sv = 0, part = 0;
    for (int32_t q = c0; q < c0 + np; ++q) {
      pp[q].sv_off = sv;
      pp[q].part_off = part;
      sv += pp[q].ntr;
      part += (int64_t)pp[q].nsplit * m;
      nsplit_max = std::max(nsplit_max, (int)pp[q].nsplit);
    }
    HIPCHK(hipMemcpyAsync(pw.ps.pairs, pp.data() + c0, sizeof(PredPair) * np, hipMemcpyHostToDevice, r.stream));
    HIPCHK(launch_predict_pairs(X, d, np, nsplit_max, alpha, gamma, X_test, m, dec + c0, P, pw.ps, r.stream));
  }
  HIPCHK(launch_ovo_vote(dec, m, k, pred, r.stream));
  HIPCHK(hipStreamSynchronize(r.stream));
  return SVM_OK;
}

svm_status svm_kernel_rows(const float *X, int64_t n, int64_t d, double gamma, const int64_t *rows, int64_t r,
                           float *out, const svm_options *o) {
  g_err.clear();
  if (!X || !rows || !out) return fail(SVM_EINVAL, "NULL pointer argument");
  if (n < 1 || d < 1 || r < 1) return fail(SVM_EINVAL, "need n, d, r >= 1");
  if (!finite_pos(gamma)) return fail(SVM_EINVAL, "gamma must be finite and > 0");
  if (d > (INT64_MAX / 8) / n || r > INT64_MAX / 8 / n) return fail(SVM_EINVAL, "sizes overflow 64-bit byte counts");
  if (2 * 4 * d > LDS_BYTES) return fail(SVM_EINVAL, "d too large for the staged rows");
  Opts op;
  if (!resolve(o, n, &op)) return fail(SVM_EINVAL, "bad options");
  std::vector<int64_t> h(r);
  HIPCHK(hipMemcpyAsync(h.data(), rows, 8 * r, hipMemcpyDeviceToHost, op.stream));
  HIPCHK(hipStreamSynchronize(op.stream));
  for (int64_t q = 0; q < r; ++q)
    if (h[q] < 0 || h[q] >= n) return fail(SVM_EINVAL, "rows[%lld] = %lld out of range", (long long)q, (long long)h[q]);
  HIPCHK(launch_kernel_rows(X, n, d, gamma, rows, r, out, op.stream));
  HIPCHK(hipStreamSynchronize(op.stream));
  return SVM_OK;
}

int64_t svm_gram_workspace_bytes(int64_t n, int64_t d, const svm_options *o) {
  Opts op;
  if (n < 1 || d < 1 || d > (INT64_MAX / 8) / n || !resolve(o, n, &op)) return -1;
  return op.gram_mfma == SVM_MFMA_SPLIT_F16 ? gram_split_scratch_bytes(n, d) : 0;
}

svm_status svm_gram(const float *X, int64_t n, int64_t d, double gamma, float *G, int64_t ld, void *workspace,
                    int64_t workspace_bytes, const svm_options *o) {
  g_err.clear();
  if (!X || !G) return fail(SVM_EINVAL, "NULL pointer argument");
  if (n < 1 || d < 1 || ld < n) return fail(SVM_EINVAL, "need n, d >= 1 and ld >= n");
  if (!finite_pos(gamma)) return fail(SVM_EINVAL, "gamma must be finite and > 0");
  if (d > (INT64_MAX / 8) / n || ld > (INT64_MAX / 8) / n) return fail(SVM_EINVAL, "sizes overflow 64-bit byte counts");
  Opts op;
  if (!resolve(o, n, &op)) return fail(SVM_EINVAL, "bad options");
  if (op.gram_mfma == SVM_MFMA_SPLIT_F16) {
    const int64_t need = gram_split_scratch_bytes(n, d);
    if (!workspace || workspace_bytes < need)
      return fail(SVM_EWORKSPACE, "workspace of %lld bytes needed, %lld given", (long long)need,
                  (long long)workspace_bytes);
    HIPCHK(launch_gram_split(X, n, d, (float)gamma, G, ld, workspace, op.stream));
  } else {
    HIPCHK(launch_gram(X, n, d, (float)gamma, G, ld, op.stream));
  }
  HIPCHK(hipStreamSynchronize(op.stream));
  return SVM_OK;
}

}  // extern "C"

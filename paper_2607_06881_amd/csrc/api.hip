// Host side of libmdgemm: argument checks, workspace, job tables, stage timing
// and the exported C ABI declared in include/mdgemm.h.
//
// The product C = A.B of multiple doubles follows the five steps of the
// overview in section 2 of Chen and Verschelde, "Multiple Double Arithmetic on
// NVIDIA Tensor Cores": split into parts, rewrite as products of doubles, run
// the products on the matrix cores, extract the parts, add them into a multiple
// double.  mdgemm_ex enqueues, on one stream, the kernels of the four stages:
// exponents (a1), splits (a2), level GEMMs (a3), accumulation and rounding
// (a4 + a5).
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "internal.h"
#include "mdgemm.h"

static_assert(MDGEMM_MAX_LIMBS == mdg::kMaxLimbs && MDGEMM_MAX_SLICES == mdg::kMaxSlices &&
                  MDGEMM_Z_WORDS == mdg::kZWords && MDGEMM_SLICE_BITS == mdg::kSliceBits &&
                  MDGEMM_MAX_LEVELS == mdg::kMaxLevels && MDGEMM_MAX_SLICE_BITS == mdg::kMaxSliceBits &&
                  MDGEMM_MAX_DIGIT_BITS == mdg::kMaxDigitBits,
              "the limits of include/mdgemm.h and csrc/internal.h must agree");

namespace {

using mdg::JobTable;

constexpr size_t kAlign = 256;
constexpr int kStages = 4;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---- exactness: pairs_t * k * (2^w - 1)^2 < 2^53 for every kept level t ------

// Pairs (p, q), 0 <= p, q < S, with p + q <= T.
int pair_count(int S, int T) {
  int n = 0;
  for (int t = 0; t <= T; ++t) {
    int lo = t - (S - 1) > 0 ? t - (S - 1) : 0;
    int hi = t < S - 1 ? t : S - 1;
    if (hi >= lo) n += hi - lo + 1;
  }
  return n;
}

int max_pairs(int S, int T) {
  int best = 0;
  for (int t = 0; t <= T; ++t) {
    int lo = t - (S - 1) > 0 ? t - (S - 1) : 0;
    int hi = t < S - 1 ? t : S - 1;
    if (hi - lo + 1 > best) best = hi - lo + 1;
  }
  return best;
}

bool exact_ok(int64_t k, int pairs, int w) {
  const uint64_t dmax = (1ull << w) - 1ull;
  const unsigned __int128 lhs =
      static_cast<unsigned __int128>(pairs) * static_cast<unsigned __int128>(k) * (dmax * dmax);
  return lhs < (static_cast<unsigned __int128>(1) << 53);
}

bool width_ok(int S, int w) { return S >= 1 && S <= MDGEMM_MAX_SLICES && w >= 1 && w <= mdg::kMaxSliceBits &&
                                     S * w <= mdg::kMaxDigitBits; }

// w (levels - 1) + 55 bits must fit the widest accumulation (kZWords words)
bool levels_ok(int levels, int w) { return levels >= 1 && levels <= mdg::kMaxLevels && mdg::accum_words(levels, w) <= mdg::kZWords; }

// ---- job tables ---------------------------------------------------------------

// Levels t = 0..T, heaviest (most pairs) first so that long K loops start early.
JobTable level_jobs(int S, int T) {
  JobTable jt;
  std::memset(&jt, 0, sizeof jt);
  std::vector<int> order;
  for (int t = 0; t <= T; ++t) order.push_back(t);
  auto npairs = [S](int t) {
    int lo = t - (S - 1) > 0 ? t - (S - 1) : 0;
    int hi = t < S - 1 ? t : S - 1;
    return hi - lo + 1;
  };
  // stable sort by decreasing pair count
  for (size_t i = 1; i < order.size(); ++i)
    for (size_t j = i; j > 0 && npairs(order[j]) > npairs(order[j - 1]); --j) std::swap(order[j], order[j - 1]);
  jt.njobs = static_cast<int>(order.size());
  for (int j = 0; j < jt.njobs; ++j) {
    int t = order[j];
    int lo = t - (S - 1) > 0 ? t - (S - 1) : 0;
    jt.p_first[j] = static_cast<uint16_t>(lo);
    jt.q_first[j] = static_cast<uint16_t>(t - lo);
    jt.npairs[j] = static_cast<uint16_t>(npairs(t));
    jt.out[j] = static_cast<uint16_t>(t);
  }
  return jt;
}

// Every pair (p, q) with p + q <= T, written to plane p*S + q; one table per
// launch of at most kMaxJobs pairs.
std::vector<JobTable> pair_jobs(int S, int T) {
  std::vector<JobTable> tables;
  for (int p = 0; p < S; ++p)
    for (int q = 0; q < S; ++q) {
      if (p + q > T) continue;
      if (tables.empty() || tables.back().njobs == mdg::kMaxJobs) {
        tables.emplace_back();
        std::memset(&tables.back(), 0, sizeof(JobTable));
      }
      JobTable& jt = tables.back();
      const int j = jt.njobs++;
      jt.p_first[j] = static_cast<uint16_t>(p);
      jt.q_first[j] = static_cast<uint16_t>(q);
      jt.npairs[j] = 1;
      jt.out[j] = static_cast<uint16_t>(p * S + q);
    }
  return tables;
}

// ---- options ----------------------------------------------------------------

struct Resolved {
  int S = 0, T = 0, w = mdg::kSliceBits;
  hipStream_t stream = nullptr;
  unsigned flags = 0;
};

// Extra digits for elements down to range_bits below their line's exponent.
inline int range_digits(int range_bits, int w) { return (range_bits + w - 1) / w; }

// The cutoff selector applied to S0 base digits and D range digits.
int cutoff_for(int cutoff, int S0, int D) {
  if (cutoff == MDGEMM_CUTOFF_DEFAULT) return S0 - 1 + 2 * D;
  if (cutoff == MDGEMM_CUTOFF_ALL) return 2 * (S0 + D) - 2;
  return cutoff;
}

// Adaptive width: among w = 13..26 with S0 = ceil(52 L / w) base digits (the digit
// bits of four 13-bit digits per limb), D = ceil(range_bits / w) extra digits,
// S = S0 + D and the requested cutoff, those that are valid and whose levels stay
// exact, the fewest pairs, the wider digit on a tie.  Returns false when none
// qualifies.
bool auto_width(int limbs, int64_t k, int range_bits, int cutoff, int* w_out, int* S0_out) {
  int best_pairs = 0;
  bool found = false;
  for (int w = mdg::kSliceBits; w <= mdg::kMaxSliceBits; ++w) {
    const int S0 = (4 * mdg::kSliceBits * limbs + w - 1) / w, D = range_digits(range_bits, w);
    const int S = S0 + D, T = cutoff_for(cutoff, S0, D);
    if (!width_ok(S, w) || T < 0 || T > 2 * S - 2 || !levels_ok(T + 1, w) || !exact_ok(k, max_pairs(S, T), w))
      continue;
    const int pairs = pair_count(S, T);
    if (!found || pairs <= best_pairs) {
      best_pairs = pairs;
      *w_out = w;
      *S0_out = S0;
      found = true;
    }
  }
  return found;
}

// Digit width, digit count and cutoff of a product with reduction length k.
int resolve(int limbs, int64_t k, const mdgemm_opts* opts, Resolved* r) {
  if (limbs < 1 || limbs > MDGEMM_MAX_LIMBS) return MDGEMM_EINVAL;
  const int bits = opts ? opts->slice_bits : 0;
  const int slices = opts ? opts->slices : 0;
  const int range_bits = opts ? opts->range_bits : 0;
  if (slices < 0 || range_bits < 0 || range_bits > mdg::kMaxDigitBits) return MDGEMM_EINVAL;
  if (bits == MDGEMM_SLICE_BITS_AUTO) {
    if (slices != 0) return MDGEMM_EINVAL;
    if (!auto_width(limbs, k, range_bits, opts->cutoff, &r->w, &r->S)) return MDGEMM_EEXACT;
  } else if (bits == 0 || bits == mdg::kSliceBits) {
    r->w = mdg::kSliceBits;
    int spl = opts ? opts->slices_per_limb : 0;
    if (spl == 0) spl = 4;
    if (spl < 0) return MDGEMM_EINVAL;
    r->S = slices ? slices : spl * limbs;
  } else if (bits >= 1 && bits <= mdg::kMaxSliceBits) {
    r->w = bits;
    r->S = slices ? slices : (4 * mdg::kSliceBits * limbs + bits - 1) / bits;
  } else {
    return MDGEMM_EINVAL;
  }
  // range balancing: D more digits on the same line grid, and the cutoff raised by
  // 2D so that a product of two elements D digits below their lines' exponents
  // keeps its S0 leading levels
  const int S0 = r->S, D = range_digits(range_bits, r->w);
  r->S = S0 + D;
  if (!width_ok(r->S, r->w)) return MDGEMM_EINVAL;
  const int cutoff = opts ? opts->cutoff : MDGEMM_CUTOFF_DEFAULT;
  if (cutoff < 0 && cutoff != MDGEMM_CUTOFF_DEFAULT && cutoff != MDGEMM_CUTOFF_ALL) return MDGEMM_EINVAL;
  r->T = cutoff_for(cutoff, S0, D);
  if (r->T < 0 || r->T > 2 * r->S - 2) return MDGEMM_EINVAL;
  if (!levels_ok(r->T + 1, r->w)) return MDGEMM_EINVAL;
  r->stream = opts ? static_cast<hipStream_t>(opts->stream) : nullptr;
  r->flags = opts ? opts->flags : 0u;
  return MDGEMM_OK;
}

struct Layout {
  size_t ea = 0, eb = 0, flag = 0, da = 0, db = 0, g = 0, total = 0;
};

bool layout(int64_t m, int64_t n, int64_t k, const Resolved& r, Layout* L) {
  // all products below 2^62 so that size arithmetic cannot overflow
  const double approx = (double)r.S * (double)m * (double)k + (double)r.S * (double)k * (double)n +
                        (double)(r.T + 1) * (double)m * (double)n;
  if (approx * 8.0 > 4.0e18) return false;
  size_t off = 0;
  L->ea = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(m));
  L->eb = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(n));
  L->flag = off;
  off += align_up(sizeof(int32_t));
  L->da = off;
  const size_t kp = static_cast<size_t>(mdg::panel_k(k)), mp = static_cast<size_t>(mdg::panel_mn(m)),
               np = static_cast<size_t>(mdg::panel_mn(n));
  off += align_up(sizeof(double) * static_cast<size_t>(r.S) * kp * mp);
  L->db = off;
  off += align_up(sizeof(double) * static_cast<size_t>(r.S) * kp * np);
  L->g = off;
  off += align_up(sizeof(double) * static_cast<size_t>(r.T + 1) * static_cast<size_t>(m) * static_cast<size_t>(n));
  L->total = off;
  return true;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// ---- library-owned workspace (one per device) ---------------------------------

// One buffer per device, shared by every call that brings no workspace.  Calls
// on different streams are ordered through `last`: a call waits for the
// previous user's event before its first kernel and records the event after its
// last one, all while holding `mu`, so two calls never use the buffer at once.
struct Cache {
  std::mutex mu;
  std::vector<void*> ptr;
  std::vector<size_t> bytes;
  std::vector<hipEvent_t> last;
};
Cache& cache() {
  static Cache c;
  return c;
}

// With c.mu held: the buffer of the current device, grown to `need` bytes.
int cached_workspace(Cache& c, size_t need, void** out, int* dev_out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MDGEMM_EHIP;
  *dev_out = dev;
  if (static_cast<size_t>(dev) >= c.ptr.size()) {
    c.ptr.resize(dev + 1, nullptr);
    c.bytes.resize(dev + 1, 0);
    c.last.resize(dev + 1, nullptr);
  }
  if (!c.last[dev] && hipEventCreateWithFlags(&c.last[dev], hipEventDisableTiming) != hipSuccess) {
    c.last[dev] = nullptr;
    return MDGEMM_EHIP;
  }
  if (c.bytes[dev] < need) {
    if (c.ptr[dev]) {
      if (hipDeviceSynchronize() != hipSuccess) return MDGEMM_EHIP;
      (void)hipFree(c.ptr[dev]);
      c.ptr[dev] = nullptr;
      c.bytes[dev] = 0;
    }
    void* p = nullptr;
    if (hipMalloc(&p, need) != hipSuccess) {
      (void)hipGetLastError();
      return MDGEMM_ENOMEM;
    }
    c.ptr[dev] = p;
    c.bytes[dev] = need;
  }
  *out = c.ptr[dev];
  return MDGEMM_OK;
}

// ---- stage timing ------------------------------------------------------------

struct Timing {
  std::mutex mu;
  hipEvent_t ev[kStages + 1] = {};
  bool created = false;
  bool valid = false;
};
Timing& timing() {
  static Timing t;
  return t;
}

int record(int i, hipStream_t s) {
  Timing& t = timing();
  if (!t.created) {
    for (auto& e : t.ev)
      if (hipEventCreate(&e) != hipSuccess) return MDGEMM_EHIP;
    t.created = true;
  }
  return hipEventRecord(t.ev[i], s) == hipSuccess ? MDGEMM_OK : MDGEMM_EHIP;
}

inline int hip_status(hipError_t e) { return e == hipSuccess ? MDGEMM_OK : MDGEMM_EHIP; }

#define MDG_TRY(expr)              \
  do {                             \
    int st_ = (expr);              \
    if (st_ != MDGEMM_OK) return st_; \
  } while (0)

}  // namespace

extern "C" {

void mdgemm_opts_init(mdgemm_opts* opts) {
  if (!opts) return;
  std::memset(opts, 0, sizeof *opts);
  opts->slices_per_limb = 4;
  opts->cutoff = MDGEMM_CUTOFF_DEFAULT;
  opts->slice_bits = 0;
  opts->slices = 0;
  opts->range_bits = 0;
}

int mdgemm_plan(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts, int* slice_bits, int* slices,
                int* cutoff) {
  Resolved r;
  if (m < 0 || n < 0 || k < 0) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, k, opts, &r));
  if (!exact_ok(k, max_pairs(r.S, r.T), r.w)) return MDGEMM_EEXACT;
  if (slice_bits) *slice_bits = r.w;
  if (slices) *slices = r.S;
  if (cutoff) *cutoff = r.T;
  return MDGEMM_OK;
}

const char* mdgemm_status_string(int status) {
  switch (status) {
    case MDGEMM_OK: return "success";
    case MDGEMM_EINVAL: return "invalid argument";
    case MDGEMM_EEXACT: return "slice sums would reach 2^53 (k too large for exact FP64 accumulation)";
    case MDGEMM_ENOMEM: return "device memory allocation failed";
    case MDGEMM_EHIP: return "HIP runtime error";
    case MDGEMM_EWORKSPACE: return "workspace too small";
    case MDGEMM_ENONFINITE: return "input contains inf or nan";
    default: return "unknown status";
  }
}

size_t mdgemm_workspace_bytes(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts) {
  Resolved r;
  if (m < 0 || n < 0 || k < 0 || resolve(limbs, k, opts, &r) != MDGEMM_OK) return SIZE_MAX;
  if (m == 0 || n == 0 || k == 0) return 0;
  Layout L;
  if (!layout(m, n, k, r, &L)) return SIZE_MAX;
  return L.total;
}

int mdgemm_ex(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
              const mdgemm_opts* opts) {
  Resolved r;
  if (m < 0 || n < 0 || k < 0) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, k, opts, &r));
  if (m == 0 || n == 0) return MDGEMM_OK;
  if (!C || (k > 0 && (!A || !B))) return MDGEMM_EINVAL;
  const size_t abytes = sizeof(double) * limbs * static_cast<size_t>(m) * static_cast<size_t>(k);
  const size_t bbytes = sizeof(double) * limbs * static_cast<size_t>(k) * static_cast<size_t>(n);
  const size_t cbytes = sizeof(double) * limbs * static_cast<size_t>(m) * static_cast<size_t>(n);
  if (k > 0 && (overlaps(C, cbytes, A, abytes) || overlaps(C, cbytes, B, bbytes))) return MDGEMM_EINVAL;
  if (!exact_ok(k, max_pairs(r.S, r.T), r.w)) return MDGEMM_EEXACT;
  hipStream_t s = r.stream;
  const bool timed = (r.flags & MDGEMM_TIME_STAGES) != 0;

  if (k == 0) {
    MDG_TRY(hip_status(mdg::launch_zero_f64(C, static_cast<int64_t>(limbs) * m * n, s)));
    if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
    return MDGEMM_OK;
  }

  Layout L;
  if (!layout(m, n, k, r, &L)) return MDGEMM_EINVAL;
  char* ws = nullptr;
  std::unique_lock<std::mutex> wlock(cache().mu, std::defer_lock);
  int wdev = -1;  // device whose library buffer this call uses, or -1
  if (opts && opts->workspace) {
    if (opts->workspace_bytes < L.total) return MDGEMM_EWORKSPACE;
    ws = static_cast<char*>(opts->workspace);
  } else {
    // a captured graph would keep the library buffer's address, which a later
    // call may free: capture needs a caller workspace
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    MDG_TRY(hip_status(hipStreamIsCapturing(s, &cap)));
    if (cap != hipStreamCaptureStatusNone) return MDGEMM_EINVAL;
    wlock.lock();
    void* p = nullptr;
    MDG_TRY(cached_workspace(cache(), L.total, &p, &wdev));
    MDG_TRY(hip_status(hipStreamWaitEvent(s, cache().last[wdev], 0)));
    ws = static_cast<char*>(p);
  }
  int32_t* EA = reinterpret_cast<int32_t*>(ws + L.ea);
  int32_t* EB = reinterpret_cast<int32_t*>(ws + L.eb);
  int32_t* flag = reinterpret_cast<int32_t*>(ws + L.flag);
  double* DA = reinterpret_cast<double*>(ws + L.da);
  double* DB = reinterpret_cast<double*>(ws + L.db);
  double* G = reinterpret_cast<double*>(ws + L.g);

  auto enqueue = [&]() -> int {
    if (r.flags & MDGEMM_CHECK_FINITE) {
      MDG_TRY(hip_status(mdg::launch_set_i32(flag, 1, 0, s)));
      MDG_TRY(hip_status(mdg::launch_nonfinite_scan(A, static_cast<int64_t>(limbs) * m * k, flag, s)));
      MDG_TRY(hip_status(mdg::launch_nonfinite_scan(B, static_cast<int64_t>(limbs) * k * n, flag, s)));
      int32_t h = 0;
      MDG_TRY(hip_status(hipMemcpyAsync(&h, flag, sizeof h, hipMemcpyDeviceToHost, s)));
      MDG_TRY(hip_status(hipStreamSynchronize(s)));
      if (h) return MDGEMM_ENONFINITE;
    }
    std::unique_lock<std::mutex> tlock(timing().mu, std::defer_lock);
    if (timed) {
      tlock.lock();
      timing().valid = false;
      MDG_TRY(record(0, s));
    }
    // a1: grid exponents per row of A and per column of B
    MDG_TRY(hip_status(mdg::launch_exponents(m, k, 0, A, EA, s)));
    MDG_TRY(hip_status(mdg::launch_exponents(k, n, 1, B, EB, s)));
    if (timed) MDG_TRY(record(1, s));
    // a2: exact splits into S digit planes
    MDG_TRY(hip_status(mdg::launch_split(m, k, limbs, r.S, r.w, 0, A, EA, DA, true, s)));
    MDG_TRY(hip_status(mdg::launch_split(k, n, limbs, r.S, r.w, 1, B, EB, DB, true, s)));
    if (timed) MDG_TRY(record(2, s));
    // a3: level GEMMs on the FP64 matrix cores
    MDG_TRY(hip_status(mdg::launch_slice_gemm(m, n, k, DA, DB, G, level_jobs(r.S, r.T), s)));
    if (timed) MDG_TRY(record(3, s));
    // a4 + a5: exact accumulation and greedy rounding into L limbs
    MDG_TRY(hip_status(mdg::launch_accum_renorm(m, n, limbs, r.T + 1, r.w, G, EA, EB, C, s)));
    if (timed) {
      MDG_TRY(record(4, s));
      timing().valid = true;
    }
    return MDGEMM_OK;
  };
  int st = enqueue();
  if (wdev >= 0) {
    // the next user of the library buffer waits for everything enqueued here,
    // also when enqueueing stopped at an error
    const int rec = hip_status(hipEventRecord(cache().last[wdev], s));
    wlock.unlock();
    if (st == MDGEMM_OK) st = rec;
  }
  if (st != MDGEMM_OK) return st;
  if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
  return MDGEMM_OK;
}

int mdgemm(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C) {
  return mdgemm_ex(m, n, k, limbs, A, B, C, nullptr);
}

int mdgemm_stage_times(float* ms, int count) {
  if (!ms || count < 0) return MDGEMM_EINVAL;
  Timing& t = timing();
  std::lock_guard<std::mutex> lock(t.mu);
  if (!t.valid) return MDGEMM_EINVAL;
  if (hipEventSynchronize(t.ev[kStages]) != hipSuccess) return MDGEMM_EHIP;
  int w = count < kStages ? count : kStages;
  for (int i = 0; i < w; ++i)
    if (hipEventElapsedTime(&ms[i], t.ev[i], t.ev[i + 1]) != hipSuccess) return MDGEMM_EHIP;
  return w;
}

void mdgemm_release(void) {
  Cache& c = cache();
  std::lock_guard<std::mutex> lock(c.mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (size_t d = 0; d < c.ptr.size(); ++d) {
    if (!c.ptr[d] && !c.last[d]) continue;
    if (hipSetDevice(static_cast<int>(d)) == hipSuccess) {
      (void)hipDeviceSynchronize();
      if (c.ptr[d]) (void)hipFree(c.ptr[d]);
      if (c.last[d]) (void)hipEventDestroy(c.last[d]);
    }
    c.ptr[d] = nullptr;
    c.bytes[d] = 0;
    c.last[d] = nullptr;
  }
  (void)hipSetDevice(cur);
}

// ---- stage entry points ----------------------------------------------------------

int mdgemm_line_spread(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, int32_t* spread,
                       void* stream) {
  if (rows < 0 || cols < 0 || (axis != 0 && axis != 1)) return MDGEMM_EINVAL;
  const int64_t lines = axis == 0 ? rows : cols;
  if (lines == 0) return MDGEMM_OK;
  if (!E || !spread || (rows > 0 && cols > 0 && !X0)) return MDGEMM_EINVAL;
  if (overlaps(E, sizeof(int32_t) * static_cast<size_t>(lines), spread, sizeof(int32_t) * static_cast<size_t>(lines)))
    return MDGEMM_EINVAL;
  return hip_status(mdg::launch_line_spread(rows, cols, axis, X0, E, spread, static_cast<hipStream_t>(stream)));
}

int mdgemm_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, void* stream) {
  if (rows < 0 || cols < 0 || (axis != 0 && axis != 1)) return MDGEMM_EINVAL;
  const int64_t lines = axis == 0 ? rows : cols;
  if (lines == 0) return MDGEMM_OK;
  if (!E || (rows > 0 && cols > 0 && !X0)) return MDGEMM_EINVAL;
  return hip_status(mdg::launch_exponents(rows, cols, axis, X0, E, static_cast<hipStream_t>(stream)));
}

int mdgemm_split(int64_t rows, int64_t cols, int limbs, int slices, int slice_bits, int axis, const double* X,
                 const int32_t* E, double* D, void* stream) {
  if (rows < 0 || cols < 0 || limbs < 1 || limbs > MDGEMM_MAX_LIMBS || !width_ok(slices, slice_bits) ||
      (axis != 0 && axis != 1))
    return MDGEMM_EINVAL;
  if (rows == 0 || cols == 0) return MDGEMM_OK;
  if (!X || !E || !D) return MDGEMM_EINVAL;
  const size_t xbytes = sizeof(double) * limbs * static_cast<size_t>(rows) * static_cast<size_t>(cols);
  const size_t dbytes = sizeof(double) * slices * static_cast<size_t>(rows) * static_cast<size_t>(cols);
  if (overlaps(D, dbytes, X, xbytes)) return MDGEMM_EINVAL;
  return hip_status(mdg::launch_split(rows, cols, limbs, slices, slice_bits, axis, X, E, D, false,
                                       static_cast<hipStream_t>(stream)));
}

int mdgemm_split_panel(int64_t rows, int64_t cols, int limbs, int slices, int slice_bits, int axis,
                       const double* X, const int32_t* E, double* D, void* stream) {
  if (rows < 0 || cols < 0 || limbs < 1 || limbs > MDGEMM_MAX_LIMBS || !width_ok(slices, slice_bits) ||
      (axis != 0 && axis != 1))
    return MDGEMM_EINVAL;
  if (rows == 0 || cols == 0) return MDGEMM_OK;
  if (!X || !E || !D) return MDGEMM_EINVAL;
  const int64_t K = axis == 0 ? cols : rows, Cn = axis == 0 ? rows : cols;
  const size_t xbytes = sizeof(double) * limbs * static_cast<size_t>(rows) * static_cast<size_t>(cols);
  const size_t dbytes = sizeof(double) * slices * static_cast<size_t>(mdg::panel_k(K)) *
                        static_cast<size_t>(mdg::panel_mn(Cn));
  if (overlaps(D, dbytes, X, xbytes)) return MDGEMM_EINVAL;
  return hip_status(mdg::launch_split(rows, cols, limbs, slices, slice_bits, axis, X, E, D, true,
                                       static_cast<hipStream_t>(stream)));
}

int mdgemm_slice_gemm(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, int per_pair,
                      const double* DAt, const double* DBp, double* out, void* stream) {
  if (m < 0 || n < 0 || k < 0 || slices < 1 || slices > MDGEMM_MAX_SLICES || slice_bits < 1 ||
      slice_bits > mdg::kMaxSliceBits || cutoff < 0 || cutoff > 2 * slices - 2)
    return MDGEMM_EINVAL;
  if (m == 0 || n == 0) return MDGEMM_OK;
  if (!out || (k > 0 && (!DAt || !DBp))) return MDGEMM_EINVAL;
  // panel rows are read 16 bytes per lane
  if ((reinterpret_cast<uintptr_t>(DAt) | reinterpret_cast<uintptr_t>(DBp)) & 15u) return MDGEMM_EINVAL;
  const size_t kp = static_cast<size_t>(mdg::panel_k(k));
  const size_t obytes = sizeof(double) * static_cast<size_t>(per_pair ? slices * slices : cutoff + 1) *
                        static_cast<size_t>(m) * static_cast<size_t>(n);
  if (k > 0 && (overlaps(out, obytes, DAt, sizeof(double) * slices * kp * static_cast<size_t>(mdg::panel_mn(m))) ||
                overlaps(out, obytes, DBp, sizeof(double) * slices * kp * static_cast<size_t>(mdg::panel_mn(n)))))
    return MDGEMM_EINVAL;
  if (!exact_ok(k, per_pair ? 1 : max_pairs(slices, cutoff), slice_bits)) return MDGEMM_EEXACT;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (!per_pair) return hip_status(mdg::launch_slice_gemm(m, n, k, DAt, DBp, out, level_jobs(slices, cutoff), s));
  for (const JobTable& jt : pair_jobs(slices, cutoff))
    MDG_TRY(hip_status(mdg::launch_slice_gemm(m, n, k, DAt, DBp, out, jt, s)));
  return MDGEMM_OK;
}

int mdgemm_accumulate(int64_t m, int64_t n, int levels, int slice_bits, const double* G, int64_t* Z, void* stream) {
  if (m < 0 || n < 0 || slice_bits < 1 || slice_bits > mdg::kMaxSliceBits || !levels_ok(levels, slice_bits))
    return MDGEMM_EINVAL;
  if (m == 0 || n == 0) return MDGEMM_OK;
  if (!G || !Z) return MDGEMM_EINVAL;
  return hip_status(mdg::launch_accumulate(m, n, levels, slice_bits, G, Z, static_cast<hipStream_t>(stream)));
}

int mdgemm_accum_renorm(int64_t m, int64_t n, int limbs, int levels, int slice_bits, const double* G,
                        const int32_t* EA, const int32_t* EB, double* C, void* stream) {
  if (m < 0 || n < 0 || limbs < 1 || limbs > MDGEMM_MAX_LIMBS || slice_bits < 1 || slice_bits > mdg::kMaxSliceBits ||
      !levels_ok(levels, slice_bits))
    return MDGEMM_EINVAL;
  if (m == 0 || n == 0) return MDGEMM_OK;
  if (!G || !EA || !EB || !C) return MDGEMM_EINVAL;
  const size_t cbytes = sizeof(double) * limbs * static_cast<size_t>(m) * static_cast<size_t>(n);
  const size_t gbytes = sizeof(double) * levels * static_cast<size_t>(m) * static_cast<size_t>(n);
  if (overlaps(C, cbytes, G, gbytes)) return MDGEMM_EINVAL;
  return hip_status(mdg::launch_accum_renorm(m, n, limbs, levels, slice_bits, G, EA, EB, C,
                                             static_cast<hipStream_t>(stream)));
}

}  // extern "C"

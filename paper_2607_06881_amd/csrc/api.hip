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

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <tuple>
#include <vector>

#include "internal.h"
#include "mdgemm.h"

// Device scratch of mdgemm_ex_noalloc: one fixed array per device, allocated
// with the code object when the library is loaded on that device and held until
// the process ends.  On the host, `scratch` is only a stand-in for the symbol,
// not a device address: host code resolves the address of each device's copy
// with hipGetSymbolAddress (noalloc_scratch below) and passes that to kernels.
static __device__ __align__(256) unsigned char scratch[MDGEMM_NOALLOC_MAX_BYTES];

static_assert(MDGEMM_MAX_LIMBS == mdg::kMaxLimbs && MDGEMM_MAX_SLICES == mdg::kMaxSlices &&
                  MDGEMM_Z_WORDS == mdg::kZWords && MDGEMM_SLICE_BITS == mdg::kSliceBits &&
                  MDGEMM_MAX_LEVELS == mdg::kMaxLevels && MDGEMM_MAX_SLICE_BITS == mdg::kMaxSliceBits &&
                  MDGEMM_MAX_DIGIT_BITS == mdg::kMaxDigitBits,
              "the limits of include/mdgemm.h and csrc/internal.h must agree");

namespace {


constexpr size_t kAlign = 256;
constexpr int kStages = 4;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

#define MDG_TRY(expr)              \
  do {                             \
    int st_ = (expr);              \
    if (st_ != MDGEMM_OK) return st_; \
  } while (0)

// Widest digit of the int8 level products: |d| <= 127 fits int8.
constexpr int kInt8MaxBits = 7;

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

// The int8 level products (MDGEMM_INT8) sum in int32: pairs_t * k * (2^w - 1)^2 < 2^31.
bool exact_ok_i32(int64_t k, int pairs, int w) {
  const uint64_t dmax = (1ull << w) - 1ull;
  const unsigned __int128 lhs =
      static_cast<unsigned __int128>(pairs) * static_cast<unsigned __int128>(k) * (dmax * dmax);
  return lhs < (static_cast<unsigned __int128>(1) << 31);
}

bool width_ok(int S, int w) { return S >= 1 && S <= MDGEMM_MAX_SLICES && w >= 1 && w <= mdg::kMaxSliceBits &&
                                     S * w <= mdg::kMaxDigitBits; }

// w (levels - 1) + 55 bits must fit the widest accumulation (kZWords words)
bool levels_ok(int levels, int w) {
  return levels >= 1 && levels <= mdg::kMaxLevels && mdg::accum_words(levels, w) <= mdg::kZWords;
}

// ---- schedules -------------------------------------------------------------

// Largest digit-count weight |combination a| |combination b| one GEMM job may
// sum: k weight (2^w - 1)^2 < 2^53, rounded down to a power of two (so that
// nearby k share a cached schedule), at most 2^20.
int64_t job_budget(int64_t k, int w) {
  const uint64_t dmax = (1ull << w) - 1ull;
  const unsigned __int128 per = static_cast<unsigned __int128>(k < 1 ? 1 : k) * (dmax * dmax);
  const unsigned __int128 lim = (static_cast<unsigned __int128>(1) << 53) - 1;
  int64_t b = static_cast<int64_t>(std::min<unsigned __int128>(lim / per, 1u << 20));
  int64_t p = 1;
  while (p * 2 <= b) p *= 2;
  return b < 1 ? 0 : p;
}

// Costs of a schedule's planes, level entries and combination panels relative
// to one GEMM term, from rates measured on MI355X: a GEMM term costs 2k flops per
// output element at ~70 TFLOP/s; a plane 16 bytes per element (written by the
// GEMM, read by the accumulation) at ~4.5 TB/s, times the accumulation's
// occupancy penalty (its LDS holds every level of a thread's element: 256
// threads per block up to 15 levels, 128 up to 31, 64 beyond, where the plane
// reads become latency-bound: measured ~1.4x and ~4x the HBM time); a level
// entry ~0.1 ps per element; a combination panel of A is written by the split
// beside the digits (8 m k bytes at ~4.5 TB/s), of B likewise with k x n.  Each
// size enters as a power of sqrt(2) (its code 2 log2(x), rounded), so that
// nearby shapes share a cached schedule.
constexpr double kTermRate = 70e12, kHbmRate = 4.5e12, kEntrySeconds = 0.1e-12;

int size_code(int64_t x) { return static_cast<int>(std::lround(2.0 * std::log2(static_cast<double>(x < 1 ? 1 : x)))); }
double from_code(int c) { return std::exp2(0.5 * c); }

mdg::ScheduleCosts schedule_costs(int mcode, int ncode, int kcode, int levels) {
  const double m = from_code(mcode), n = from_code(ncode), k = from_code(kcode);
  const double term = 2.0 * k / kTermRate;  // seconds per output element
  const double occupancy = levels < 16 ? 1.0 : (levels < 32 ? 1.4 : 4.0);
  mdg::ScheduleCosts c;
  c.plane = 16.0 * occupancy / kHbmRate / term;
  c.entry = kEntrySeconds / term;
  c.combo_a = 8.0 * m * k / kHbmRate / (term * m * n);
  c.combo_b = 8.0 * k * n / kHbmRate / (term * m * n);
  return c;
}

// A schedule with its device table.
struct Planned {
  mdg::Schedule s;
  mdg::ScheduleTable t;
  int max_digits = 1;  // digits in the largest combination of A or B
};

struct ScheduleCache {
  std::mutex mu;
  std::map<std::tuple<int, int, int64_t, int, int, int, int, int>, std::shared_ptr<const Planned>> map;
};
ScheduleCache& schedule_cache() {
  static ScheduleCache c;
  return c;
}

// kKaratsuba: the cost model's choice (may be the pair schedule);
// kKaratsubaMin: the Karatsuba schedule with the fewest GEMM terms.
// kGroups: the grouped pair schedule (exponent classes and / or sign groups).
enum class Kind { kLevels = 0, kPerPair = 1, kKaratsuba = 2, kKaratsubaMin = 3, kGroups = 4 };

Kind kind_of(unsigned flags) {
  if (flags & MDGEMM_KARATSUBA_MIN_TERMS) return Kind::kKaratsubaMin;
  return (flags & MDGEMM_KARATSUBA) ? Kind::kKaratsuba : Kind::kLevels;
}

// The schedule of the level products for S digits, cutoff T, an m x k by k x n
// product and width w, its jobs split into `sigma` k chunks; built once per key
// and kept for the life of the process.
// group: 2 Ge + sign for Kind::kGroups (Ge exponent classes, sign groups or not).
std::shared_ptr<const Planned> schedule_for(int S, int T, int64_t m, int64_t n, int64_t k, int w, Kind kind,
                                            int sigma = 1, int group = 0) {
  const bool kara = kind == Kind::kKaratsuba || kind == Kind::kKaratsubaMin;
  const bool model = kind == Kind::kKaratsuba;
  const int64_t budget = kara ? job_budget(k, w) : (kind == Kind::kGroups ? group : 0);
  const int mc = model ? size_code(m) : 0, nc = model ? size_code(n) : 0, kc = model ? size_code(k) : 0;
  const auto key = std::make_tuple(S, T, budget, mc, nc, kc, static_cast<int>(kind), sigma);
  ScheduleCache& c = schedule_cache();
  {
    std::lock_guard<std::mutex> lock(c.mu);
    auto it = c.map.find(key);
    if (it != c.map.end()) return it->second;
  }
  auto pl = std::make_shared<Planned>();
  if (sigma > 1) pl->s = mdg::split_k(schedule_for(S, T, m, n, k, w, kind, 1, group)->s, sigma);
  else if (kind == Kind::kLevels) pl->s = mdg::pair_schedule(S, T);
  else if (kind == Kind::kGroups) pl->s = mdg::group_schedule(S, T, group / 2, (group & 1) != 0);
  else if (kind == Kind::kPerPair) pl->s = mdg::per_pair_schedule(S, T);
  else if (kind == Kind::kKaratsuba)
    pl->s = mdg::karatsuba_schedule(S, T, budget, schedule_costs(mc, nc, kc, T + 1), true);
  else pl->s = mdg::karatsuba_schedule(S, T, budget, mdg::ScheduleCosts{}, false);
  pl->t = mdg::schedule_table(pl->s);
  for (uint64_t x : pl->s.mask_a) pl->max_digits = std::max(pl->max_digits, __builtin_popcountll(x));
  for (uint64_t x : pl->s.mask_b) pl->max_digits = std::max(pl->max_digits, __builtin_popcountll(x));
  std::shared_ptr<const Planned> sp = pl;
  std::lock_guard<std::mutex> lock(c.mu);
  return c.map.emplace(key, sp).first->second;
}

// Every job's digit weight within the exactness bound (the budget guarantees it
// for Karatsuba schedules; pair schedules are covered by the level check).
bool schedule_exact(const mdg::Schedule& s, int64_t k, int w) {
  return s.direct_levels || exact_ok(k, static_cast<int>(s.max_job_weight), w);
}

// ---- options ----------------------------------------------------------------

struct Resolved {
  int S = 0, T = 0, w = mdg::kSliceBits;
  int Ge = 1;         // exponent classes (MDGEMM_GROUP_EXPONENT)
  bool sign = false;  // sign groups (MDGEMM_GROUP_SIGN)
  hipStream_t stream = nullptr;
  unsigned flags = 0;
  Kind kind = Kind::kLevels;  // pair schedule, or Karatsuba (see kind_of), or groups
};

// The group parameters of a grouped schedule (0 for the others) and the levels
// of the product: T + 1, and 2 (Ge - 1) more with exponent classes (the class
// pairs' levels start up to 2 (Ge - 1) digits further down).
int group_code(const Resolved& r) { return r.kind == Kind::kGroups ? 2 * r.Ge + (r.sign ? 1 : 0) : 0; }
int total_levels(const Resolved& r) { return r.T + 1 + 2 * (r.Ge - 1); }

// The default count of 13-bit digits for L limbs.  Up to quad doubles, four per
// limb: section 2's quarters of each limb, 52 L bits, which cover the 53 L - 4
// bits of the tolerance 4 k 2^-(53 L - 4) (|A||B|).  Beyond four limbs four
// digits per limb fall short of those bits (by L - 4), so the count is the
// 53 L - 4 bits in whole digits plus one guard digit for the levels dropped at
// T = S - 1 (up to S - 1 products of the first dropped level): 34 for octo and
// 66 for hexa doubles instead of 32 and 64.
int default_digits(int limbs) {
  return limbs <= 4 ? 4 * limbs : (53 * limbs - 4 + mdg::kSliceBits - 1) / mdg::kSliceBits + 1;
}

// The digit bits the other widths cover by default: those of the 13-bit default.
int default_digit_bits(int limbs) { return mdg::kSliceBits * default_digits(limbs); }

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
// exact, the cheapest, the wider digit on a tie.  The cost is the pair count, or
// with the Karatsuba schedule the schedule's cost for this shape (GEMM terms plus
// planes, level entries and combinations; wider digits leave less room for
// digit sums).  Returns false when none qualifies.
bool auto_width(int limbs, int64_t m, int64_t n, int64_t k, int range_bits, int cutoff, Kind kind, int* w_out,
                int* S0_out) {
  double best_cost = 0.0;
  bool found = false;
  for (int w = mdg::kSliceBits; w <= mdg::kMaxSliceBits; ++w) {
    const int S0 = (default_digit_bits(limbs) + w - 1) / w, D = range_digits(range_bits, w);
    const int S = S0 + D, T = cutoff_for(cutoff, S0, D);
    if (!width_ok(S, w) || T < 0 || T > 2 * S - 2 || !levels_ok(T + 1, w) || !exact_ok(k, max_pairs(S, T), w))
      continue;
    double cost = pair_count(S, T);
    if (kind == Kind::kKaratsuba) {
      const auto pl = schedule_for(S, T, m, n, k, w, kind);
      cost = mdg::schedule_cost(pl->s, schedule_costs(size_code(m), size_code(n), size_code(k), T + 1));
    } else if (kind == Kind::kKaratsubaMin) {
      cost = schedule_for(S, T, m, n, k, w, kind)->s.terms;
    }
    if (!found || cost <= best_cost) {
      best_cost = cost;
      *w_out = w;
      *S0_out = S0;
      found = true;
    }
  }
  return found;
}

// Widest digit for the int8 level products: w = 7 down to 1 with S0 =
// ceil(52 L / w), D range digits and the requested cutoff, valid and exact in
// int32.  Returns MDGEMM_EINVAL when no width has S <= 64, MDGEMM_EEXACT when
// none of those is exact for this k.
int int8_width(int limbs, int64_t k, int range_bits, int cutoff, int* w_out, int* S0_out) {
  bool sized = false;
  for (int w = kInt8MaxBits; w >= 1; --w) {
    const int S0 = (default_digit_bits(limbs) + w - 1) / w, D = range_digits(range_bits, w);
    const int S = S0 + D, T = cutoff_for(cutoff, S0, D);
    if (!width_ok(S, w) || S > mdg::kI8MaxSlices || T < 0 || T > 2 * S - 2 || !levels_ok(T + 1, w)) continue;
    sized = true;
    if (!exact_ok_i32(k, max_pairs(S, T), w)) continue;
    *w_out = w;
    *S0_out = S0;
    return MDGEMM_OK;
  }
  return sized ? MDGEMM_EEXACT : MDGEMM_EINVAL;
}

// Digit width, digit count and cutoff of a product with reduction length k.
int resolve(int limbs, int64_t m, int64_t n, int64_t k, const mdgemm_opts* opts, Resolved* r) {
  if (limbs < 1 || limbs > MDGEMM_MAX_LIMBS) return MDGEMM_EINVAL;
  r->kind = kind_of(opts ? opts->flags : 0u);
  const int bits = opts ? opts->slice_bits : 0;
  const int slices = opts ? opts->slices : 0;
  const int range_bits = opts ? opts->range_bits : 0;
  if (slices < 0 || range_bits < 0 || range_bits > mdg::kMaxDigitBits) return MDGEMM_EINVAL;
  const bool int8 = opts && (opts->flags & MDGEMM_INT8);
  if (int8) {
    if (opts->flags & (MDGEMM_KARATSUBA | MDGEMM_KARATSUBA_MIN_TERMS)) return MDGEMM_EINVAL;
    if (bits == 0 || bits == MDGEMM_SLICE_BITS_AUTO) {
      if (slices != 0) return MDGEMM_EINVAL;
      MDG_TRY(int8_width(limbs, k, range_bits, opts->cutoff, &r->w, &r->S));
    } else if (bits >= 1 && bits <= kInt8MaxBits) {
      r->w = bits;
      r->S = slices ? slices : (default_digit_bits(limbs) + bits - 1) / bits;
    } else {
      return MDGEMM_EINVAL;
    }
  } else if (bits == MDGEMM_SLICE_BITS_AUTO) {
    if (slices != 0) return MDGEMM_EINVAL;
    if (!auto_width(limbs, m, n, k, range_bits, opts->cutoff, r->kind, &r->w, &r->S)) return MDGEMM_EEXACT;
  } else if (bits == 0 || bits == mdg::kSliceBits) {
    r->w = mdg::kSliceBits;
    const int spl = opts ? opts->slices_per_limb : 0;
    if (spl < 0) return MDGEMM_EINVAL;
    r->S = slices ? slices : (spl ? spl * limbs : default_digits(limbs));
  } else if (bits >= 1 && bits <= mdg::kMaxSliceBits) {
    r->w = bits;
    r->S = slices ? slices : (default_digit_bits(limbs) + bits - 1) / bits;
  } else {
    return MDGEMM_EINVAL;
  }
  // range balancing: D more digits on the same line grid, and the cutoff raised by
  // 2D so that a product of two elements D digits below their lines' exponents
  // keeps its S0 leading levels.  With exponent classes the range sets the
  // number of classes instead, Ge = 1 + ceil(range_bits / w), and each class
  // element gets one more digit (it lies up to one digit below its class grid),
  // with the cutoff of one such digit per factor.
  const unsigned flags = opts ? opts->flags : 0u;
  const bool gexp = (flags & MDGEMM_GROUP_EXPONENT) != 0;
  const int S0 = r->S, D = gexp ? (range_bits > 0 ? 1 : 0) : range_digits(range_bits, r->w);
  r->Ge = gexp ? 1 + range_digits(range_bits, r->w) : 1;
  r->sign = (flags & MDGEMM_GROUP_SIGN) != 0;
  r->S = S0 + D;
  if (!width_ok(r->S, r->w) || (int8 && r->S > mdg::kI8MaxSlices)) return MDGEMM_EINVAL;
  const int cutoff = opts ? opts->cutoff : MDGEMM_CUTOFF_DEFAULT;
  if (cutoff < 0 && cutoff != MDGEMM_CUTOFF_DEFAULT && cutoff != MDGEMM_CUTOFF_ALL) return MDGEMM_EINVAL;
  r->T = cutoff_for(cutoff, S0, D);
  if (r->T < 0 || r->T > 2 * r->S - 2) return MDGEMM_EINVAL;
  if (!levels_ok(r->T + 1 + 2 * (r->Ge - 1), r->w)) return MDGEMM_EINVAL;
  if (r->Ge > 1 || r->sign) {
    // grouped products: the pair schedule over group pairs, up to 4 limbs, the
    // split's integer in kGroupSplitWords words, at most 4096 panels (G S)
    if (int8 || (flags & (MDGEMM_KARATSUBA | MDGEMM_KARATSUBA_MIN_TERMS)) || bits == MDGEMM_SLICE_BITS_AUTO ||
        limbs > 4 || (r->w * r->S + 52 + 63) / 64 > mdg::kGroupSplitWords ||
        (r->sign ? 2 : 1) * r->Ge * r->S > 4096)
      return MDGEMM_EINVAL;
    r->kind = Kind::kGroups;
  }
  r->stream = opts ? static_cast<hipStream_t>(opts->stream) : nullptr;
  r->flags = opts ? opts->flags : 0u;
  return MDGEMM_OK;
}

// FP32 panels when every panel value (a digit, or a combination of up to
// max_digits digits) is an integer below 2^24, so that FP32 holds it exactly.
bool panels_f32(const Planned& pl, int w) {
  return static_cast<uint64_t>(pl.max_digits) * ((1ull << w) - 1ull) < (1ull << 24);
}

// K split of a product whose tile jobs would not fill the chip: below 1.5
// rounds of the 512 blocks resident at a time (two 256-thread blocks per CU),
// split to about 2.5 rounds, at most 8 chunks, each at least 8 k steps of every
// pair.  (Measured on 1024^3 double-double: 384 blocks split 4 ways run the
// level GEMM at 87% of peak instead of 58%; 960 blocks gain nothing from a
// split and the extra planes cost accumulation time.)
int ksplit_count(int64_t blocks, int64_t nkb) {
  constexpr int64_t kFull = 768, kTarget = 1280;
  if (blocks <= 0 || blocks >= kFull) return 1;
  int64_t sigma = (kTarget + blocks - 1) / blocks;
  sigma = std::min<int64_t>(sigma, std::min<int64_t>(8, nkb / 8));
  return static_cast<int>(std::max<int64_t>(sigma, 1));
}

int ksplit_for(int64_t m, int64_t n, int64_t k, const Planned& pl, bool f32) {
  const int64_t tiles = (mdg::panel_mn(m) / mdg::kTileMN) * (mdg::panel_mn(n) / mdg::kTileMN);
  const int64_t blocks = tiles * static_cast<int64_t>(pl.s.job_first.size());
  const int64_t nkb = f32 ? mdg::panel_k32(k) / mdg::kTileK32 : mdg::panel_k(k) / mdg::kTileK;
  return ksplit_count(blocks, nkb);
}

// The schedule a product runs: the planned one, split in k when it is small.
std::shared_ptr<const Planned> planned_for(int S, int T, int64_t m, int64_t n, int64_t k, int w, Kind kind,
                                           int group = 0) {
  auto base = schedule_for(S, T, m, n, k, w, kind, 1, group);
  const int sigma = ksplit_for(m, n, k, *base, panels_f32(*base, w));
  return sigma > 1 ? schedule_for(S, T, m, n, k, w, kind, sigma, group) : base;
}

// The fused small-product kernel (one block per 16 x 16 tile of C runs all five
// steps) instead of the staged path, for outputs of at most 256 such tiles whose
// levels fit its limits, when its estimated time is below the staged path's.
// The staged path is bound by launch latency and by its level GEMM's 128 x 128
// (or 64 x 128) tiles: one block per tile, level and k chunk, the heaviest
// level's pairs in series.  The fused kernel's time grows with k (S + L), the
// limbs read and digits written per line of a tile.  Both paths give the same
// limbs, so the choice moves only time.  The estimates, in microseconds, were
// fitted to 139 products measured side by side on MI355X (1 to 4 limbs, 13- to
// 21-bit digits, outputs from 17 x 33 to 256 x 256 and 16 x 4096, k up to 4096);
// they pick the faster path on all but five near-ties, each within 6%:
//  fused: 17, plus the split at 15.7, 16.5, 19 or 22 ns (1 to 4 limbs) per unit
//    of k (S + L), plus the most loaded SIMD's level products (one
//    v_mfma_f64_16x16x4f64 per pair and 4 of k, 64 cycles at 2.4 GHz): the two
//    phases alternate per k chunk;
//  staged: 57 for its exponent, split, accumulation and rounding launches, plus
//    1.13 times its level GEMM, the larger of its heaviest block (the heaviest
//    level's pairs over one k chunk) and all its MFMAs spread over 1024 SIMDs.
// Levels are dealt to the four SIMDs heaviest first to the least loaded, and
// within a SIMD to the lighter of its two waves.  kc: the largest k chunk (a
// multiple of 4, at most 256) whose digits fit the kernel's LDS beside the
// levels.
constexpr int64_t kSmallMaxTiles = 256;
constexpr double kMfmaUs = 64.0 / 2400.0;  // one v_mfma_f64_16x16x4f64 on one SIMD

double fused_estimate_us(int64_t k, int limbs, int S, int simd_pairs) {
  static constexpr double kSplitNs[mdg::kSmallMaxLimbs + 1] = {0.0, 15.7, 16.5, 19.0, 22.0};
  return 17.0 + 1e-3 * kSplitNs[limbs] * static_cast<double>(k * (S + limbs)) +
         kMfmaUs * simd_pairs * static_cast<double>((k + 3) / 4);
}

// The staged pair schedule: T + 1 level jobs per tile, FP32 panels of 32-deep k
// steps, split in k by ksplit_count.
double staged_estimate_us(int64_t m, int64_t n, int64_t k, int T, int heaviest_pairs, int total_pairs) {
  const int64_t tiles = (mdg::panel_mn(m) / mdg::kTileMN) * (mdg::panel_mn(n) / mdg::kTileMN);
  const int64_t nkb = mdg::panel_k32(k) / mdg::kTileK32;
  const int64_t sigma = ksplit_count(tiles * (T + 1), nkb);
  const int64_t chunk = (nkb + sigma - 1) / sigma;
  const int rows = m <= 64 ? 64 : mdg::kTileMN;
  // MFMAs per SIMD for one pair over one k step of a tile (four waves per block)
  const double per_step = (rows / 16) * (mdg::kTileMN / 16) * (mdg::kTileK32 / 4) / 4.0;
  const double heavy = static_cast<double>(heaviest_pairs) * chunk * per_step;
  const double spread = static_cast<double>(total_pairs) * tiles * nkb * per_step * 4.0 / 1024.0;
  return 57.0 + 1.13 * kMfmaUs * std::max(heavy, spread);
}

bool small_plan(int64_t m, int64_t n, int64_t k, int limbs, const Resolved& r, int* kc_out,
                mdg::SmallLevelOwners* owners) {
  if (r.kind == Kind::kGroups ||
      (r.flags & (MDGEMM_INT8 | MDGEMM_KARATSUBA | MDGEMM_KARATSUBA_MIN_TERMS | MDGEMM_STAGED | MDGEMM_CHECK_FINITE)))
    return false;
  // digits are held in LDS as FP32 values: exact while below 2^24
  if (limbs < 1 || limbs > mdg::kSmallMaxLimbs || r.T + 1 > mdg::kSmallMaxLevels || k < 1 || r.w > 24) return false;
  if (r.w * r.S + 52 > 64 * mdg::kSmallSplitWords || r.w * r.T + 55 > 64 * mdg::kSmallAccumWords) return false;
  if (((m + 15) / 16) * ((n + 15) / 16) > kSmallMaxTiles) return false;
  int load[4] = {0, 0, 0, 0}, wload[mdg::kSmallWaves] = {};
  int heaviest = 0, total = 0;
  bool done[mdg::kSmallMaxLevels] = {};
  for (int rep = 0; rep <= r.T; ++rep) {
    int best = -1, bp = -1;
    for (int t = 0; t <= r.T; ++t) {
      const int lo = t - (r.S - 1) > 0 ? t - (r.S - 1) : 0, hi = t < r.S - 1 ? t : r.S - 1;
      const int p = hi - lo + 1;
      if (!done[t] && p > bp) {
        bp = p;
        best = t;
      }
    }
    int wv = 0;
    for (int v = 1; v < 4; ++v)
      if (load[v] < load[wv]) wv = v;
    done[best] = true;
    load[wv] += bp;
    const int wave = wload[wv + 4] < wload[wv] ? wv + 4 : wv;
    wload[wave] += bp;
    owners->wave[best] = static_cast<int8_t>(wave);
    heaviest = std::max(heaviest, bp);
    total += bp;
  }
  const int maxload = std::max(std::max(load[0], load[1]), std::max(load[2], load[3]));
  if (fused_estimate_us(k, limbs, r.S, maxload) > staged_estimate_us(m, n, k, r.T, heaviest, total)) return false;
  int kc = static_cast<int>(std::min<int64_t>(256, (k + 3) / 4 * 4));
  while (kc > 4 && mdg::small_product_lds(r.S, r.T, kc) > mdg::kSmallMaxLds) kc -= 4;
  if (mdg::small_product_lds(r.S, r.T, kc) > mdg::kSmallMaxLds) return false;
  *kc_out = kc;
  return true;
}

struct Layout {
  size_t ea = 0, eb = 0, flag = 0, table = 0, da = 0, db = 0, g = 0, total = 0;
  bool f32 = false;  // FP32 panels with panel_k32 rows, else FP64 with panel_k rows
};

// EA | EB | flag | schedule table | A's combinations | B's combinations | planes,
// each aligned to 256 bytes (combinations 0..S-1 are the digit panels).
bool layout(int64_t m, int64_t n, int64_t k, const Planned& pl, int w, Layout* L) {
  const mdg::Schedule& sch = pl.s;
  const double ca = static_cast<double>(sch.mask_a.size()), cb = static_cast<double>(sch.mask_b.size());
  // all products below 2^62 so that size arithmetic cannot overflow
  const double approx = ca * (double)m * (double)(k + 32) + cb * (double)(k + 32) * (double)n +
                        (double)sch.planes * (double)m * (double)n;
  if (approx * 8.0 > 4.0e18) return false;
  // the level GEMM addresses panel rows with 32-bit lane offsets (m, n up to 2^27)
  // and numbers its tiles in 31 bits
  const int64_t mp = mdg::panel_mn(m), np = mdg::panel_mn(n);
  if (mp > (int64_t{1} << 27) || np > (int64_t{1} << 27) || (mp / mdg::kTileMN) * (np / mdg::kTileMN) > INT_MAX)
    return false;
  L->f32 = panels_f32(pl, w);
  const size_t esz = L->f32 ? sizeof(float) : sizeof(double);
  size_t off = 0;
  L->ea = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(m));
  L->eb = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(n));
  L->flag = off;
  off += align_up(sizeof(int32_t));
  L->table = off;
  off += align_up(sizeof(uint32_t) * pl.t.words.size());
  L->da = off;
  const size_t kp = static_cast<size_t>(L->f32 ? mdg::panel_k32(k) : mdg::panel_k(k));
  off += align_up(esz * sch.mask_a.size() * kp * static_cast<size_t>(mp));
  L->db = off;
  off += align_up(esz * sch.mask_b.size() * kp * static_cast<size_t>(np));
  L->g = off;
  off += align_up(sizeof(double) * static_cast<size_t>(sch.planes) * static_cast<size_t>(m) * static_cast<size_t>(n));
  L->total = off;
  return true;
}

// The level sums of a resolved product stay exact: below 2^53 on the FP64
// matrix cores, below 2^31 on the int8 ones.
bool resolved_exact(const Resolved& r, int64_t k) {
  const int pairs = max_pairs(r.S, r.T);
  return (r.flags & MDGEMM_INT8) ? exact_ok_i32(k, pairs, r.w) : exact_ok(k, pairs, r.w);
}

// Workspace of the int8 level products: EA | EB | flag | A's digits
// [mp][kI8Pad + S kp] | B's digits [np][kI8Pad + S kp] | int32 levels [T+1][m][n],
// each aligned to 256 bytes; kp = k rounded up to 128, mp and np = m and n
// rounded up to 256 (the layout of csrc/level_gemm_i8.hip).
struct LayoutI8 {
  size_t ea = 0, eb = 0, flag = 0, da = 0, dbt = 0, g = 0, total = 0;
  int64_t kp = 0, mp = 0, np = 0;
};
bool layout_int8(int64_t m, int64_t n, int64_t k, int S, int T, LayoutI8* L) {
  L->kp = mdg::i8_kp(k);
  L->mp = mdg::i8_rows(m);
  L->np = mdg::i8_rows(n);
  if (!mdg::level_gemm_i8_fits(L->kp, S)) return false;
  const double ld = mdg::kI8Pad + (double)S * (double)L->kp;
  const double approx = ld * ((double)L->mp + (double)L->np) + 4.0 * (T + 1) * (double)m * (double)n;
  if (approx > 4.0e18 || m > (int64_t{1} << 31) || n > (int64_t{1} << 31)) return false;
  const size_t pitch = mdg::kI8Pad + static_cast<size_t>(S) * static_cast<size_t>(L->kp);
  size_t off = 0;
  L->ea = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(m));
  L->eb = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(n));
  L->flag = off;
  off += align_up(sizeof(int32_t));
  L->da = off;
  off += align_up(static_cast<size_t>(L->mp) * pitch);
  L->dbt = off;
  off += align_up(static_cast<size_t>(L->np) * pitch);
  L->g = off;
  off += align_up(sizeof(int32_t) * static_cast<size_t>(T + 1) * static_cast<size_t>(m) * static_cast<size_t>(n));
  L->total = off;
  return true;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// A caller workspace of `bytes` bytes that overlaps A [L][m][k], B [L][k][n] or
// C [L][m][n] (the workspace is written while A and B are still read).
bool workspace_overlaps(const void* ws, size_t bytes, int64_t m, int64_t n, int64_t k, int limbs, const double* A,
                        const double* B, const double* C) {
  const size_t L = static_cast<size_t>(limbs);
  const size_t abytes = sizeof(double) * L * static_cast<size_t>(m) * static_cast<size_t>(k);
  const size_t bbytes = sizeof(double) * L * static_cast<size_t>(k) * static_cast<size_t>(n);
  const size_t cbytes = sizeof(double) * L * static_cast<size_t>(m) * static_cast<size_t>(n);
  return overlaps(ws, bytes, A, abytes) || overlaps(ws, bytes, B, bbytes) || overlaps(ws, bytes, C, cbytes);
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

// The library buffer of the current device, held for one call: acquire() takes
// the cache's mutex, grows the buffer and makes `stream` wait for the previous
// user's work; release() records this call's end for the next user and lets go
// of the mutex (also when enqueueing stopped at an error).  Refused while
// `stream` is capturing a graph: the graph would keep an address that a later,
// larger call may free.
class LibraryBuffer {
 public:
  ~LibraryBuffer() { release(MDGEMM_OK); }
  int acquire(size_t need, hipStream_t stream, char** out) {
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cap) != hipSuccess) return MDGEMM_EHIP;
    if (cap != hipStreamCaptureStatusNone) return MDGEMM_EINVAL;
    lock_ = std::unique_lock<std::mutex>(cache().mu);
    void* p = nullptr;
    int dev = -1;
    const int st = cached_workspace(cache(), need, &p, &dev);
    if (st != MDGEMM_OK) {
      lock_.unlock();
      return st;
    }
    dev_ = dev;
    stream_ = stream;
    if (hipStreamWaitEvent(stream, cache().last[dev_], 0) != hipSuccess) return release(MDGEMM_EHIP);
    *out = static_cast<char*>(p);
    return MDGEMM_OK;
  }
  int release(int st) {
    if (dev_ < 0) return st;
    const bool ok = hipEventRecord(cache().last[dev_], stream_) == hipSuccess;
    dev_ = -1;
    lock_.unlock();
    return (st == MDGEMM_OK && !ok) ? MDGEMM_EHIP : st;
  }

 private:
  std::unique_lock<std::mutex> lock_;
  int dev_ = -1;
  hipStream_t stream_ = nullptr;
};

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

// Pointers into a workspace laid out by layout(); DA / DB are float* for FP32 panels.
struct Parts {
  int32_t *EA, *EB, *flag;
  uint32_t* table;
  void *DA, *DB;
  double* G;
  bool f32;
};
Parts parts(char* ws, const Layout& L) {
  return Parts{reinterpret_cast<int32_t*>(ws + L.ea), reinterpret_cast<int32_t*>(ws + L.eb),
               reinterpret_cast<int32_t*>(ws + L.flag), reinterpret_cast<uint32_t*>(ws + L.table),
               ws + L.da,
               ws + L.db,
               reinterpret_cast<double*>(ws + L.g),
               L.f32};
}

// Before the level GEMMs, when the digit panels are given (not split here): the
// combinations of both operands from the panels, and the schedule's device table.
int enqueue_schedule_inputs(const Planned& pl, int64_t m, int64_t n, int64_t k, const Parts& w, hipStream_t s) {
  const int64_t kp = w.f32 ? mdg::panel_k32(k) : mdg::panel_k(k), mp = mdg::panel_mn(m), np = mdg::panel_mn(n);
  if (w.f32) {
    MDG_TRY(hip_status(mdg::launch_combinations32(pl.s, true, static_cast<float*>(w.DA), kp * mp, s)));
    MDG_TRY(hip_status(mdg::launch_combinations32(pl.s, false, static_cast<float*>(w.DB), kp * np, s)));
  } else {
    MDG_TRY(hip_status(mdg::launch_combinations(pl.s, true, static_cast<double*>(w.DA), kp * mp, s)));
    MDG_TRY(hip_status(mdg::launch_combinations(pl.s, false, static_cast<double*>(w.DB), kp * np, s)));
  }
  return hip_status(mdg::launch_upload(pl.t.words, w.table, s));
}

int enqueue_gemm(const Planned& pl, int64_t m, int64_t n, int64_t k, const Parts& w, double* out, hipStream_t s) {
  mdg::GemmJobs jobs;
  jobs.jobs = w.table + pl.t.jobs_off;
  jobs.pairs = w.table + pl.t.pairs_off;
  jobs.njobs = static_cast<int>(pl.s.job_first.size());
  if (w.f32)
    return hip_status(mdg::launch_slice_gemm32(m, n, k, static_cast<const float*>(w.DA),
                                               static_cast<const float*>(w.DB), out, jobs, s));
  return hip_status(mdg::launch_slice_gemm(m, n, k, static_cast<const double*>(w.DA),
                                           static_cast<const double*>(w.DB), out, jobs, s));
}

// MDGEMM_CHECK_FINITE: scan A and B for inf/nan (synchronizes the stream).
int check_finite(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, int32_t* flag,
                 hipStream_t s) {
  MDG_TRY(hip_status(mdg::launch_set_i32(flag, 1, 0, s)));
  MDG_TRY(hip_status(mdg::launch_nonfinite_scan(A, static_cast<int64_t>(limbs) * m * k, flag, s)));
  MDG_TRY(hip_status(mdg::launch_nonfinite_scan(B, static_cast<int64_t>(limbs) * k * n, flag, s)));
  int32_t h = 0;
  MDG_TRY(hip_status(hipMemcpyAsync(&h, flag, sizeof h, hipMemcpyDeviceToHost, s)));
  MDG_TRY(hip_status(hipStreamSynchronize(s)));
  return h ? MDGEMM_ENONFINITE : MDGEMM_OK;
}

// mdgemm_ex with MDGEMM_INT8 (m, n, k > 0, arguments checked): exponents, int8
// digits, one int8 GEMM per level into int32 planes, exact accumulation.
int run_int8(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
             const mdgemm_opts* opts, const Resolved& r) {
  LayoutI8 L;
  if (!layout_int8(m, n, k, r.S, r.T, &L)) return MDGEMM_EINVAL;
  hipStream_t s = r.stream;
  const bool timed = (r.flags & MDGEMM_TIME_STAGES) != 0;
  char* ws = nullptr;
  LibraryBuffer lib;
  if (opts && opts->workspace) {
    if (opts->workspace_bytes < L.total) return MDGEMM_EWORKSPACE;
    if (workspace_overlaps(opts->workspace, L.total, m, n, k, limbs, A, B, C)) return MDGEMM_EINVAL;
    ws = static_cast<char*>(opts->workspace);
  } else {
    MDG_TRY(lib.acquire(L.total, s, &ws));
  }
  int32_t* EA = reinterpret_cast<int32_t*>(ws + L.ea);
  int32_t* EB = reinterpret_cast<int32_t*>(ws + L.eb);
  int32_t* flag = reinterpret_cast<int32_t*>(ws + L.flag);
  int8_t* DA = reinterpret_cast<int8_t*>(ws + L.da);
  int8_t* DBt = reinterpret_cast<int8_t*>(ws + L.dbt);
  int32_t* G = reinterpret_cast<int32_t*>(ws + L.g);
  auto enqueue = [&]() -> int {
    if (r.flags & MDGEMM_CHECK_FINITE) MDG_TRY(check_finite(m, n, k, limbs, A, B, flag, s));
    std::unique_lock<std::mutex> tlock(timing().mu, std::defer_lock);
    if (timed) {
      tlock.lock();
      timing().valid = false;
      MDG_TRY(record(0, s));
    }
    MDG_TRY(hip_status(mdg::launch_exponents(m, k, 0, A, EA, s)));
    MDG_TRY(hip_status(mdg::launch_exponents(k, n, 1, B, EB, s)));
    if (timed) MDG_TRY(record(1, s));
    MDG_TRY(hip_status(mdg::launch_split_int8(m, k, limbs, r.S, r.w, A, EA, DA, L.kp, s)));
    MDG_TRY(hip_status(mdg::launch_split_int8t(k, n, limbs, r.S, r.w, B, EB, DBt, L.kp, L.np, s)));
    if (timed) MDG_TRY(record(2, s));
    MDG_TRY(hip_status(mdg::launch_level_gemm_i8(m, n, L.kp, r.S, r.T, DA, DBt, G, s)));
    if (timed) MDG_TRY(record(3, s));
    MDG_TRY(hip_status(mdg::launch_accum_renorm_i32(m, n, limbs, r.T + 1, r.w, G, EA, EB, C, s)));
    if (timed) {
      MDG_TRY(record(4, s));
      timing().valid = true;
    }
    return MDGEMM_OK;
  };
  const int st = lib.release(enqueue());
  if (st != MDGEMM_OK) return st;
  if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
  return MDGEMM_OK;
}

}  // namespace

extern "C" {

void mdgemm_opts_init(mdgemm_opts* opts) {
  if (!opts) return;
  std::memset(opts, 0, sizeof *opts);
  opts->slices_per_limb = 0;
  opts->cutoff = MDGEMM_CUTOFF_DEFAULT;
  opts->slice_bits = 0;
  opts->slices = 0;
  opts->range_bits = 0;
}

int mdgemm_plan(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts, int* slice_bits, int* slices,
                int* cutoff) {
  Resolved r;
  if (m < 0 || n < 0 || k < 0) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, m, n, k, opts, &r));
  if (!resolved_exact(r, k)) return MDGEMM_EEXACT;
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
  if (m < 0 || n < 0 || k < 0 || resolve(limbs, m, n, k, opts, &r) != MDGEMM_OK) return SIZE_MAX;
  if (m == 0 || n == 0 || k == 0) return 0;
  if (r.flags & MDGEMM_INT8) {
    LayoutI8 L8;
    return layout_int8(m, n, k, r.S, r.T, &L8) ? L8.total : SIZE_MAX;
  }
  Layout L;
  if (!layout(m, n, k, *planned_for(r.S, r.T, m, n, k, r.w, r.kind, group_code(r)), r.w, &L)) return SIZE_MAX;
  return L.total;
}

int mdgemm_workspace_layout(int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts, int64_t* info,
                            int count) {
  Resolved r;
  if (m < 0 || n < 0 || k < 0 || count < 0 || (count > 0 && !info)) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, m, n, k, opts, &r));
  if (m == 0 || n == 0 || k == 0 || (r.flags & MDGEMM_INT8)) return MDGEMM_EINVAL;
  if (!resolved_exact(r, k)) return MDGEMM_EEXACT;
  int kc = 0;
  mdg::SmallLevelOwners owners{};
  if (small_plan(m, n, k, limbs, r, &kc, &owners)) return MDGEMM_EINVAL;
  const auto pl = planned_for(r.S, r.T, m, n, k, r.w, r.kind, group_code(r));
  Layout L;
  if (!layout(m, n, k, *pl, r.w, &L)) return MDGEMM_EINVAL;
  const int64_t v[MDGEMM_LAYOUT_INFO] = {static_cast<int64_t>(L.ea),
                                         static_cast<int64_t>(L.eb),
                                         static_cast<int64_t>(L.da),
                                         static_cast<int64_t>(L.db),
                                         static_cast<int64_t>(L.g),
                                         L.f32 ? 4 : 8,
                                         L.f32 ? mdg::panel_k32(k) : mdg::panel_k(k),
                                         mdg::panel_mn(m),
                                         mdg::panel_mn(n),
                                         pl->s.planes,
                                         pl->s.direct_levels ? 1 : 0,
                                         static_cast<int64_t>(L.total)};
  const int nw = std::min(count, MDGEMM_LAYOUT_INFO);
  for (int i = 0; i < nw; ++i) info[i] = v[i];
  return nw;
}

}  // extern "C"

namespace {

// The product; *path names the branch taken (for MDGEMM_LOG).
int ex_impl(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
            const mdgemm_opts* opts, const char** path) {
  Resolved r;
  *path = "refused";
  if (m < 0 || n < 0 || k < 0) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, m, n, k, opts, &r));
  *path = "empty";
  if (m == 0 || n == 0) return MDGEMM_OK;
  *path = "refused";
  if (!C || (k > 0 && (!A || !B))) return MDGEMM_EINVAL;
  const size_t abytes = sizeof(double) * limbs * static_cast<size_t>(m) * static_cast<size_t>(k);
  const size_t bbytes = sizeof(double) * limbs * static_cast<size_t>(k) * static_cast<size_t>(n);
  const size_t cbytes = sizeof(double) * limbs * static_cast<size_t>(m) * static_cast<size_t>(n);
  if (k > 0 && (overlaps(C, cbytes, A, abytes) || overlaps(C, cbytes, B, bbytes))) return MDGEMM_EINVAL;
  if (!resolved_exact(r, k)) return MDGEMM_EEXACT;
  hipStream_t s = r.stream;
  const bool timed = (r.flags & MDGEMM_TIME_STAGES) != 0;

  if (k == 0) {
    *path = "zero (k = 0)";
    MDG_TRY(hip_status(mdg::launch_zero_f64(C, static_cast<int64_t>(limbs) * m * n, s)));
    if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
    return MDGEMM_OK;
  }

  if (r.flags & MDGEMM_INT8) {
    *path = "int8 levels";
    return run_int8(m, n, k, limbs, A, B, C, opts, r);
  }
  const auto pl = planned_for(r.S, r.T, m, n, k, r.w, r.kind, group_code(r));
  if (!schedule_exact(pl->s, k, r.w)) return MDGEMM_EEXACT;
  Layout L;
  if (!layout(m, n, k, *pl, r.w, &L)) return MDGEMM_EINVAL;
  if (opts && opts->workspace) {
    if (opts->workspace_bytes < L.total) return MDGEMM_EWORKSPACE;
    if (workspace_overlaps(opts->workspace, L.total, m, n, k, limbs, A, B, C)) return MDGEMM_EINVAL;
  }
  int kc = 0;
  mdg::SmallLevelOwners owners{};
  if (small_plan(m, n, k, limbs, r, &kc, &owners)) {
    // the fused small-product kernel: no workspace
    *path = "fused small product";
    std::unique_lock<std::mutex> tlock(timing().mu, std::defer_lock);
    if (timed) {
      tlock.lock();
      timing().valid = false;
      for (int i = 0; i < 3; ++i) MDG_TRY(record(i, s));
    }
    MDG_TRY(hip_status(mdg::launch_small_product(m, n, k, limbs, r.S, r.T, r.w, kc, owners, A, B, C, s)));
    if (timed) {
      MDG_TRY(record(3, s));
      MDG_TRY(record(4, s));
      timing().valid = true;
    }
    if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
    return MDGEMM_OK;
  }
  *path = r.kind == Kind::kGroups ? "staged: grouped products"
          : (r.kind == Kind::kLevels ? "staged: pair levels"
                                     : (r.kind == Kind::kPerPair ? "staged: per pair" : "staged: karatsuba"));
  char* ws = nullptr;
  LibraryBuffer lib;
  if (opts && opts->workspace) {
    ws = static_cast<char*>(opts->workspace);
  } else {
    MDG_TRY(lib.acquire(L.total, s, &ws));
  }
  const Parts w = parts(ws, L);

  auto enqueue = [&]() -> int {
    if (r.flags & MDGEMM_CHECK_FINITE) MDG_TRY(check_finite(m, n, k, limbs, A, B, w.flag, s));
    std::unique_lock<std::mutex> tlock(timing().mu, std::defer_lock);
    if (timed) {
      tlock.lock();
      timing().valid = false;
      MDG_TRY(record(0, s));
    }
    // a1: grid exponents per row of A and per column of B (partial column maxima
    // in B's panel region, which the split overwrites next)
    MDG_TRY(hip_status(mdg::launch_exponents_ab(m, k, n, A, B, w.EA, w.EB, w.DB, L.g - L.db, s)));
    if (timed) MDG_TRY(record(1, s));
    // a2: exact splits into S digit panels and, beside them, the schedule's
    // combinations (digit sums) from the same integers
    MDG_TRY(hip_status(mdg::launch_upload(pl->t.words, w.table, s)));
    if (r.kind == Kind::kGroups) {
      // grouped digits: each element's S digits in its group's panels, on its class grid
      MDG_TRY(hip_status(mdg::launch_split_groups(m, k, limbs, r.S, r.w, 0, A, w.EA, w.DA, w.f32, r.Ge, r.sign, s)));
      MDG_TRY(hip_status(mdg::launch_split_groups(k, n, limbs, r.S, r.w, 1, B, w.EB, w.DB, w.f32, r.Ge, r.sign, s)));
    } else {
      MDG_TRY(hip_status(mdg::launch_split(m, k, limbs, r.S, r.w, 0, A, w.EA, w.DA, true, s,
                                           w.table + pl->t.masks_a_off, static_cast<int>(pl->s.mask_a.size()),
                                           w.f32)));
      MDG_TRY(hip_status(mdg::launch_split(k, n, limbs, r.S, r.w, 1, B, w.EB, w.DB, true, s,
                                           w.table + pl->t.masks_b_off, static_cast<int>(pl->s.mask_b.size()),
                                           w.f32)));
    }
    if (timed) MDG_TRY(record(2, s));
    // a3: level GEMMs (or the Karatsuba products) on the FP64 matrix cores
    MDG_TRY(enqueue_gemm(*pl, m, n, k, w, w.G, s));
    if (timed) MDG_TRY(record(3, s));
    // a4 + a5: exact accumulation and greedy rounding into L limbs
    if (pl->s.direct_levels) {
      MDG_TRY(hip_status(mdg::launch_accum_renorm(m, n, limbs, total_levels(r), r.w, w.G, w.EA, w.EB, C, s)));
    } else {
      MDG_TRY(hip_status(mdg::launch_plan_accum(m, n, limbs, total_levels(r), r.w, pl->s.planes, w.G,
                                                w.table + pl->t.chunk_first_off, w.table + pl->t.chunks_off, w.EA,
                                                w.EB, C, nullptr, s)));
    }
    if (timed) {
      MDG_TRY(record(4, s));
      timing().valid = true;
    }
    return MDGEMM_OK;
  };
  // the next user of the library buffer waits for everything enqueued here,
  // also when enqueueing stopped at an error
  const int st = lib.release(enqueue());
  if (st != MDGEMM_OK) return st;
  if (r.flags & MDGEMM_SYNC) MDG_TRY(hip_status(hipStreamSynchronize(s)));
  return MDGEMM_OK;
}

// One line per call on stderr: the arguments, the plan, the branch and the status.
void log_product(const char* entry, int64_t m, int64_t n, int64_t k, int limbs, const mdgemm_opts* opts,
                 const char* ws, const char* path, int status) {
  int w = 0, S = 0, T = 0;
  const bool planned = mdgemm_plan(m, n, k, limbs, opts, &w, &S, &T) == MDGEMM_OK;
  const unsigned flags = opts ? opts->flags : 0u;
  char plan[64] = "unplanned";
  if (planned) std::snprintf(plan, sizeof plan, "w=%d S=%d T=%d", w, S, T);
  mdg::log_line("%s m=%lld n=%lld k=%lld limbs=%d %s flags=0x%x workspace=%s stream=%p path=%s -> %s", entry,
                static_cast<long long>(m), static_cast<long long>(n), static_cast<long long>(k), limbs, plan, flags,
                ws, opts ? opts->stream : nullptr, path, mdgemm_status_string(status));
}

}  // namespace

namespace mdg {

int log_level() {
  static const int level = [] {
    const char* v = std::getenv("MDGEMM_LOG");
    return v ? std::atoi(v) : 0;
  }();
  return level;
}

thread_local int log_depth = 0;

void log_line(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  std::fprintf(stderr, "[mdgemm] %s\n", buf);
}

}  // namespace mdg

extern "C" {

int mdgemm_ex(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
              const mdgemm_opts* opts) {
  const char* path = "refused";
  const int st = ex_impl(m, n, k, limbs, A, B, C, opts, &path);
  if (mdg::log_level() > mdg::log_depth)
    log_product("mdgemm_ex", m, n, k, limbs, opts, opts && opts->workspace ? "caller" : "library", path, st);
  return st;
}

int mdgemm(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C) {
  return mdgemm_ex(m, n, k, limbs, A, B, C, nullptr);
}

}  // extern "C"

namespace {

// The device address of `scratch` on the current device, resolved once per
// device (with that device current) and kept.
struct NoallocScratch {
  std::mutex mu;
  std::vector<void*> ptr;
};
NoallocScratch& noalloc_state() {
  static NoallocScratch s;
  return s;
}

int noalloc_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MDGEMM_EHIP;
  NoallocScratch& s = noalloc_state();
  std::lock_guard<std::mutex> lock(s.mu);
  if (static_cast<size_t>(dev) >= s.ptr.size()) s.ptr.resize(dev + 1, nullptr);
  if (!s.ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return MDGEMM_EHIP;
    }
    s.ptr[dev] = p;
  }
  *out = s.ptr[dev];
  return MDGEMM_OK;
}

}  // namespace

namespace {

int noalloc_impl(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
                 const mdgemm_opts* opts, const char** path) {
  *path = "refused";
  mdgemm_opts o;
  if (opts) {
    o = *opts;
  } else {
    mdgemm_opts_init(&o);
  }
  // the scratch array is the workspace; timing events and the finiteness
  // check's host copy are left out so that nothing is allocated on the way
  if (o.workspace || o.workspace_bytes || (o.flags & (MDGEMM_TIME_STAGES | MDGEMM_CHECK_FINITE)))
    return MDGEMM_EINVAL;
  Resolved r;
  if (m < 0 || n < 0 || k < 0) return MDGEMM_EINVAL;
  MDG_TRY(resolve(limbs, m, n, k, &o, &r));
  if (m == 0 || n == 0) return MDGEMM_OK;
  const size_t need = mdgemm_workspace_bytes(m, n, k, limbs, &o);
  if (need == SIZE_MAX) return MDGEMM_EINVAL;
  if (need > MDGEMM_NOALLOC_MAX_BYTES) return MDGEMM_EWORKSPACE;
  void* p = nullptr;
  MDG_TRY(noalloc_scratch(&p));
  o.workspace = p;
  o.workspace_bytes = MDGEMM_NOALLOC_MAX_BYTES;
  return ex_impl(m, n, k, limbs, A, B, C, &o, path);
}

}  // namespace

extern "C" {

int mdgemm_ex_noalloc(int64_t m, int64_t n, int64_t k, int limbs, const double* A, const double* B, double* C,
                      const mdgemm_opts* opts) {
  const char* path = "refused";
  const int st = noalloc_impl(m, n, k, limbs, A, B, C, opts, &path);
  if (mdg::log_level() > mdg::log_depth)
    log_product("mdgemm_ex_noalloc", m, n, k, limbs, opts, "scratch array", path, st);
  return st;
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
  const auto pl = schedule_for(slices, cutoff, m, n, k, slice_bits, per_pair ? Kind::kPerPair : Kind::kLevels);
  // the job table goes into the library buffer
  LibraryBuffer lib;
  char* tab = nullptr;
  MDG_TRY(lib.acquire(sizeof(uint32_t) * pl->t.words.size(), s, &tab));
  Parts w{};
  w.table = reinterpret_cast<uint32_t*>(tab);
  w.DA = const_cast<double*>(DAt);  // the caller's FP64 panels, read in place
  w.DB = const_cast<double*>(DBp);
  w.f32 = false;
  int st = hip_status(mdg::launch_upload(pl->t.words, w.table, s));
  if (st == MDGEMM_OK) st = enqueue_gemm(*pl, m, n, k, w, out, s);
  return lib.release(st);
}

int mdgemm_schedule_info(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                         int64_t* info, int count) {
  if (m < 0 || n < 0 || slices < 1 || slices > MDGEMM_MAX_SLICES || slice_bits < 1 || slice_bits > mdg::kMaxSliceBits ||
      cutoff < 0 || cutoff > 2 * slices - 2 || k < 0 || count < 0 || (count > 0 && !info))
    return MDGEMM_EINVAL;
  const auto pl = planned_for(slices, cutoff, m, n, k, slice_bits, kind_of(flags));
  const mdg::Schedule& sc = pl->s;
  int max_depth = 0;
  for (int d : sc.depth_a) max_depth = std::max(max_depth, d);
  for (int d : sc.depth_b) max_depth = std::max(max_depth, d);
  const int64_t v[MDGEMM_SCHEDULE_INFO] = {sc.terms,
                                           static_cast<int64_t>(sc.job_first.size()),
                                           sc.planes,
                                           static_cast<int64_t>(sc.mask_a.size()),
                                           static_cast<int64_t>(sc.mask_b.size()),
                                           static_cast<int64_t>(sc.entry_level.size()),
                                           sc.max_job_weight,
                                           max_depth,
                                           sc.direct_levels ? 1 : 0,
                                           pl->max_digits,
                                           panels_f32(*pl, slice_bits) ? 1 : 0,
                                           sc.ksplit};
  const int nw = std::min(count, MDGEMM_SCHEDULE_INFO);
  for (int i = 0; i < nw; ++i) info[i] = v[i];
  return nw;
}

int mdgemm_schedule_export(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                           uint64_t* mask_a, int32_t* parents_a, uint64_t* mask_b, int32_t* parents_b, int32_t* jobs,
                           int32_t* pairs, int32_t* plane_first, int32_t* entries) {
  if (m < 0 || n < 0 || slices < 1 || slices > MDGEMM_MAX_SLICES || slice_bits < 1 || slice_bits > mdg::kMaxSliceBits ||
      cutoff < 0 || cutoff > 2 * slices - 2 || k < 0)
    return MDGEMM_EINVAL;
  const auto pl = planned_for(slices, cutoff, m, n, k, slice_bits, kind_of(flags));
  const mdg::Schedule& sc = pl->s;
  for (size_t c = 0; c < sc.mask_a.size(); ++c) {
    if (mask_a) mask_a[c] = sc.mask_a[c];
    if (parents_a) {
      parents_a[2 * c] = sc.par1_a[c];
      parents_a[2 * c + 1] = sc.par2_a[c];
    }
  }
  for (size_t c = 0; c < sc.mask_b.size(); ++c) {
    if (mask_b) mask_b[c] = sc.mask_b[c];
    if (parents_b) {
      parents_b[2 * c] = sc.par1_b[c];
      parents_b[2 * c + 1] = sc.par2_b[c];
    }
  }
  for (size_t j = 0; jobs && j < sc.job_first.size(); ++j) {
    jobs[4 * j] = sc.job_first[j];
    jobs[4 * j + 1] = sc.job_count[j];
    jobs[4 * j + 2] = sc.job_out[j];
    jobs[4 * j + 3] = sc.job_chunk.empty() ? 0 : sc.job_chunk[j];
  }
  for (size_t i = 0; pairs && i < sc.pair_a.size(); ++i) {
    pairs[2 * i] = sc.pair_a[i];
    pairs[2 * i + 1] = sc.pair_b[i];
  }
  for (size_t i = 0; plane_first && i < sc.plane_first.size(); ++i) plane_first[i] = sc.plane_first[i];
  for (size_t e = 0; entries && e < sc.entry_level.size(); ++e) {
    entries[2 * e] = sc.entry_level[e];
    entries[2 * e + 1] = sc.entry_coef[e];
  }
  return MDGEMM_OK;
}

size_t mdgemm_schedule_workspace_bytes(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff,
                                       unsigned flags) {
  if (m < 0 || n < 0 || k < 0 || slices < 1 || slices > MDGEMM_MAX_SLICES || slice_bits < 1 ||
      slice_bits > mdg::kMaxSliceBits || cutoff < 0 || cutoff > 2 * slices - 2)
    return SIZE_MAX;
  const auto pl = planned_for(slices, cutoff, m, n, k, slice_bits, kind_of(flags));
  Layout L;
  if (!layout(m, n, k, *pl, slice_bits, &L)) return SIZE_MAX;
  return L.total;
}

int mdgemm_schedule_levels(int64_t m, int64_t n, int64_t k, int slices, int slice_bits, int cutoff, unsigned flags,
                           const double* DAt, const double* DBp, double* G, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (m < 0 || n < 0 || k < 0 || slices < 1 || slices > MDGEMM_MAX_SLICES || slice_bits < 1 ||
      slice_bits > mdg::kMaxSliceBits || cutoff < 0 || cutoff > 2 * slices - 2 || !levels_ok(cutoff + 1, slice_bits))
    return MDGEMM_EINVAL;
  if (m == 0 || n == 0) return MDGEMM_OK;
  if (!G || (k > 0 && (!DAt || !DBp))) return MDGEMM_EINVAL;
  if (!exact_ok(k, max_pairs(slices, cutoff), slice_bits)) return MDGEMM_EEXACT;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t levels = cutoff + 1;
  if (k == 0) return hip_status(mdg::launch_zero_f64(G, levels * m * n, s));
  const auto pl = planned_for(slices, cutoff, m, n, k, slice_bits, kind_of(flags));
  if (!schedule_exact(pl->s, k, slice_bits)) return MDGEMM_EEXACT;
  Layout L;
  if (!layout(m, n, k, *pl, slice_bits, &L)) return MDGEMM_EINVAL;
  const size_t kp = static_cast<size_t>(mdg::panel_k(k)), mp = static_cast<size_t>(mdg::panel_mn(m)),
               np = static_cast<size_t>(mdg::panel_mn(n));
  const size_t abytes = sizeof(double) * slices * kp * mp, bbytes = sizeof(double) * slices * kp * np;
  const size_t gbytes = sizeof(double) * static_cast<size_t>(levels) * static_cast<size_t>(m) * static_cast<size_t>(n);
  if (overlaps(G, gbytes, DAt, abytes) || overlaps(G, gbytes, DBp, bbytes)) return MDGEMM_EINVAL;
  char* ws = nullptr;
  LibraryBuffer lib;
  if (workspace) {
    if (workspace_bytes < L.total) return MDGEMM_EWORKSPACE;
    if (overlaps(workspace, L.total, G, gbytes) || overlaps(workspace, L.total, DAt, abytes) ||
        overlaps(workspace, L.total, DBp, bbytes))
      return MDGEMM_EINVAL;
    ws = static_cast<char*>(workspace);
  } else {
    MDG_TRY(lib.acquire(L.total, s, &ws));
  }
  const Parts w = parts(ws, L);
  auto enqueue = [&]() -> int {
    // the digit panels are combinations 0..S-1 of the schedule (as FP32 panels
    // with 32-row k steps when every value fits, like mdgemm_ex)
    if (w.f32) {
      const int64_t kp32 = mdg::panel_k32(k);
      MDG_TRY(hip_status(mdg::launch_panel_to_f32(DAt, static_cast<float*>(w.DA), static_cast<int64_t>(kp), kp32,
                                                  static_cast<int64_t>(mp), slices, s)));
      MDG_TRY(hip_status(mdg::launch_panel_to_f32(DBp, static_cast<float*>(w.DB), static_cast<int64_t>(kp), kp32,
                                                  static_cast<int64_t>(np), slices, s)));
    } else {
      MDG_TRY(hip_status(hipMemcpyAsync(w.DA, DAt, abytes, hipMemcpyDeviceToDevice, s)));
      MDG_TRY(hip_status(hipMemcpyAsync(w.DB, DBp, bbytes, hipMemcpyDeviceToDevice, s)));
    }
    MDG_TRY(enqueue_schedule_inputs(*pl, m, n, k, w, s));
    if (pl->s.direct_levels) return enqueue_gemm(*pl, m, n, k, w, G, s);
    MDG_TRY(enqueue_gemm(*pl, m, n, k, w, w.G, s));
    return hip_status(mdg::launch_plan_accum(m, n, 1, static_cast<int>(levels), slice_bits, pl->s.planes, w.G,
                                             w.table + pl->t.chunk_first_off, w.table + pl->t.chunks_off, nullptr,
                                             nullptr, nullptr, G, s));
  };
  return lib.release(enqueue());
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

// Exact integer arithmetic on the device shared by the kernels that split
// operands into digits and that accumulate and round level products (the
// staged kernels and the fused small-product kernel use the same functions, so
// that both paths compute the same digits and limbs).
//
// Split (section 2: the fraction cut into 13-bit parts on a shared grid;
// section 3: a limb of opposite sign moves a unit to the next, which is the
// floor below): D = floor(|V| / u) of an element with limbs x_0..x_{L-1} on the
// grid unit u = 2^g, formed exactly as a fixed-point integer with 52 fraction
// bits in NW 64-bit words; its w-bit fields are the digits.
//
// Accumulation (section 2, steps 4-5; section 1, renormalization): the levels'
// weighted sum N = sum_t G_t 2^(w (T - t)) as a two's-complement integer,
// added in increasing significance, then peeled greedily into L limbs rounded
// to nearest (ties to even).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <climits>
#include <type_traits>

namespace mdg {
namespace {

constexpr int kNoExp = INT_MIN;

// frexp exponent of x; INT_MIN for +-0.  Subnormals: bit length of the
// significand minus 1074.
__device__ inline int frexp_exp_or_min(double x) {
  uint64_t mag = static_cast<uint64_t>(__double_as_longlong(x)) & 0x7fffffffffffffffull;
  if (mag == 0) return kNoExp;
  int be = static_cast<int>(mag >> 52);
  if (be == 0) return (64 - __clzll(static_cast<long long>(mag))) - 1074;
  return be - 1022;
}

// acc += M 2^sh (neg == false) or acc -= M 2^sh (neg == true), modulo 2^(64 NW);
// M < 2^53 and sh + 53 <= 64 NW.
template <int NW>
__device__ inline void add_shifted(uint64_t (&acc)[NW], uint64_t M, int sh, bool neg) {
  const int w = sh >> 6, b = sh & 63;
  const uint64_t lo = M << b;
  const uint64_t hi = b ? (M >> (64 - b)) : 0ull;
  uint64_t carry = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint64_t t = (i == w) ? lo : ((i == w + 1) ? hi : 0ull);
    const uint64_t a = acc[i];
    if (!neg) {
      const uint64_t s = a + t;
      const uint64_t c1 = s < a;
      const uint64_t s2 = s + carry;
      const uint64_t c2 = s2 < s;
      acc[i] = s2;
      carry = c1 | c2;
    } else {
      const uint64_t s = a - t;
      const uint64_t b1 = a < t;
      const uint64_t s2 = s - carry;
      const uint64_t b2 = s < carry;
      acc[i] = s2;
      carry = b1 | b2;
    }
  }
}

// D = floor(|V| / u) for one element with limbs xs[0..L-1] (L <= ML) on the
// grid unit 2^g, as an NW-word integer; returns true when V < 0.
template <int NW, int ML>
__device__ inline bool floor_on_grid(const double (&xs)[ML], int L, int g, uint64_t (&I)[NW]) {
  const double x0 = xs[0];
  const bool neg = x0 < 0.0;
  uint64_t acc[NW];
#pragma unroll
  for (int i = 0; i < NW; ++i) acc[i] = 0;
  int tail = 0;  // +1 / -1: sign, relative to V, of the part of V below u that is not in acc
  if (x0 != 0.0) {
#pragma unroll
    for (int l = 0; l < ML; ++l) {
      const double xl = xs[l];
      if (l >= L || xl == 0.0) break;  // normalized: every later limb is zero too
      const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(xl));
      const bool lneg = (bits >> 63) != 0;
      const uint64_t mag = bits & 0x7fffffffffffffffull;
      const int be = static_cast<int>(mag >> 52);
      uint64_t M;
      int ex;  // |xl| = M 2^ex
      if (be != 0) {
        M = (mag & 0x000fffffffffffffull) | 0x0010000000000000ull;
        ex = be - 1075;
      } else {
        M = mag;
        ex = -1074;
      }
      const int fe = ex + (64 - __clzll(static_cast<long long>(M)));  // frexp exponent of xl
      if (fe <= g) {  // |xl| < u: xl and the rest of the limbs lie below the grid unit
        tail = (lneg == neg) ? 1 : -1;
        break;
      }
      add_shifted<NW>(acc, M, ex - g + 52, lneg != neg);
    }
  }
  // I = floor(acc / 2^52), lowered by one when the fraction is zero and the
  // part below u is negative (relative to the sign of V).
  const bool frac_zero = (acc[0] & 0x000fffffffffffffull) == 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) I[i] = (acc[i] >> 52) | (i + 1 < NW ? acc[i + 1] << 12 : 0ull);
  if (frac_zero && tail < 0) {
    uint64_t borrow = 1;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint64_t v = I[i];
      I[i] = v - borrow;
      borrow = (v < borrow) ? 1ull : 0ull;
    }
  }
  return neg;
}

// The same floor for digit windows of at most 128 bits (w S <= 128), held in one
// 128-bit integer without fraction bits.  By nonoverlap (|x_{l+1}| <= ulp(x_l)/2)
// only the first limb with bits below the grid unit matters below it: the
// limbs after it are smaller than one unit of its last place, so the fraction
// of |V| / u has that limb's sign relative to V and lies strictly between -1 and
// 1.  Hence D = sum over the limbs up to it of +-floor(|x_l| / u), lowered by
// one when that limb has the opposite sign of V.  Every partial sum stays in
// [0, 2^(w S)) and |x_0| < 2^(g + w S) keeps each shift below 128 - 53.
template <int ML>
__device__ inline bool floor_on_grid_128(const double (&xs)[ML], int L, int g, uint64_t (&I)[2]) {
  const bool neg = xs[0] < 0.0;
  unsigned __int128 acc = 0;
  bool lower = false;
#pragma unroll
  for (int l = 0; l < ML; ++l) {
    const double xl = xs[l];
    if (l >= L || xl == 0.0) break;  // normalized: every later limb is zero too
    const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(xl));
    const bool sub = ((bits >> 63) != 0) != neg;
    const uint64_t mag = bits & 0x7fffffffffffffffull;
    const int be = static_cast<int>(mag >> 52);
    const uint64_t M = be != 0 ? ((mag & 0x000fffffffffffffull) | 0x0010000000000000ull) : mag;
    int k = (be != 0 ? be - 1075 : -1074) - g;  // |x_l| / u = M 2^k
    if (k <= -53) {  // the whole limb lies below the grid unit
      lower = sub;
      break;
    }
    k = k < 127 ? k : 127;  // only for exponents that are not the line's maximum
    const unsigned __int128 part = k >= 0 ? static_cast<unsigned __int128>(M) << k : M >> -k;
    acc = sub ? acc - part : acc + part;
    if (k < 0 && (M & ((1ull << -k) - 1ull)) != 0) {  // bits below the unit: the last limb that counts
      lower = sub;
      break;
    }
  }
  if (lower) acc -= 1;
  I[0] = static_cast<uint64_t>(acc);
  I[1] = static_cast<uint64_t>(acc >> 64);
  return neg;
}

// The same floor for windows of at most 256 bits, in two 128-bit halves with the
// carry (or borrow) between them formed by comparison.
template <int ML>
__device__ inline bool floor_on_grid_256(const double (&xs)[ML], int L, int g, uint64_t (&I)[4]) {
  typedef unsigned __int128 u128;
  const bool neg = xs[0] < 0.0;
  u128 lo = 0, hi = 0;
  bool lower = false;
#pragma unroll
  for (int l = 0; l < ML; ++l) {
    const double xl = xs[l];
    if (l >= L || xl == 0.0) break;
    const uint64_t bits = static_cast<uint64_t>(__double_as_longlong(xl));
    const bool sub = ((bits >> 63) != 0) != neg;
    const uint64_t mag = bits & 0x7fffffffffffffffull;
    const int be = static_cast<int>(mag >> 52);
    const uint64_t M = be != 0 ? ((mag & 0x000fffffffffffffull) | 0x0010000000000000ull) : mag;
    int k = (be != 0 ? be - 1075 : -1074) - g;
    if (k <= -53) {
      lower = sub;
      break;
    }
    k = k < 255 ? k : 255;
    u128 plo, phi;  // M 2^k (integer part) as two halves
    if (k < 0) {
      plo = M >> -k;
      phi = 0;
    } else if (k < 128) {
      plo = static_cast<u128>(M) << k;
      phi = k > 75 ? static_cast<u128>(M) >> (128 - k) : 0;  // the bits that pass bit 127
    } else {
      plo = 0;
      phi = static_cast<u128>(M) << (k - 128);
    }
    if (sub) {
      const u128 borrow = lo < plo ? 1 : 0;
      lo -= plo;
      hi = hi - phi - borrow;
    } else {
      lo += plo;
      hi = hi + phi + (lo < plo ? 1 : 0);
    }
    if (k < 0 && (M & ((1ull << -k) - 1ull)) != 0) {
      lower = sub;
      break;
    }
  }
  if (lower) {
    hi -= lo == 0 ? 1 : 0;
    lo -= 1;
  }
  I[0] = static_cast<uint64_t>(lo);
  I[1] = static_cast<uint64_t>(lo >> 64);
  I[2] = static_cast<uint64_t>(hi);
  I[3] = static_cast<uint64_t>(hi >> 64);
  return neg;
}

// The L limbs of the element at idx (limb stride ls), all loads issued together;
// limbs beyond L are +0.0 (L is the same for every thread).
template <int ML>
__device__ inline void load_limbs(const double* __restrict__ X, int64_t ls, int L, int64_t idx, double (&xs)[ML]) {
#pragma unroll
  for (int l = 0; l < ML; ++l) xs[l] = l < L ? X[static_cast<int64_t>(l) * ls + idx] : 0.0;
}

__device__ inline double signed_digit(uint32_t d, bool neg) {
  const double v = static_cast<double>(d);
  return (d == 0u) ? 0.0 : (neg ? -v : v);  // zero digits are +0.0
}

// Word i of v (0 beyond the top), by an unrolled select: no dynamic register indexing.
template <int NW>
__device__ inline uint64_t word_or_zero(const uint64_t (&v)[NW], int i) {
  uint64_t r = 0;
#pragma unroll
  for (int j = 0; j < NW; ++j) r = (j == i) ? v[j] : r;
  return r;
}

// Digit s of I (bits w(S-1-s) .. w(S-s)-1) to out[s * stride] for every s, read
// upward from bit 0 through a two-word window: one select over the words per
// 64 bits consumed instead of one per digit.
template <int NW, class OutT>
__device__ inline void store_digits(const uint64_t (&I)[NW], int S, int w, bool neg, OutT* __restrict__ out,
                                    int64_t stride) {
  const uint64_t mask = (1ull << w) - 1ull;
  uint64_t cur = I[0], nxt = NW > 1 ? I[1] : 0ull;
  int wi = 0, b = 0;  // cur = word wi of I; b = next unread bit of cur
  for (int j = 0; j < S; ++j) {
    uint64_t f = cur >> b;
    if (b + w > 64) f |= nxt << (64 - b);  // b > 64 - w > 0 here
    const uint32_t d = static_cast<uint32_t>(f & mask);
    if constexpr (std::is_integral<OutT>::value) {
      const int32_t v = static_cast<int32_t>(d);  // int8 digits: the sign in integer arithmetic
      out[static_cast<int64_t>(S - 1 - j) * stride] = static_cast<OutT>(neg ? -v : v);
    } else {
      out[static_cast<int64_t>(S - 1 - j) * stride] = static_cast<OutT>(signed_digit(d, neg));
    }
    b += w;
    if (b >= 64) {
      b -= 64;
      cur = nxt;
      ++wi;
      nxt = word_or_zero<NW>(I, wi + 1);
    }
  }
}

// N += g 2^sh (g sign-extended), modulo 2^(64 NW).
template <int NW>
__device__ inline void add_shifted_signed(uint64_t (&N)[NW], int64_t g, int sh) {
  const int w = sh >> 6, b = sh & 63;
  const uint64_t lo = static_cast<uint64_t>(g) << b;
  const uint64_t hi = b ? static_cast<uint64_t>(g >> (64 - b)) : static_cast<uint64_t>(g >> 63);
  const uint64_t ext = static_cast<uint64_t>(g >> 63);  // 0 or all ones
  uint64_t carry = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint64_t t = (i < w) ? 0ull : ((i == w) ? lo : ((i == w + 1) ? hi : ext));
    const uint64_t s = N[i] + t;
    const uint64_t c1 = s < t;
    const uint64_t s2 = s + carry;
    const uint64_t c2 = s2 < s;
    N[i] = s2;
    carry = c1 | c2;
  }
}

// N = sum_t G_t 2^(w (T - t)) exactly.  Level t is column j = T - t of weight
// 2^(w j); the columns are visited in increasing significance (t = T down to
// 0) with a running carry in base 2^w: v = G_t + carry, the low w bits of v
// are the digit of column j (placed into N, whose bits there are still zero)
// and carry = floor(v / 2^w).  |G_t| < 2^53 keeps |v| < 2^54, so int64 never
// overflows; the last carry, signed, is added above column T.
// The digits fill N from bit 0 upward: `word` collects the bits of word wi of
// N, `fill` of them so far; a full word is placed with one select over the words.
template <int NW>
struct CarryChain {
  uint64_t word = 0;
  int fill = 0, wi = 0;
  int64_t carry = 0;

  __device__ inline void step(uint64_t (&N)[NW], int64_t g, int w, uint64_t mask) {
    const int64_t v = g + carry;
    const uint64_t d = static_cast<uint64_t>(v) & mask;
    carry = v >> w;  // arithmetic shift: floor division
    word |= d << fill;
    fill += w;
    if (fill >= 64) {
#pragma unroll
      for (int i = 0; i < NW; ++i) N[i] = (i == wi) ? word : N[i];
      ++wi;
      fill -= 64;
      word = fill ? d >> (w - fill) : 0ull;  // the bits of d beyond the full word
    }
  }
  __device__ inline void finish(uint64_t (&N)[NW], int w, int T) {
#pragma unroll
    for (int i = 0; i < NW; ++i) N[i] = (i == wi) ? word : N[i];
    if (carry != 0) add_shifted_signed<NW>(N, carry, w * (T + 1));
  }
};

// Bit `pos` (0 <= pos < 64 NW) of v.
template <int NW>
__device__ inline uint64_t word_at(const uint64_t (&v)[NW], int w) {
  uint64_t r = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) r = (i == w) ? v[i] : r;
  return r;
}

template <int NW>
__device__ inline void round_limbs(uint64_t (&N)[NW], int L, int scale, double* __restrict__ C, int64_t plane,
                                   int64_t idx) {
  // sign and magnitude
  bool neg = (N[NW - 1] >> 63) != 0;
  if (neg) {
    uint64_t carry = 1;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint64_t v = ~N[i] + carry;
      carry = (carry && v == 0) ? 1ull : 0ull;
      N[i] = v;
    }
  }
  for (int l = 0; l < L; ++l) {
    // position of the leading one
    int h = -1;
#pragma unroll
    for (int i = 0; i < NW; ++i)
      if (N[i] != 0) h = 64 * i + 63 - __clzll(static_cast<long long>(N[i]));
    double c;
    if (h < 0) {
      c = 0.0;
    } else if (h <= 52) {
      const double v = static_cast<double>(N[0]);  // below 2^53: exact
      c = ldexp(neg ? -v : v, scale);
#pragma unroll
      for (int i = 0; i < NW; ++i) N[i] = 0;
    } else {
      const int sh = h - 52;  // the 53 leading bits start at bit sh
      const int w = sh >> 6, b = sh & 63;
      const uint64_t lo = word_at<NW>(N, w), hi = word_at<NW>(N, w + 1);
      uint64_t M = (lo >> b) | (b ? (hi << (64 - b)) : 0ull);
      M &= 0x001fffffffffffffull;
      // round bit (bit sh-1) and sticky (any bit below sh-1)
      const int rpos = sh - 1, rw = rpos >> 6, rb = rpos & 63;
      const uint64_t rword = word_at<NW>(N, rw);
      const bool round_bit = ((rword >> rb) & 1ull) != 0;
      bool sticky = (rword & ((1ull << rb) - 1ull)) != 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) sticky |= (i < rw) && (N[i] != 0);
      const bool up = round_bit && (sticky || (M & 1ull));
      const double v = static_cast<double>(M + (up ? 1ull : 0ull));  // <= 2^53: exact
      c = ldexp(neg ? -v : v, scale + sh);
      // remainder: the bits below sh, or 2^sh minus them (and the sign flips)
#pragma unroll
      for (int i = 0; i < NW; ++i) {
        const int lo_bit = 64 * i;
        uint64_t keep;
        if (lo_bit + 64 <= sh) keep = ~0ull;
        else if (lo_bit >= sh) keep = 0ull;
        else keep = (1ull << (sh - lo_bit)) - 1ull;
        N[i] &= keep;
      }
      if (up) {
        uint64_t carry = 1;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
          const int lo_bit = 64 * i;
          uint64_t keep;
          if (lo_bit + 64 <= sh) keep = ~0ull;
          else if (lo_bit >= sh) keep = 0ull;
          else keep = (1ull << (sh - lo_bit)) - 1ull;
          const uint64_t v = ~N[i] + carry;
          carry = (carry && v == 0) ? 1ull : 0ull;
          N[i] = v & keep;
        }
        neg = !neg;
      }
    }
    // a limb that underflows in the final scaling is +0.0, like every zero limb
    C[static_cast<int64_t>(l) * plane + idx] = c == 0.0 ? 0.0 : c;
  }
}

}  // namespace
}  // namespace mdg

// Double-double arithmetic on the device, for the downstream use of the
// product in a blocked Householder QR (the application the paper names as
// future work).  A double-double (hi, lo) is the unevaluated sum of two
// nonoverlapping doubles (section 1).  The operations are the error-free
// transformations of section 1 composed as in Dekker (1971) and Hida, Li and
// Bailey (2001): TwoSum (Knuth), FastTwoSum (Dekker), TwoProd with a fused
// multiply-add, and the accurate double-double add, multiply, divide and square
// root built from them.  Floating-point contraction is switched off inside
// every function (a fused multiply-add appears only where it is written), so
// each sum and product is rounded on its own as the transformations require.
#pragma once

#include <hip/hip_runtime.h>

namespace mdg {
namespace {

struct dd {
  double hi, lo;
};

// Every function below starts with `#pragma clang fp contract(off)`: no sum or
// product is fused with another (the error-free transformations need each
// operation rounded on its own); fused multiply-adds are written explicitly.

// s + e = a + b exactly (Knuth's TwoSum).
__device__ inline dd two_sum(double a, double b) {
#pragma clang fp contract(off)
  const double s = a + b;
  const double bb = s - a;
  const double e = (a - (s - bb)) + (b - bb);
  return {s, e};
}

// s + e = a + b exactly when |a| >= |b| or a == 0 (Dekker's FastTwoSum).
__device__ inline dd fast_two_sum(double a, double b) {
#pragma clang fp contract(off)
  const double s = a + b;
  return {s, b - (s - a)};
}

// p + e = a b exactly (barring underflow), with one fused multiply-add.
__device__ inline dd two_prod(double a, double b) {
#pragma clang fp contract(off)
  const double p = a * b;
  return {p, __builtin_fma(a, b, -p)};
}

// Accurate double-double sum: both partial sums error-free, renormalized twice.
__device__ inline dd dd_add(dd a, dd b) {
#pragma clang fp contract(off)
  dd s = two_sum(a.hi, b.hi);
  const dd t = two_sum(a.lo, b.lo);
  s.lo = s.lo + t.hi;
  s = fast_two_sum(s.hi, s.lo);
  s.lo = s.lo + t.lo;
  return fast_two_sum(s.hi, s.lo);
}

__device__ inline dd dd_neg(dd a) { return {-a.hi, -a.lo}; }
__device__ inline dd dd_sub(dd a, dd b) { return dd_add(a, dd_neg(b)); }

// Double-double product: TwoProd of the leading parts plus the cross terms.
__device__ inline dd dd_mul(dd a, dd b) {
#pragma clang fp contract(off)
  dd p = two_prod(a.hi, b.hi);
  p.lo = __builtin_fma(a.hi, b.lo, p.lo);
  p.lo = __builtin_fma(a.lo, b.hi, p.lo);
  return fast_two_sum(p.hi, p.lo);
}

__device__ inline dd dd_mul_d(dd a, double b) {
#pragma clang fp contract(off)
  dd p = two_prod(a.hi, b);
  p.lo = __builtin_fma(a.lo, b, p.lo);
  return fast_two_sum(p.hi, p.lo);
}

// Quotient by long division: q1 = a.hi / b.hi, the remainder a - q1 b formed in
// double-double, q2 = remainder / b.hi, one more correction q3, renormalized.
__device__ inline dd dd_div(dd a, dd b) {
#pragma clang fp contract(off)
  const double q1 = a.hi / b.hi;
  dd r = dd_sub(a, dd_mul_d(b, q1));
  const double q2 = r.hi / b.hi;
  r = dd_sub(r, dd_mul_d(b, q2));
  const double q3 = r.hi / b.hi;
  dd q = fast_two_sum(q1, q2);
  return dd_add(q, dd{q3, 0.0});
}

// Square root by one Newton step on the double root (Karp's form):
// x = 1 / sqrt(a.hi) in double, y = a.hi x, sqrt(a) ~ y + x (a - y^2) / 2.
__device__ inline dd dd_sqrt(dd a) {
#pragma clang fp contract(off)
  if (a.hi <= 0.0) return {0.0, 0.0};
  const double x = 1.0 / __builtin_sqrt(a.hi);
  const double y = a.hi * x;
  const dd y2 = two_prod(y, y);
  const dd diff = dd_sub(a, y2);
  const double corr = (diff.hi * x) * 0.5;
  return two_sum(y, corr);
}

}  // namespace
}  // namespace mdg

/*
 * CPU oracle for the multiple-double matrix product C = A.B -- TEST INFRASTRUCTURE.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg load this
 * library.  The GPU product path never links, loads or calls it, and it shares no
 * code with that path: everything here is written from the paper (Chen and
 * Verschelde, "Multiple Double Arithmetic on NVIDIA Tensor Cores") and from the
 * published error-free transformation literature, in plain C11 with OpenMP.
 *
 * Contents
 *   1. Error-free transformations (section 1: the next double of a multiple
 *      double carries the error of the working precision).
 *   2. Classic multiple-double arithmetic and the classic GEMM, one inner
 *      product per output element computed sequentially in k -- the
 *      regular-core comparison of section 4 (bottom-up method).  Double-double
 *      uses the Dekker / Hida-Li-Bailey add and multiply; any limb count uses
 *      an exact expansion (Shewchuk's grow-expansion and compress) rounded to
 *      L limbs after every multiply-add.
 *   3. Exponents and the exact splitter (sections 2 and 3): the value of every
 *      element is formed exactly as a big integer and its magnitude is cut into
 *      13-bit fields on the shared grid of its row (A) or column (B).
 *   4. Slice-pair and level products in exact int64 arithmetic (section 2,
 *      equations (1)-(3) and the rewritten product).
 *
 * Layouts match the product's boundary: an operand with L limbs is
 * [L][rows][cols] float64, digits are [S][rows][cols] float64 (integer valued),
 * level products are [T+1][m][n] int64.
 *
 * Build with -ffp-contract=off: the error-free transformations rely on every
 * sum and product being rounded separately.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_ERANGE -2 /* an element violates |V(x)| < 2^E on its grid */

/* ------------------------------------------------------------------------- */
/* 1. Error-free transformations                                             */
/* ------------------------------------------------------------------------- */

/* Knuth's TwoSum: s = fl(a+b), e = a + b - s exactly (no ordering condition). */
static inline void two_sum(double a, double b, double* s, double* e) {
  double x = a + b;
  double bv = x - a;
  double av = x - bv;
  *e = (a - av) + (b - bv);
  *s = x;
}

/* Dekker's FastTwoSum: exact when a == 0 or exponent(a) >= exponent(b). */
static inline void fast_two_sum(double a, double b, double* s, double* e) {
  double x = a + b;
  *e = b - (x - a);
  *s = x;
}

/* TwoProd with a fused multiply-add: p = fl(ab), e = ab - p exactly (no underflow). */
static inline void two_prod(double a, double b, double* p, double* e) {
  double x = a * b;
  *e = fma(a, b, -x);
  *p = x;
}

void oracle_two_sum(int64_t n, const double* a, const double* b, double* s, double* e) {
  for (int64_t i = 0; i < n; ++i) two_sum(a[i], b[i], &s[i], &e[i]);
}

void oracle_fast_two_sum(int64_t n, const double* a, const double* b, double* s, double* e) {
  for (int64_t i = 0; i < n; ++i) fast_two_sum(a[i], b[i], &s[i], &e[i]);
}

void oracle_two_prod(int64_t n, const double* a, const double* b, double* p, double* e) {
  for (int64_t i = 0; i < n; ++i) two_prod(a[i], b[i], &p[i], &e[i]);
}

/* ------------------------------------------------------------------------- */
/* 2a. Double-double arithmetic (Dekker 1971; Hida, Li and Bailey 2001)       */
/* ------------------------------------------------------------------------- */

/* Accurate double-double addition: both pairs of limbs are added with TwoSum and
 * the result is renormalized twice with FastTwoSum. */
static inline void dd_add(const double* a, const double* b, double* r) {
  double s1, s2, t1, t2;
  two_sum(a[0], b[0], &s1, &s2);
  two_sum(a[1], b[1], &t1, &t2);
  s2 += t1;
  fast_two_sum(s1, s2, &s1, &s2);
  s2 += t2;
  fast_two_sum(s1, s2, &r[0], &r[1]);
}

/* Double-double multiplication: exact product of the leading limbs plus the two
 * cross products, renormalized with FastTwoSum. */
static inline void dd_mul(const double* a, const double* b, double* r) {
  double p1, p2;
  two_prod(a[0], b[0], &p1, &p2);
  p2 += a[0] * b[1] + a[1] * b[0];
  fast_two_sum(p1, p2, &r[0], &r[1]);
}

/* ------------------------------------------------------------------------- */
/* 2b. Any limb count: exact expansions (Shewchuk 1997) rounded to L limbs    */
/* ------------------------------------------------------------------------- */

#define MAXLIMBS 16
/* terms of one multiply-add: L + L(L+1) + L - 1 = 303 for L = 16 */
#define MAXTERMS 320

/* Grow-Expansion with zero elimination: h = e + b exactly.  e holds elen
 * nonoverlapping components in increasing magnitude; so does h. */
static int grow_expansion(const double* e, int elen, double b, double* h) {
  double q = b, hh;
  int hlen = 0;
  for (int i = 0; i < elen; ++i) {
    two_sum(q, e[i], &q, &hh);
    if (hh != 0.0) h[hlen++] = hh;
  }
  if (q != 0.0 || hlen == 0) h[hlen++] = q;
  return hlen;
}

/* Compress: same value, nonoverlapping, increasing magnitude, and the largest
 * component approximates the whole sum to within one of its ulps. */
static int compress(const double* e, int elen, double* h) {
  double g[MAXTERMS];
  double q = e[elen - 1], small;
  int bottom = elen - 1;
  for (int i = elen - 2; i >= 0; --i) {
    double big;
    fast_two_sum(q, e[i], &big, &small);
    if (small != 0.0) {
      g[bottom--] = big;
      q = small;
    } else {
      q = big;
    }
  }
  g[bottom] = q;
  int top = 0;
  for (int i = bottom + 1; i < elen; ++i) {
    double big;
    fast_two_sum(g[i], q, &big, &small);
    if (small != 0.0) h[top++] = small;
    q = big;
  }
  h[top] = q;
  return top + 1;
}

/* acc <- acc + a*b rounded to L limbs.  The exact products a_i b_j with
 * i + j < L (both TwoProd halves) and the rounded products with i + j == L are
 * summed exactly with the L limbs of acc; the exact sum is then cut into L
 * limbs from the top, each the leading component of the compressed remainder. */
static void md_fma(int L, double* acc, const double* a, const double* b) {
  double terms[MAXTERMS];
  int nt = 0;
  for (int l = 0; l < L; ++l) terms[nt++] = acc[l];
  for (int i = 0; i < L; ++i)
    for (int j = 0; j < L; ++j) {
      if (i + j < L) {
        double p, e;
        two_prod(a[i], b[j], &p, &e);
        terms[nt++] = p;
        terms[nt++] = e;
      } else if (i + j == L) {
        terms[nt++] = a[i] * b[j];
      }
    }
  double h[MAXTERMS], h2[MAXTERMS];
  int hlen = 0;
  for (int t = 0; t < nt; ++t) {
    if (terms[t] == 0.0) continue;
    hlen = grow_expansion(h, hlen, terms[t], h2);
    memcpy(h, h2, sizeof(double) * (size_t)hlen);
  }
  for (int l = 0; l < L; ++l) {
    if (hlen == 0 || (hlen == 1 && h[0] == 0.0)) {
      acc[l] = 0.0;
      hlen = 0;
      continue;
    }
    hlen = compress(h, hlen, h2);
    memcpy(h, h2, sizeof(double) * (size_t)hlen);
    acc[l] = h[hlen - 1];
    hlen -= 1;
  }
}

/* Per-operation entry points, vectorized over n elements (limb-major [L][n]). */
void oracle_md_fma(int L, int64_t n, const double* acc, const double* a, const double* b, double* out) {
  double x[MAXLIMBS], y[MAXLIMBS], z[MAXLIMBS];
  if (L < 1 || L > MAXLIMBS) return;
  for (int64_t e = 0; e < n; ++e) {
    for (int l = 0; l < L; ++l) {
      z[l] = acc[l * n + e];
      x[l] = a[l * n + e];
      y[l] = b[l * n + e];
    }
    md_fma(L, z, x, y);
    for (int l = 0; l < L; ++l) out[l * n + e] = z[l];
  }
}

void oracle_dd_add(int64_t n, const double* a, const double* b, double* out) {
  for (int64_t e = 0; e < n; ++e) {
    double x[2] = {a[e], a[n + e]}, y[2] = {b[e], b[n + e]}, r[2];
    dd_add(x, y, r);
    out[e] = r[0];
    out[n + e] = r[1];
  }
}

void oracle_dd_mul(int64_t n, const double* a, const double* b, double* out) {
  for (int64_t e = 0; e < n; ++e) {
    double x[2] = {a[e], a[n + e]}, y[2] = {b[e], b[n + e]}, r[2];
    dd_mul(x, y, r);
    out[e] = r[0];
    out[n + e] = r[1];
  }
}

/* Classic GEMM: C[i][j] = sum over kk of A[i][kk] * B[kk][j], each inner product
 * accumulated sequentially in kk in L-limb arithmetic, one element at a time.
 * variant 0: double-double add and multiply (L must be 2), rounded twice per step;
 * variant 1: exact multiply-add rounded once per step (any L in 1..16).
 * Rows [row_begin, row_end) are computed; nthreads <= 0 uses the OpenMP default.
 * Returns the number of threads used, or a negative status. */
int oracle_classic_gemm(int64_t m, int64_t n, int64_t k, int L, const double* A, const double* B, double* C,
                        int64_t row_begin, int64_t row_end, int variant, int nthreads) {
  if (L < 1 || L > MAXLIMBS || m < 0 || n < 0 || k < 0) return ORACLE_EINVAL;
  if (variant == 0 && L != 2) return ORACLE_EINVAL;
  if (row_begin < 0) row_begin = 0;
  if (row_end > m || row_end < 0) row_end = m;
  /* B transposed once so that every inner product reads contiguous limbs. */
  double* Bt = (double*)malloc(sizeof(double) * (size_t)(n * k * L + 1));
  if (!Bt) return ORACLE_EINVAL;
  for (int64_t kk = 0; kk < k; ++kk)
    for (int64_t j = 0; j < n; ++j)
      for (int l = 0; l < L; ++l) Bt[(j * k + kk) * L + l] = B[(int64_t)l * k * n + kk * n + j];
  int used = 1;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#endif
#pragma omp parallel
  {
#ifdef _OPENMP
#pragma omp single
    used = omp_get_num_threads();
#endif
    double* a = (double*)malloc(sizeof(double) * (size_t)(k * L + 1));
#pragma omp for schedule(dynamic, 1)
    for (int64_t i = row_begin; i < row_end; ++i) {
      for (int64_t kk = 0; kk < k; ++kk)
        for (int l = 0; l < L; ++l) a[kk * L + l] = A[(int64_t)l * m * k + i * k + kk];
      for (int64_t j = 0; j < n; ++j) {
        double acc[MAXLIMBS] = {0};
        const double* bj = Bt + j * k * L;
        if (variant == 0) {
          for (int64_t kk = 0; kk < k; ++kk) {
            double p[2];
            dd_mul(a + kk * 2, bj + kk * 2, p);
            dd_add(acc, p, acc);
          }
        } else {
          for (int64_t kk = 0; kk < k; ++kk) md_fma(L, acc, a + kk * L, bj + kk * L);
        }
        for (int l = 0; l < L; ++l) C[(int64_t)l * m * n + i * n + j] = acc[l];
      }
    }
    free(a);
  }
  free(Bt);
  return used;
}

/* ------------------------------------------------------------------------- */
/* 3. Exponents and the exact splitter                                        */
/* ------------------------------------------------------------------------- */

/* frexp exponent: x = f 2^e with 1/2 <= |f| < 1; the exponent of 0 is "minus infinity". */
static inline int frexp_exp(double x) {
  int e;
  (void)frexp(x, &e);
  return e;
}

/* E of every row (axis 0) or column (axis 1) of the leading-limb plane X0
 * [rows][cols]: the largest frexp exponent of a nonzero entry; 0 when the line
 * is all zero (the paper's zero case: nothing to balance). */
int oracle_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E) {
  if (rows < 0 || cols < 0 || (axis != 0 && axis != 1)) return ORACLE_EINVAL;
  int64_t nlines = axis == 0 ? rows : cols, len = axis == 0 ? cols : rows;
#pragma omp parallel for schedule(static)
  for (int64_t line = 0; line < nlines; ++line) {
    int have = 0, best = 0;
    for (int64_t t = 0; t < len; ++t) {
      double x = axis == 0 ? X0[line * cols + t] : X0[t * cols + line];
      if (x == 0.0) continue;
      int e = frexp_exp(x);
      if (!have || e > best) best = e;
      have = 1;
    }
    E[line] = have ? best : 0;
  }
  return ORACLE_OK;
}

/* A big signed integer, two's complement, little-endian 64-bit words, wide
 * enough for any finite double times 2^1074 (below 2^2098) and the sum of a
 * few of them. */
#define BIGW 36
typedef struct {
  uint64_t w[BIGW];
} bigint;

/* x += sgn * M * 2^sh, with M < 2^64 and 0 <= sh. */
static void big_add_shifted(bigint* x, uint64_t M, int sh, int sgn) {
  bigint t;
  memset(&t, 0, sizeof t);
  int wi = sh / 64, bi = sh % 64;
  if (wi < BIGW) t.w[wi] = M << bi;
  if (bi && wi + 1 < BIGW) t.w[wi + 1] = M >> (64 - bi);
  if (sgn < 0) { /* t = -t */
    uint64_t carry = 1;
    for (int i = 0; i < BIGW; ++i) {
      uint64_t v = ~t.w[i] + carry;
      carry = (carry && v == 0) ? 1 : 0;
      t.w[i] = v;
    }
  }
  uint64_t carry = 0;
  for (int i = 0; i < BIGW; ++i) {
    uint64_t s = x->w[i] + t.w[i];
    uint64_t c1 = s < x->w[i];
    uint64_t s2 = s + carry;
    uint64_t c2 = s2 < s;
    x->w[i] = s2;
    carry = c1 | c2;
  }
}

static int big_is_negative(const bigint* x) { return (int)(x->w[BIGW - 1] >> 63); }

static void big_negate(bigint* x) {
  uint64_t carry = 1;
  for (int i = 0; i < BIGW; ++i) {
    uint64_t v = ~x->w[i] + carry;
    carry = (carry && v == 0) ? 1 : 0;
    x->w[i] = v;
  }
}

/* Bit `pos` of a nonnegative big integer (0 for pos < 0 or beyond the top). */
static inline int big_bit(const bigint* x, int pos) {
  if (pos < 0 || pos >= 64 * BIGW) return 0;
  return (int)((x->w[pos / 64] >> (pos % 64)) & 1u);
}

/* Split one element with L limbs (stride between limbs `ls`) on the grid of
 * exponent E into S digits of w bits (stride between digits `ds`).
 *
 * The exact value V = sum of the limbs is formed as the integer V * 2^1074.  Its
 * magnitude, read on the grid whose unit is u = 2^(E - w S), gives
 * D = floor(|V| / u) < 2^(w S); digit s is the w-bit field of D holding
 * 2^(w (S-1-s)) .. 2^(w (S-s)) - 1, carrying the sign of V.  For w = 13 these are
 * the truncated 13-bit quarters of the worked example of section 2, taken of the
 * exact value on a balanced grid (sections 2 and 3), so a limb of opposite sign
 * borrows from the limbs above it exactly as the 2^-52 transfer of section 3 does.
 * Wider digits are the same cut with fewer, longer fields (the slice width is
 * bounded by the exactness condition (NBound) of section 2, not by 13). */
static int split_one(const double* x, int64_t ls, int L, int E, int S, int w, double* d, int64_t ds) {
  bigint v;
  memset(&v, 0, sizeof v);
  for (int l = 0; l < L; ++l) {
    double xl = x[l * ls];
    if (xl == 0.0) continue;
    int e;
    double f = frexp(fabs(xl), &e);          /* |xl| = f 2^e, f in [1/2, 1) */
    uint64_t M = (uint64_t)ldexp(f, 53);      /* integer significand, exact */
    int sh = e - 53 + 1074;                   /* |xl| 2^1074 = M 2^sh */
    if (sh < 0) {                             /* subnormal: drop the zero low bits */
      M >>= -sh;
      sh = 0;
    }
    big_add_shifted(&v, M, sh, xl < 0 ? -1 : 1);
  }
  int neg = big_is_negative(&v);
  if (neg) big_negate(&v);
  /* bit position (in v) of the grid unit u = 2^(E - w S) */
  int base = E - w * S + 1074;
  /* every bit of |V| at or above 2^E must be zero */
  for (int pos = (base + w * S < 0 ? 0 : base + w * S); pos < 64 * BIGW; ++pos)
    if (big_bit(&v, pos)) return ORACLE_ERANGE;
  for (int s = 0; s < S; ++s) {
    int lo = base + w * (S - 1 - s);
    int digit = 0;
    for (int b = w - 1; b >= 0; --b) digit = 2 * digit + big_bit(&v, lo + b);
    d[s * ds] = neg ? -(double)digit : (double)digit;
    if (digit == 0) d[s * ds] = 0.0;
  }
  return ORACLE_OK;
}

/* Digits of w bits (1 <= w <= 26) of an operand X [L][rows][cols] on the grids E
 * (per row for axis 0, per column for axis 1), written to D [S][rows][cols]. */
int oracle_split_bits(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X, const int32_t* E,
                      double* D) {
  if (rows < 0 || cols < 0 || L < 1 || L > 16 || S < 1 || S > 128 || w < 1 || w > 26 || (axis != 0 && axis != 1))
    return ORACLE_EINVAL;
  int64_t plane = rows * cols;
  int status = ORACLE_OK;
#pragma omp parallel for schedule(static)
  for (int64_t idx = 0; idx < plane; ++idx) {
    int64_t r = idx / (cols ? cols : 1), c = idx % (cols ? cols : 1);
    int e = axis == 0 ? E[r] : E[c];
    int st = split_one(X + idx, plane, L, e, S, w, D + idx, plane);
    if (st != ORACLE_OK) {
#pragma omp atomic write
      status = st;
    }
  }
  return status;
}

/* The 13-bit digits of section 2. */
int oracle_split(int64_t rows, int64_t cols, int L, int S, int axis, const double* X, const int32_t* E, double* D) {
  return oracle_split_bits(rows, cols, L, S, 13, axis, X, E, D);
}

/* ------------------------------------------------------------------------- */
/* 4. Slice-pair and level products in int64                                  */
/* ------------------------------------------------------------------------- */

/* Level products G_t = sum over p + q = t (0 <= p, q < S) of DA_p DB_q for
 * t = 0..T, accumulated exactly in int64 (|G_t| < 2^63 is checked by the caller's
 * choice of k).  DA [S][m][k], DB [S][k][n], G [T+1][m][n].
 * per_pair != 0 instead writes every kept pair P_pq = DA_p DB_q to G [S][S][m][n]
 * (pairs with p + q > T are left untouched). */
int oracle_levels(int64_t m, int64_t n, int64_t k, int S, int T, int per_pair, const double* DA, const double* DB,
                  int64_t* G) {
  if (m < 0 || n < 0 || k < 0 || S < 1 || T < 0 || T > 2 * S - 2) return ORACLE_EINVAL;
  int64_t* ia = (int64_t*)malloc(sizeof(int64_t) * (size_t)(S * m * k + 1));
  int64_t* ib = (int64_t*)malloc(sizeof(int64_t) * (size_t)(S * k * n + 1));
  if (!ia || !ib) {
    free(ia);
    free(ib);
    return ORACLE_EINVAL;
  }
  for (int64_t i = 0; i < S * m * k; ++i) ia[i] = (int64_t)DA[i];
  for (int64_t i = 0; i < S * k * n; ++i) ib[i] = (int64_t)DB[i];
  int64_t mn = m * n;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t i = 0; i < m; ++i) {
    int64_t* row = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1));
    if (!per_pair)
      for (int t = 0; t <= T; ++t)
        for (int64_t j = 0; j < n; ++j) G[(int64_t)t * mn + i * n + j] = 0;
    for (int p = 0; p < S; ++p)
      for (int q = 0; q < S; ++q) {
        if (p + q > T) continue;
        for (int64_t j = 0; j < n; ++j) row[j] = 0;
        const int64_t* a = ia + (int64_t)p * m * k + i * k;
        const int64_t* b = ib + (int64_t)q * k * n;
        for (int64_t kk = 0; kk < k; ++kk) {
          int64_t av = a[kk];
          if (av == 0) continue;
          const int64_t* bk = b + kk * n;
          for (int64_t j = 0; j < n; ++j) row[j] += av * bk[j];
        }
        int64_t* out = per_pair ? G + ((int64_t)p * S + q) * mn + i * n : G + (int64_t)(p + q) * mn + i * n;
        if (per_pair) {
          for (int64_t j = 0; j < n; ++j) out[j] = row[j];
        } else {
          for (int64_t j = 0; j < n; ++j) out[j] += row[j];
        }
      }
    free(row);
  }
  free(ia);
  free(ib);
  return ORACLE_OK;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------- */
/* 5. Householder QR in double-double arithmetic (the downstream application  */
/*    of multiple-double products that the paper names as future work)        */
/* ------------------------------------------------------------------------- */

/* Double-double quotient by long division (Hida, Li and Bailey): q1 = a0 / b0,
 * the remainder a - q1 b in double-double, q2 and q3 from the next remainders. */
static void dd_mul_d(const double* a, double b, double* r) {
  double p1, p2;
  two_prod(a[0], b, &p1, &p2);
  p2 += a[1] * b;
  fast_two_sum(p1, p2, &r[0], &r[1]);
}

static void dd_sub(const double* a, const double* b, double* r) {
  double nb[2] = {-b[0], -b[1]};
  dd_add(a, nb, r);
}

static void dd_div(const double* a, const double* b, double* q) {
  double t[2], r[2], r2[2];
  double q1 = a[0] / b[0];
  dd_mul_d(b, q1, t);
  dd_sub(a, t, r);
  double q2 = r[0] / b[0];
  dd_mul_d(b, q2, t);
  dd_sub(r, t, r2);
  double q3 = r2[0] / b[0];
  double s[2], e3[2] = {q3, 0.0};
  fast_two_sum(q1, q2, &s[0], &s[1]);
  dd_add(s, e3, q);
}

/* Double-double square root by one Newton step on the double root (Karp):
 * x = 1/sqrt(a0), y = a0 x, sqrt(a) = y + x (a - y^2) / 2. */
static void dd_sqrt(const double* a, double* r) {
  if (a[0] <= 0.0) {
    r[0] = r[1] = 0.0;
    return;
  }
  double x = 1.0 / sqrt(a[0]);
  double y = a[0] * x;
  double y2[2], d[2];
  two_prod(y, y, &y2[0], &y2[1]);
  dd_sub(a, y2, d);
  two_sum(y, d[0] * x * 0.5, &r[0], &r[1]);
}

/* A = Q R for A [2][m][n] (double-double, m >= n), unblocked: for each column j
 * the Householder vector of x = A(j:m, j) after Golub and Van Loan (v_1 without
 * cancellation, R(j, j) = ||x|| >= 0), then H_j applied to the columns right of
 * j, each by w = v^T a, a <- a - tau w v.  On return A holds R on and above the
 * diagonal and v (v_1 = 1 implicit) below it; tau [2][n]. */
int oracle_qr_dd(int64_t m, int64_t n, double* A, double* tau) {
  if (m < 1 || n < 1 || m < n) return ORACLE_EINVAL;
  const int64_t P = m * n;
#define AT(r, c, l) A[(l) * P + (r) * n + (c)]
  for (int64_t j = 0; j < n; ++j) {
    double sigma[2] = {0.0, 0.0}, t[2];
    for (int64_t r = j + 1; r < m; ++r) {
      double a[2] = {AT(r, j, 0), AT(r, j, 1)};
      dd_mul(a, a, t);
      dd_add(sigma, t, sigma);
    }
    double x1[2] = {AT(j, j, 0), AT(j, j, 1)}, tj[2], diag[2];
    int mode;
    double v1[2] = {1.0, 0.0};
    if (sigma[0] == 0.0) {
      mode = x1[0] < 0.0 ? 1 : 0;
      tj[0] = mode ? 2.0 : 0.0;
      tj[1] = 0.0;
      diag[0] = mode ? -x1[0] : x1[0];
      diag[1] = mode ? -x1[1] : x1[1];
    } else {
      double s2[2], mu[2], v1sq[2], num[2], den[2];
      dd_mul(x1, x1, s2);
      dd_add(s2, sigma, s2);
      dd_sqrt(s2, mu);
      if (x1[0] <= 0.0) {
        dd_sub(x1, mu, v1);
      } else {
        double xs[2], q[2];
        dd_add(x1, mu, xs);
        dd_div(sigma, xs, q);
        v1[0] = -q[0];
        v1[1] = -q[1];
      }
      dd_mul(v1, v1, v1sq);
      dd_mul_d(v1sq, 2.0, num);
      dd_add(sigma, v1sq, den);
      dd_div(num, den, tj);
      diag[0] = mu[0];
      diag[1] = mu[1];
      mode = 2;
    }
    AT(j, j, 0) = diag[0];
    AT(j, j, 1) = diag[1];
    tau[j] = tj[0];
    tau[n + j] = tj[1];
    if (mode == 2)
      for (int64_t r = j + 1; r < m; ++r) {
        double a[2] = {AT(r, j, 0), AT(r, j, 1)}, q[2];
        dd_div(a, v1, q);
        AT(r, j, 0) = q[0];
        AT(r, j, 1) = q[1];
      }
    if (mode == 0) continue;
    for (int64_t c = j + 1; c < n; ++c) {
      double w[2] = {AT(j, c, 0), AT(j, c, 1)};
      if (mode == 2)
        for (int64_t r = j + 1; r < m; ++r) {
          double v[2] = {AT(r, j, 0), AT(r, j, 1)}, a[2] = {AT(r, c, 0), AT(r, c, 1)};
          dd_mul(v, a, t);
          dd_add(w, t, w);
        }
      double tw[2], a0[2] = {AT(j, c, 0), AT(j, c, 1)};
      dd_mul(tj, w, tw);
      dd_sub(a0, tw, a0);
      AT(j, c, 0) = a0[0];
      AT(j, c, 1) = a0[1];
      if (mode == 2)
        for (int64_t r = j + 1; r < m; ++r) {
          double v[2] = {AT(r, j, 0), AT(r, j, 1)}, a[2] = {AT(r, c, 0), AT(r, c, 1)};
          dd_mul(tw, v, t);
          dd_sub(a, t, a);
          AT(r, c, 0) = a[0];
          AT(r, c, 1) = a[1];
        }
    }
  }
#undef AT
  return ORACLE_OK;
}

/* Check a factorization in double-double arithmetic: QR [2][m][n] holds R and
 * the vectors as oracle_qr_dd leaves them, tau [2][n].  Forms the thin Q (m x n:
 * the reflections applied, last to first, to the first n columns of I), then
 * out[0] = max |A0 - Q R| / max |A0| and out[1] = max |Q^T Q - I|, each entry
 * formed in double-double.  Q [2][m][n] is returned as well (may be NULL). */
int oracle_qr_dd_check(int64_t m, int64_t n, const double* A0, const double* QR, const double* tau, double* out,
                       double* Qout) {
  if (m < 1 || n < 1 || m < n) return ORACLE_EINVAL;
  const int64_t P = m * n;
  double* Q = (double*)malloc(sizeof(double) * 2 * (size_t)P);
  if (!Q) return ORACLE_EINVAL;
#define QV(r, c, l) QR[(l) * P + (r) * n + (c)]
#define QQ(r, c, l) Q[(l) * P + (r) * n + (c)]
  for (int64_t r = 0; r < m; ++r)
    for (int64_t c = 0; c < n; ++c) {
      QQ(r, c, 0) = r == c ? 1.0 : 0.0;
      QQ(r, c, 1) = 0.0;
    }
  for (int64_t j = n - 1; j >= 0; --j) {
    double tj[2] = {tau[j], tau[n + j]}, t[2];
    if (tj[0] == 0.0) continue;
    for (int64_t c = 0; c < n; ++c) {
      double w[2] = {QQ(j, c, 0), QQ(j, c, 1)};
      for (int64_t r = j + 1; r < m; ++r) {
        double v[2] = {QV(r, j, 0), QV(r, j, 1)}, q[2] = {QQ(r, c, 0), QQ(r, c, 1)};
        dd_mul(v, q, t);
        dd_add(w, t, w);
      }
      double tw[2], q0[2] = {QQ(j, c, 0), QQ(j, c, 1)};
      dd_mul(tj, w, tw);
      dd_sub(q0, tw, q0);
      QQ(j, c, 0) = q0[0];
      QQ(j, c, 1) = q0[1];
      for (int64_t r = j + 1; r < m; ++r) {
        double v[2] = {QV(r, j, 0), QV(r, j, 1)}, q[2] = {QQ(r, c, 0), QQ(r, c, 1)};
        dd_mul(tw, v, t);
        dd_sub(q, t, q);
        QQ(r, c, 0) = q[0];
        QQ(r, c, 1) = q[1];
      }
    }
  }
  double amax = 0.0, res = 0.0, orth = 0.0;
  for (int64_t e = 0; e < P; ++e) amax = fmax(amax, fabs(A0[e]));
#pragma omp parallel for reduction(max : res) schedule(static)
  for (int64_t r = 0; r < m; ++r)
    for (int64_t c = 0; c < n; ++c) {
      double s[2] = {0.0, 0.0}, t[2];
      for (int64_t l = 0; l <= c; ++l) {
        double q[2] = {QQ(r, l, 0), QQ(r, l, 1)}, rr[2] = {QV(l, c, 0), QV(l, c, 1)};
        dd_mul(q, rr, t);
        dd_add(s, t, s);
      }
      double a[2] = {A0[r * n + c], A0[P + r * n + c]}, d[2];
      dd_sub(a, s, d);
      res = fmax(res, fabs(d[0]));
    }
#pragma omp parallel for reduction(max : orth) schedule(static)
  for (int64_t i = 0; i < n; ++i)
    for (int64_t c = 0; c < n; ++c) {
      double s[2] = {i == c ? -1.0 : 0.0, 0.0}, t[2];
      for (int64_t r = 0; r < m; ++r) {
        double a[2] = {QQ(r, i, 0), QQ(r, i, 1)}, b[2] = {QQ(r, c, 0), QQ(r, c, 1)};
        dd_mul(a, b, t);
        dd_add(s, t, s);
      }
      orth = fmax(orth, fabs(s[0]));
    }
#undef QV
#undef QQ
  out[0] = amax > 0.0 ? res / amax : res;
  out[1] = orth;
  if (Qout) memcpy(Qout, Q, sizeof(double) * 2 * (size_t)P);
  free(Q);
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* 6. Taylor series of the solution of a linear system of power series (the   */
/*    application the paper names for the QR, section 5)                        */
/* ------------------------------------------------------------------------- */

/* A(t) X(t) = B(t) modulo t^(d+1) for A [d+1][2][n][n], B [d+1][2][n][r]:
 * comparing the coefficients of t^k, A_0 X_k = B_k - sum_{i=1..k} A_i X_{k-i}.
 * Each X_k is formed as written, in double-double: the right-hand side entry by
 * entry (each product sum in increasing index, then subtracted), then the
 * solve with the QR of A_0 (oracle_qr_dd): y = Q^T rhs by the reflections
 * H_0, H_1, ... in turn, then back substitution R x = y.  X [d+1][2][n][r]. */
int oracle_taylor_dd(int64_t n, int64_t r, int d, const double* A, const double* B, double* X) {
  if (n < 1 || r < 1 || d < 0) return ORACLE_EINVAL;
  const int64_t PA = n * n, PB = n * r;
  double* QR = (double*)malloc(sizeof(double) * 2 * (size_t)PA);
  double* tau = (double*)malloc(sizeof(double) * 2 * (size_t)n);
  double* y = (double*)malloc(sizeof(double) * 2 * (size_t)PB);
  if (!QR || !tau || !y) {
    free(QR);
    free(tau);
    free(y);
    return ORACLE_EINVAL;
  }
  memcpy(QR, A, sizeof(double) * 2 * (size_t)PA);
  int st = oracle_qr_dd(n, n, QR, tau);
#define QA(i, c, l) QR[(l) * PA + (i) * n + (c)]
#define YY(i, c, l) y[(l) * PB + (i) * r + (c)]
  for (int k = 0; st == ORACLE_OK && k <= d; ++k) {
    const double* Bk = B + (int64_t)k * 2 * PB;
    double* Xk = X + (int64_t)k * 2 * PB;
    /* rhs = B_k - sum_{i=1..k} A_i X_{k-i} */
    for (int64_t i = 0; i < n; ++i)
      for (int64_t c = 0; c < r; ++c) {
        double v[2] = {Bk[i * r + c], Bk[PB + i * r + c]}, t[2];
        for (int a = 1; a <= k; ++a) {
          const double* Ai = A + (int64_t)a * 2 * PA;
          const double* Xj = X + (int64_t)(k - a) * 2 * PB;
          double s[2] = {0.0, 0.0};
          for (int64_t l = 0; l < n; ++l) {
            double p[2] = {Ai[i * n + l], Ai[PA + i * n + l]}, q[2] = {Xj[l * r + c], Xj[PB + l * r + c]};
            dd_mul(p, q, t);
            dd_add(s, t, s);
          }
          dd_sub(v, s, v);
        }
        YY(i, c, 0) = v[0];
        YY(i, c, 1) = v[1];
      }
    /* y = Q^T rhs: H_j = I - tau_j v_j v_j^T for j = 0, 1, ... (v_j(j) = 1) */
    for (int64_t j = 0; j < n; ++j) {
      double tj[2] = {tau[j], tau[n + j]}, t[2];
      if (tj[0] == 0.0) continue;
      for (int64_t c = 0; c < r; ++c) {
        double w[2] = {YY(j, c, 0), YY(j, c, 1)};
        for (int64_t i = j + 1; i < n; ++i) {
          double v[2] = {QA(i, j, 0), QA(i, j, 1)}, q[2] = {YY(i, c, 0), YY(i, c, 1)};
          dd_mul(v, q, t);
          dd_add(w, t, w);
        }
        double tw[2], q0[2] = {YY(j, c, 0), YY(j, c, 1)};
        dd_mul(tj, w, tw);
        dd_sub(q0, tw, q0);
        YY(j, c, 0) = q0[0];
        YY(j, c, 1) = q0[1];
        for (int64_t i = j + 1; i < n; ++i) {
          double v[2] = {QA(i, j, 0), QA(i, j, 1)}, q[2] = {YY(i, c, 0), YY(i, c, 1)};
          dd_mul(tw, v, t);
          dd_sub(q, t, q);
          YY(i, c, 0) = q[0];
          YY(i, c, 1) = q[1];
        }
      }
    }
    /* R x = y, rows from the bottom */
    for (int64_t c = 0; c < r; ++c)
      for (int64_t i = n - 1; i >= 0; --i) {
        double s[2] = {YY(i, c, 0), YY(i, c, 1)}, t[2];
        for (int64_t l = i + 1; l < n; ++l) {
          double rr[2] = {QA(i, l, 0), QA(i, l, 1)}, x[2] = {Xk[l * r + c], Xk[PB + l * r + c]};
          dd_mul(rr, x, t);
          dd_sub(s, t, s);
        }
        double rii[2] = {QA(i, i, 0), QA(i, i, 1)}, q[2];
        dd_div(s, rii, q);
        Xk[i * r + c] = q[0];
        Xk[PB + i * r + c] = q[1];
      }
  }
#undef QA
#undef YY
  free(QR);
  free(tau);
  free(y);
  return st;
}

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

// Blocked Householder QR of a double-double matrix: the downstream
// application the paper names as future work (section 5), with its trailing
// updates on the multiple-double product of this library.
//
// A [2][m][n] (limb-major double-double, m >= n) is factored as A = Q R with
// Q = H_0 H_1 ... H_{n-1}, H_j = I - tau_j v_j v_j^T (Householder reflections,
// v_j(j) = 1, v_j zero above row j).  Panels of nb <= 64 columns are factored in
// double-double arithmetic (dd.h) by many workgroups, one launch per column
// (see qr_col_step_kernel); the panel's reflections are
// accumulated in the compact form I - V T V^T (T upper triangular, by the
// recursive form of Elmroth and Gustavson), and the trailing columns are updated as
//     A2 <- A2 - V (T^T (V^T A2))
// with three products on mdgemm_ex (double-double in, double-double out, at the
// adaptive digit width).  On return A holds R on and above the diagonal and the
// vectors v_j below it (LAPACK's convention), tau the scalars tau_j.
//
// Householder vector of x = A(j:m, j) (Golub and Van Loan, the algorithm that
// keeps v_1 free of cancellation): sigma = x(2:)^T x(2:), mu = sqrt(x_1^2 +
// sigma); v_1 = x_1 - mu if x_1 <= 0, else -sigma / (x_1 + mu); tau = 2 v_1^2 /
// (sigma + v_1^2); v = x / v_1; then H x = mu e_1, so the diagonal of R is
// nonnegative.  sigma = 0: tau = 0 (x_1 >= 0) or tau = 2 (x_1 < 0), v = e_1 (the
// stored entries below the pivot are set to zero).  Squares that underflow
// (|a| below about 1e-154) count as zero: columns of such entries only are
// outside the range of this factorization.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <type_traits>

#include "dd.h"
#include "internal.h"
#include "mdgemm.h"

namespace mdg {
namespace {

constexpr int kMaxNb = 64;  // panel width; the kernels take its columns 32 at a time

__device__ inline dd ldd(const double* P, int64_t plane, int64_t idx) { return {P[idx], P[plane + idx]}; }
__device__ inline void std_(double* P, int64_t plane, int64_t idx, dd v) {
  P[idx] = v.hi;
  P[plane + idx] = v.lo;
}

// The sum of x[0 .. N) (N a power of two) in a fixed pairwise tree,
// ((x0 + x1) + (x2 + x3)) + ...: depth log2 N instead of N - 1 dependent adds,
// the same order wherever it is called.  x is overwritten.
template <int N>
__device__ inline dd tree_sum(dd* x) {
  static_assert(N > 0 && (N & (N - 1)) == 0, "a power of two");
#pragma unroll
  for (int w = 1; w < N; w *= 2)
#pragma unroll
    for (int i = 0; i + w < N; i += 2 * w) x[i] = dd_add(x[i], x[i + w]);
  return x[0];
}

// A panel is factored by many workgroups, one launch per step s = 0 .. jb, each
// workgroup owning kRows consecutive panel rows (8 for panels of at most
// kSmallPanel rows and 16 for at most kShortPanel, so that short panels still
// spread over the chip, 32 above).  Step s finishes column s - 1 and starts
// column s:
//   every block sums the partials of step s - 1 in the same order (so all
//   blocks agree bit for bit): d_c = x^T a_c over the rows below the pivot, x
//   the column s - 1, c >= s - 1 (d_{s-1} = sigma), and takes the pivot row's
//   entries p_c (p_{s-1} = x1); it forms the Householder scalars, block 0 writes
//   the diagonal and tau, and each block scales its rows of x into v = x / v1
//   and applies the reflection to columns c >= s at its rows from the pivot
//   down with w_c = v^T a_c = p_c + d_c / v1 (v is 1 at the pivot);
//   then each block writes its part of d_c for column s (c >= s) and the block
//   holding the pivot row writes that row's entries p_c.
// One reduction per column serves both the norm and the reflection's dot
// products, since both are sums over the rows below the pivot.  The partials
// alternate between two buffers (step s reads buffer (s - 1) & 1 and writes
// s & 1), and every block writes all of its partial slots (zeros where it holds
// no row below the pivot), so a sum never reads a stale or concurrently written
// slot.
constexpr int kPanelRowsSmall = 8, kPanelRowsShort = 16, kPanelRowsTall = 32;
constexpr int64_t kSmallPanel = 1024, kShortPanel = 2048;
constexpr int kColThreads = 256;  // 32 column lanes x 8 row groups
constexpr int kFoldBatch = 8;    // partial sums a thread loads per column group before adding them

constexpr int kRowGroups = kColThreads / 32;                // 8: rows rb + rg + 8 q
constexpr int kColGroups = kMaxNb / 32;                      // columns c0 + 32 h + cc, h < 2
static_assert(kPanelRowsSmall % kRowGroups == 0 && kPanelRowsShort % kRowGroups == 0 &&
                  kPanelRowsTall % kRowGroups == 0 && kMaxNb % 32 == 0,
              "thread layout of the column kernels");
static_assert(kPanelRowsShort <= 64 && kPanelRowsTall <= 64, "one row per thread of the first two waves");

// pd: two buffers of [2][G][kMaxNb] (hi plane, lo plane); prow: two of [2][kMaxNb]
template <int kRows>
__global__ void __launch_bounds__(kColThreads) qr_col_step_kernel(int64_t m, int64_t n, int64_t j0, int jb, int s,
                                                                  double* __restrict__ A, double* __restrict__ tau,
                                                                  double* __restrict__ pd,
                                                                  double* __restrict__ prow) {
  constexpr int kRPT = kRows / kRowGroups;  // rows per thread
  __shared__ dd red2[kColGroups][kColThreads];
  __shared__ dd td[kMaxNb], tw[kMaxNb], vs[kRows], xs[kRows];
  __shared__ dd s_scale, s_tau;
  __shared__ int s_mode;
  const int64_t plane = m * n;
  const int tid = threadIdx.x, cc = tid & 31, rg = tid >> 5;
  const int64_t G = gridDim.x, pplane = G * kMaxNb;
  const int64_t rb = j0 + static_cast<int64_t>(blockIdx.x) * kRows, re = min(m, rb + kRows);
  const int64_t r0 = j0 + s, rp = r0 - 1;  // the pivot rows of column s and of column s - 1
  const double* pd_in = pd + ((s + 1) & 1) * 2 * pplane;
  double* pd_out = pd + (s & 1) * 2 * pplane;
  const double* prow_in = prow + ((s + 1) & 1) * 2 * kMaxNb;
  double* prow_out = prow + (s & 1) * 2 * kMaxNb;

  // Loaded first (none depends on the sums): columns s + 32 h + cc at rows
  // rb + rg + 8 q from the previous pivot down (from the pivot of column s when
  // s = 0), column s - 1 below its pivot (one row per thread of the first
  // kRows), and the pivot row's entries of step s - 1.
  const int64_t rlo = s > 0 ? rp : r0;
  dd av[kColGroups][kRPT];
#pragma unroll
  for (int h = 0; h < kColGroups; ++h) {
    const int c = s + 32 * h + cc;
#pragma unroll
    for (int q = 0; q < kRPT; ++q) {
      const int64_t r = rb + rg + kRowGroups * q;
      av[h][q] = c < jb && r >= rlo && r < re ? ldd(A, plane, r * n + j0 + c) : dd{0.0, 0.0};
    }
  }
  if (s > 0) {
    const int ncols = jb - s + 1;  // c = s - 1 .. jb - 1
    dd xv = {0.0, 0.0}, pv = {0.0, 0.0};
    if (tid < kRows) {
      const int64_t r = rb + tid;
      if (r > rp && r < re) xv = ldd(A, plane, r * n + j0 + s - 1);
    }
    // x1 for thread 0; p_c (c = s + t) for thread 64 + t, which forms tau w_c
    if (tid == 0) pv = ldd(prow_in, kMaxNb, 0);
    if (tid >= 64 && tid < 64 + ncols - 1) pv = ldd(prow_in, kMaxNb, tid - 63);
    // d_c for the columns g = cc and g = 32 + cc of both groups at once:
    // partials b = rg, rg + 8, ... in batches of kFoldBatch loads in flight per
    // group (all of them when G <= 8 kFoldBatch), each batch summed in a tree
    // (entries beyond G are zeros) and the batches in order, then the eight row
    // groups in a tree
    {
      dd sum[kColGroups];
#pragma unroll
      for (int h = 0; h < kColGroups; ++h) sum[h] = {0.0, 0.0};
      for (int64_t b0 = rg; b0 < G; b0 += kRowGroups * kFoldBatch) {
        dd v[kColGroups][kFoldBatch];
#pragma unroll
        for (int h = 0; h < kColGroups; ++h)
#pragma unroll
          for (int u = 0; u < kFoldBatch; ++u) {
            const int64_t b = b0 + kRowGroups * u;
            v[h][u] = b < G && 32 * h + cc < ncols ? ldd(pd_in, pplane, b * kMaxNb + 32 * h + cc) : dd{0.0, 0.0};
          }
#pragma unroll
        for (int h = 0; h < kColGroups; ++h) sum[h] = dd_add(sum[h], tree_sum<kFoldBatch>(v[h]));
      }
#pragma unroll
      for (int h = 0; h < kColGroups; ++h) red2[h][tid] = sum[h];
      __syncthreads();
      if (rg < kColGroups) {
        dd t[kRowGroups];
#pragma unroll
        for (int g = 0; g < kRowGroups; ++g) t[g] = red2[rg][g * 32 + cc];
        td[32 * rg + cc] = tree_sum<kRowGroups>(t);
      }
      __syncthreads();
    }
    // the Householder scalars of column s - 1 from sigma = d_{s-1} and x1 = p_{s-1}
    if (tid == 0) {
      const dd sigma = td[0], x1 = pv;
      dd diag;
      if (sigma.hi == 0.0) {
        s_mode = x1.hi < 0.0 ? 1 : 0;
        s_tau = s_mode ? dd{2.0, 0.0} : dd{0.0, 0.0};
        diag = s_mode ? dd_neg(x1) : x1;
      } else {
        const dd mu = dd_sqrt(dd_add(dd_mul(x1, x1), sigma));
        const dd v1 = x1.hi <= 0.0 ? dd_sub(x1, mu) : dd_neg(dd_div(sigma, dd_add(x1, mu)));
        const dd v1sq = dd_mul(v1, v1);
        s_tau = dd_div(dd_mul_d(v1sq, 2.0), dd_add(sigma, v1sq));
        s_scale = v1;
        s_mode = 2;
        diag = mu;
      }
      if (blockIdx.x == 0) {
        std_(A, plane, rp * n + j0 + s - 1, diag);
        std_(tau, n, j0 + s - 1, s_tau);
      }
    }
    __syncthreads();
    const int mode = s_mode;
    // v at the block's rows (1 at the pivot; mode 2: x / v1 below it, else 0),
    // and tau w_c for c = s + tid: w_c = p_c + d_c / v1 (p_c alone when v = e_1)
    if (tid < kRows) {
      const int64_t r = rb + tid;
      dd v = {0.0, 0.0};
      if (r == rp) {
        v = {1.0, 0.0};
      } else if (r > rp && r < re) {
        v = mode == 2 ? dd_div(xv, s_scale) : dd{0.0, 0.0};
        std_(A, plane, r * n + j0 + s - 1, v);
      }
      vs[tid] = v;
    }
    if (tid >= 64 && tid < 64 + ncols - 1) {
      const int t = tid - 64;
      const dd w = mode == 2 ? dd_add(pv, dd_div(td[t + 1], s_scale)) : pv;
      tw[t] = dd_mul(s_tau, w);
    }
    __syncthreads();
    // a_c <- a_c - (tau w_c) v at the rows from the previous pivot down
#pragma unroll
    for (int h = 0; h < kColGroups; ++h) {
      const int c = s + 32 * h + cc;
      if (c < jb) {
        const dd t = tw[32 * h + cc];
#pragma unroll
        for (int q = 0; q < kRPT; ++q) {
          const int64_t r = rb + rg + kRowGroups * q;
          if (r >= rp && r < re) {
            av[h][q] = dd_sub(av[h][q], dd_mul(t, vs[r - rb]));
            std_(A, plane, r * n + j0 + c, av[h][q]);
          }
        }
      }
    }
  }
  if (s == jb) return;
  // column s below its pivot, from lane cc = 0 of each row group, for all lanes
  if (cc == 0) {
#pragma unroll
    for (int q = 0; q < kRPT; ++q) {
      const int64_t r = rb + rg + kRowGroups * q;
      xs[rg + kRowGroups * q] = r > r0 && r < re ? av[0][q] : dd{0.0, 0.0};
    }
  }
  __syncthreads();
  // partial d_c = x^T a_c over the block's rows below the pivot, for
  // c = s + 32 h + cc (slot 32 h + cc): each thread's rows and then the eight
  // row groups in trees, both column groups in one pass; the pivot row's
  // entries from the block that holds it
  {
    dd acc[kColGroups];
#pragma unroll
    for (int h = 0; h < kColGroups; ++h) {
      const int c = s + 32 * h + cc;
      dd pr[kRPT];
#pragma unroll
      for (int q = 0; q < kRPT; ++q) {
        const int64_t r = rb + rg + kRowGroups * q;
        pr[q] = c < jb && r > r0 && r < re ? dd_mul(xs[rg + kRowGroups * q], av[h][q]) : dd{0.0, 0.0};
        if (c < jb && r == r0) std_(prow_out, kMaxNb, 32 * h + cc, av[h][q]);
      }
      acc[h] = tree_sum<kRPT>(pr);
      red2[h][tid] = acc[h];
    }
    __syncthreads();
    if (rg < kColGroups && 32 * rg < jb - s) {
      dd t[kRowGroups];
#pragma unroll
      for (int g = 0; g < kRowGroups; ++g) t[g] = red2[rg][g * 32 + cc];
      std_(pd_out, pplane, static_cast<int64_t>(blockIdx.x) * kMaxNb + 32 * rg + cc, tree_sum<kRowGroups>(t));
    }
  }
}

// V (mp x jb, dense: 1 on the diagonal, the stored vectors below, 0 above) and
// its transpose Vt (jb x mp), from the factored panel; rows of the panel start
// at row j0 of A.
__global__ void __launch_bounds__(256) qr_pack_v_kernel(int64_t m, int64_t n, int64_t j0, int jb,
                                                        const double* __restrict__ A, double* __restrict__ V,
                                                        double* __restrict__ Vt) {
  const int64_t mp = m - j0, planeA = m * n, planeV = mp * jb;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= planeV) return;
  const int64_t i = e / jb;
  const int c = static_cast<int>(e - i * jb);
  dd v = {0.0, 0.0};
  if (i == c) v = {1.0, 0.0};
  else if (i > c) v = ldd(A, planeA, (j0 + i) * n + j0 + c);
  std_(V, planeV, i * jb + c, v);
  std_(Vt, planeV, static_cast<int64_t>(c) * mp + i, v);
}

// G = V^T V (jb x jb) of the factored panel, in double-double arithmetic, in
// two launches: workgroups of kGramRows rows stage their rows of V (1 on the
// diagonal, the stored vectors below, 0 above) in LDS and write the partial sums
// of all kMaxNb x kMaxNb entries; a second launch (one thread per entry) adds the
// partials of each entry in workgroup order and writes G [2][jb][jb].
constexpr int kGramRows = 32;

__global__ void __launch_bounds__(kColThreads) qr_gram_partial_kernel(int64_t m, int64_t n, int64_t j0, int jb,
                                                                      const double* __restrict__ A,
                                                                      double* __restrict__ pg) {
  __shared__ dd Vs[kGramRows][kMaxNb + 1];
  const int64_t plane = m * n, G = gridDim.x;
  const int tid = threadIdx.x;
  const int64_t rb = j0 + static_cast<int64_t>(blockIdx.x) * kGramRows;
  for (int e = tid; e < kGramRows * kMaxNb; e += kColThreads) {
    const int rr = e / kMaxNb, c = e % kMaxNb;
    const int64_t r = rb + rr;
    dd v = {0.0, 0.0};
    if (r < m && c < jb) {
      if (r == j0 + c) v = {1.0, 0.0};
      else if (r > j0 + c) v = ldd(A, plane, r * n + j0 + c);
    }
    Vs[rr][c] = v;
  }
  __syncthreads();
  for (int e = tid; e < kMaxNb * kMaxNb; e += kColThreads) {
    const int l = e / kMaxNb, c = e % kMaxNb;
    dd s = {0.0, 0.0};
    if (l < jb && c < jb)
      for (int rr = 0; rr < kGramRows; ++rr) s = dd_add(s, dd_mul(Vs[rr][l], Vs[rr][c]));
    std_(pg, G * kMaxNb * kMaxNb, static_cast<int64_t>(blockIdx.x) * kMaxNb * kMaxNb + e, s);
  }
}

// one thread per entry of G, the partials added in workgroup order, eight loads
// issued at a time
constexpr int kGramThreads = 256;

__global__ void __launch_bounds__(kGramThreads) qr_gram_reduce_kernel(int jb, int64_t groups,
                                                                      const double* __restrict__ pg,
                                                                      double* __restrict__ Gout) {
  const int e = blockIdx.x * kGramThreads + threadIdx.x;
  const int l = e / kMaxNb, c = e % kMaxNb;
  if (l >= jb || c >= jb) return;
  const int64_t plane = groups * kMaxNb * kMaxNb;
  dd s = {0.0, 0.0};
  for (int64_t b0 = 0; b0 < groups; b0 += 8) {
    dd v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = b0 + u < groups ? ldd(pg, plane, (b0 + u) * kMaxNb * kMaxNb + e) : dd{0.0, 0.0};
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (b0 + u < groups) s = dd_add(s, v[u]);
  }
  std_(Gout, static_cast<int64_t>(jb) * jb, static_cast<int64_t>(l) * jb + c, s);
}

// T (upper triangular, jb x jb) of I - V T V^T = H_0 ... H_{jb-1} from
// G = V^T V and tau, by the recursive form of the compact WY factor (Elmroth
// and Gustavson): for V = [V1 V2], T = [T11 T12; 0 T22] with T12 = -T11
// (V1^T V2) T22.  The jb columns are padded to 64 (tau = 0, G = 0 there, which
// leaves the leading jb x jb block unchanged) and the recursion runs bottom up:
// at half width h = 1, 2, .., 32, the 32 / h diagonal blocks of width 2h form
// X = G12 T22 (phase 1) and then T12 = -T11 X (phase 2), one entry per thread,
// each a dot product in increasing index order.  Six levels of two phases
// instead of 64 dependent steps.  Writes the transpose Tt.  T, G and X in
// dynamic LDS (kTLds bytes).
constexpr int kTThreads = 1024;
constexpr int kTPad = 64;                                     // the padded width
constexpr int kTX = kTPad * kTPad / 4;                        // entries of X at h = 32
constexpr size_t kTLds = sizeof(dd) * (2 * kTPad * kTPad + kTX);  // 144 KB
static_assert(kMaxNb <= kTPad && kTX <= kTThreads, "one X entry per thread");

__global__ void __launch_bounds__(kTThreads) qr_t_kernel(int jb, int64_t n, int64_t j0,
                                                        const double* __restrict__ G,
                                                        const double* __restrict__ tau,
                                                        double* __restrict__ Tt) {
  extern __shared__ dd tsm[];
  dd* T = tsm;                     // T[i * kTPad + c]
  dd* Gs = tsm + kTPad * kTPad;    // G[l * kTPad + c]
  dd* X = Gs + kTPad * kTPad;      // X of every block of a level, h x h each
  const int tid = threadIdx.x;
  const int64_t pg = static_cast<int64_t>(jb) * jb;
  for (int e = tid; e < kTPad * kTPad; e += kTThreads) {
    const int r = e / kTPad, c = e % kTPad;
    const bool in = r < jb && c < jb;
    Gs[e] = in ? ldd(G, pg, static_cast<int64_t>(r) * jb + c) : dd{0.0, 0.0};
    T[e] = r == c && r < jb ? ldd(tau, n, j0 + r) : dd{0.0, 0.0};
  }
  __syncthreads();
  for (int h = 1; h < kTPad; h *= 2) {
    const int e = tid, hh = h * h, bb = e / hh, w = e % hh, i = w / h, j = w % h;
    const int a = 2 * h * bb;  // the block's first index
    const bool act = e < (kTPad / 2) * h;
    if (act) {  // X(i, j) = sum over l <= j of G(a + i, a + h + l) T(a + h + l, a + h + j)
      dd s = {0.0, 0.0};
      for (int l = 0; l <= j; ++l)
        s = dd_add(s, dd_mul(Gs[(a + i) * kTPad + a + h + l], T[(a + h + l) * kTPad + a + h + j]));
      X[e] = s;
    }
    __syncthreads();
    if (act) {  // T(a + i, a + h + j) = -sum over l >= i of T(a + i, a + l) X(l, j)
      dd s = {0.0, 0.0};
      for (int l = i; l < h; ++l) s = dd_add(s, dd_mul(T[(a + i) * kTPad + a + l], X[bb * hh + l * h + j]));
      T[(a + i) * kTPad + a + h + j] = dd_neg(s);
    }
    __syncthreads();
  }
  for (int e = tid; e < jb * jb; e += kTThreads) {
    const int r = e / jb, c = e % jb;
    std_(Tt, pg, static_cast<int64_t>(c) * jb + r, T[r * kTPad + c]);
  }
}

// Copy the trailing block A(j0:m, c0:n) into a contiguous [2][mp][nc] array.
__global__ void __launch_bounds__(256) qr_pack_block_kernel(int64_t m, int64_t n, int64_t j0, int64_t c0,
                                                            const double* __restrict__ A, double* __restrict__ X) {
  const int64_t mp = m - j0, nc = n - c0, planeX = mp * nc;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= planeX) return;
  const int64_t i = e / nc, c = e - i * nc;
  std_(X, planeX, e, ldd(A, m * n, (j0 + i) * n + c0 + c));
}

// A(j0:m, c0:n) <- X - P (double-double difference).
__global__ void __launch_bounds__(256) qr_update_kernel(int64_t m, int64_t n, int64_t j0, int64_t c0,
                                                        const double* __restrict__ X, const double* __restrict__ P,
                                                        double* __restrict__ A) {
  const int64_t mp = m - j0, nc = n - c0, planeX = mp * nc;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= planeX) return;
  const int64_t i = e / nc, c = e - i * nc;
  std_(A, m * n, (j0 + i) * n + c0 + c, dd_sub(ldd(X, planeX, e), ldd(P, planeX, e)));
}

inline unsigned blocks_for(int64_t count) { return static_cast<unsigned>((count + 255) / 256); }

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Workspace parts of the QR: V, Vt, G (V^T V), Tt, X (trailing block), W, W2, P,
// then the workspace of the largest mdgemm_ex call.
struct QrLayout {
  size_t v = 0, vt = 0, g = 0, tt = 0, x = 0, w = 0, w2 = 0, p = 0, pd = 0, prow = 0, pgram = 0, gemm = 0,
         gemm_bytes = 0, total = 0;
};

// The options of the trailing products: the adaptive digit width (fewer, wider
// digits whose level sums stay exact at the product's k), default cutoff.
mdgemm_opts qr_gemm_opts() {
  mdgemm_opts o;
  mdgemm_opts_init(&o);
  o.slice_bits = MDGEMM_SLICE_BITS_AUTO;
  return o;
}

// nf: the columns factored; n: all columns of A (the reflections are applied to
// columns nf .. n - 1 as well)
bool qr_layout(int64_t m, int64_t nf, int64_t n, int nb, QrLayout* L) {
  const size_t dd_bytes = 2 * sizeof(double);
  const size_t vbytes = align256(dd_bytes * static_cast<size_t>(m) * nb);
  const size_t xbytes = align256(dd_bytes * static_cast<size_t>(m) * static_cast<size_t>(n));
  const size_t wbytes = align256(dd_bytes * static_cast<size_t>(nb) * static_cast<size_t>(n));
  const size_t gbytes = align256(dd_bytes * nb * nb);
  size_t off = 0;
  L->v = off;
  off += vbytes;
  L->vt = off;
  off += vbytes;
  L->g = off;
  off += gbytes;
  L->tt = off;
  off += gbytes;
  L->x = off;
  off += xbytes;
  L->w = off;
  off += wbytes;
  L->w2 = off;
  off += wbytes;
  L->p = off;
  off += xbytes;
  // partial sums of the multi-workgroup panel, two buffers each: the dot
  // products [G][kMaxNb] and the pivot row [kMaxNb]
  const size_t groups = static_cast<size_t>((m + kPanelRowsSmall - 1) / kPanelRowsSmall);  // at most
  L->pd = off;
  off += align256(2 * dd_bytes * groups * kMaxNb);
  L->prow = off;
  off += align256(2 * dd_bytes * kMaxNb);
  L->pgram = off;
  off += align256(dd_bytes * static_cast<size_t>((m + kGramRows - 1) / kGramRows) * kMaxNb * kMaxNb);
  // the largest workspace of the three products of any panel: V^T X, T^T W, V W2
  mdgemm_opts o = qr_gemm_opts();
  size_t need = 0;
  for (int64_t j0 = 0; j0 < nf; j0 += nb) {
    const int64_t jb = std::min<int64_t>(nb, nf - j0), mp = m - j0, nc = n - j0 - jb;
    const size_t c[3] = {nc ? mdgemm_workspace_bytes(jb, nc, mp, 2, &o) : 0,
                         nc ? mdgemm_workspace_bytes(jb, nc, jb, 2, &o) : 0,
                         nc ? mdgemm_workspace_bytes(mp, nc, jb, 2, &o) : 0};
    for (size_t x : c) {
      if (x == SIZE_MAX) return false;
      need = std::max(need, x);
    }
  }
  L->gemm = off;
  L->gemm_bytes = std::max<size_t>(need, 256);
  off += align256(L->gemm_bytes);
  L->total = off;
  return true;
}

}  // namespace
}  // namespace mdg

extern "C" {

size_t mdgemm_qr_dd_workspace_bytes(int64_t m, int64_t n, int nb) {
  if (m < 1 || n < 1 || m < n || nb < 1 || nb > mdg::kMaxNb || m > (int64_t{1} << 20) || n > (int64_t{1} << 20))
    return SIZE_MAX;
  return mdg::qr_core_workspace(m, n, n, nb);
}

}  // extern "C"

namespace {

int qr_impl(int64_t m, int64_t n, int nb, double* A, double* tau, void* workspace, size_t workspace_bytes,
            void* stream) {
  if (m < 1 || n < 1 || m < n || nb < 1 || nb > mdg::kMaxNb || !A || !tau || !workspace) return MDGEMM_EINVAL;
  if (m > (int64_t{1} << 20) || n > (int64_t{1} << 20)) return MDGEMM_EINVAL;
  const size_t need = mdg::qr_core_workspace(m, n, n, nb);
  if (need == SIZE_MAX) return MDGEMM_EINVAL;
  if (workspace_bytes < need) return MDGEMM_EWORKSPACE;
  const uintptr_t w0 = reinterpret_cast<uintptr_t>(workspace), a0 = reinterpret_cast<uintptr_t>(A),
                  t0 = reinterpret_cast<uintptr_t>(tau);
  const uintptr_t abytes = sizeof(double) * 2 * static_cast<uintptr_t>(m) * n, tbytes = sizeof(double) * 2 * n;
  if ((w0 < a0 + abytes && a0 < w0 + need) || (w0 < t0 + tbytes && t0 < w0 + need) ||
      (a0 < t0 + tbytes && t0 < a0 + abytes))
    return MDGEMM_EINVAL;
  return mdg::qr_core(m, n, n, nb, A, tau, workspace, static_cast<hipStream_t>(stream));
}

}  // namespace

namespace mdg {

size_t qr_core_workspace(int64_t m, int64_t nf, int64_t n, int nb) {
  if (m < 1 || nf < 1 || nf > m || n < nf || nb < 1 || nb > kMaxNb) return SIZE_MAX;
  QrLayout L;
  return qr_layout(m, nf, n, nb, &L) ? L.total : SIZE_MAX;
}

int qr_core(int64_t m, int64_t nf, int64_t n, int nb, double* A, double* tau, void* workspace, hipStream_t s) {
  QrLayout L;
  if (!qr_layout(m, nf, n, nb, &L)) return MDGEMM_EINVAL;
  void* const stream = s;
  // the T kernel's dynamic LDS beyond 64 KB: allowed once for the kernel (a
  // failure shows up as a launch error below)
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&mdg::qr_t_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              static_cast<int>(mdg::kTLds));
    (void)hipGetLastError();
  });
  char* ws = static_cast<char*>(workspace);
  double* V = reinterpret_cast<double*>(ws + L.v);
  double* Vt = reinterpret_cast<double*>(ws + L.vt);
  double* G = reinterpret_cast<double*>(ws + L.g);
  double* Tt = reinterpret_cast<double*>(ws + L.tt);
  double* X = reinterpret_cast<double*>(ws + L.x);
  double* W = reinterpret_cast<double*>(ws + L.w);
  double* W2 = reinterpret_cast<double*>(ws + L.w2);
  double* P = reinterpret_cast<double*>(ws + L.p);
  double* pd = reinterpret_cast<double*>(ws + L.pd);
  double* prow = reinterpret_cast<double*>(ws + L.prow);
  double* pgram = reinterpret_cast<double*>(ws + L.pgram);
  mdgemm_opts o = mdg::qr_gemm_opts();
  o.stream = stream;
  o.workspace = ws + L.gemm;
  o.workspace_bytes = L.gemm_bytes;
  for (int64_t j0 = 0; j0 < nf; j0 += nb) {
    const int jb = static_cast<int>(std::min<int64_t>(nb, nf - j0));
    const int64_t mp = m - j0, c0 = j0 + jb, nc = n - c0;
    auto columns = [&](auto rows) {
      constexpr int kRows = decltype(rows)::value;
      const unsigned groups = static_cast<unsigned>((mp + kRows - 1) / kRows);
      for (int step = 0; step <= jb; ++step)
        hipLaunchKernelGGL(mdg::qr_col_step_kernel<kRows>, dim3(groups), dim3(mdg::kColThreads), 0, s, m, n, j0, jb,
                           step, A, tau, pd, prow);
    };
    if (mp > mdg::kShortPanel)
      columns(std::integral_constant<int, mdg::kPanelRowsTall>{});
    else if (mp > mdg::kSmallPanel)
      columns(std::integral_constant<int, mdg::kPanelRowsShort>{});
    else
      columns(std::integral_constant<int, mdg::kPanelRowsSmall>{});
    if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
    if (nc == 0) break;
    hipLaunchKernelGGL(mdg::qr_pack_v_kernel, dim3(mdg::blocks_for(mp * jb)), dim3(256), 0, s, m, n, j0, jb, A, V,
                       Vt);
    hipLaunchKernelGGL(mdg::qr_pack_block_kernel, dim3(mdg::blocks_for(mp * nc)), dim3(256), 0, s, m, n, j0, c0, A,
                       X);
    if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
    // G = V^T V (double-double dot products over the panel's rows)
    const unsigned ggroups = static_cast<unsigned>((mp + mdg::kGramRows - 1) / mdg::kGramRows);
    hipLaunchKernelGGL(mdg::qr_gram_partial_kernel, dim3(ggroups), dim3(mdg::kColThreads), 0, s, m, n, j0, jb, A,
                       pgram);
    hipLaunchKernelGGL(mdg::qr_gram_reduce_kernel, dim3(mdg::kMaxNb * mdg::kMaxNb / mdg::kGramThreads),
                       dim3(mdg::kGramThreads), 0, s, jb, static_cast<int64_t>(ggroups), pgram, G);
    if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
    int st = MDGEMM_OK;
    hipLaunchKernelGGL(mdg::qr_t_kernel, dim3(1), dim3(mdg::kTThreads), mdg::kTLds, s, jb, n, j0, G, tau, Tt);
    if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
    if ((st = mdgemm_ex(jb, nc, mp, 2, Vt, X, W, &o)) != MDGEMM_OK) return st;   // W = V^T X
    if ((st = mdgemm_ex(jb, nc, jb, 2, Tt, W, W2, &o)) != MDGEMM_OK) return st;  // W2 = T^T W
    if ((st = mdgemm_ex(mp, nc, jb, 2, V, W2, P, &o)) != MDGEMM_OK) return st;   // P = V W2
    hipLaunchKernelGGL(mdg::qr_update_kernel, dim3(mdg::blocks_for(mp * nc)), dim3(256), 0, s, m, n, j0, c0, X, P, A);
    if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
  }
  return MDGEMM_OK;
}

}  // namespace mdg

extern "C" {

int mdgemm_qr_dd(int64_t m, int64_t n, int nb, double* A, double* tau, void* workspace, size_t workspace_bytes,
                 void* stream) {
  // the products inside log at MDGEMM_LOG=2 only
  ++mdg::log_depth;
  const int st = qr_impl(m, n, nb, A, tau, workspace, workspace_bytes, stream);
  --mdg::log_depth;
  if (mdg::log_level() > mdg::log_depth)
    mdg::log_line("mdgemm_qr_dd m=%lld n=%lld nb=%d workspace=%zu stream=%p -> %s", static_cast<long long>(m),
                  static_cast<long long>(n), nb, workspace_bytes, stream, mdgemm_status_string(st));
  return st;
}

}  // extern "C"

// Taylor series of the solution of a linear system of power series in
// double-double: the application the paper names for its blocked Householder QR
// (section 5, future work), built on the QR and the multiple-double product of
// this library.
//
// A(t) = A_0 + A_1 t + ... + A_d t^d (n x n), B(t) = B_0 + ... + B_d t^d (n x r);
// X(t) = X_0 + ... + X_d t^d solves A(t) X(t) = B(t) modulo t^(d+1).  Comparing
// the coefficients of t^k:
//     A_0 X_k = B_k - sum_{i=1..k} A_i X_{k-i},   k = 0 .. d,
// a lower triangular block Toeplitz system with A_0 on its diagonal.
//
// The QR of A_0 is formed once, with its reflections applied to an identity
// block beside it, which leaves Q^T there; back substitution with R then turns
// Q^T into M = R^-1 Q^T = A_0^-1 (blocked: the block rows of R from the bottom,
// each block's coupling to the rows below it a product, its diagonal block a
// triangular solve).  Every degree is then two products on mdgemm_ex:
//     P_k = [A_k ... A_1] [X_0; ...; X_{k-1}],   X_k = M (B_k - P_k),
// so the whole series runs on the FP64 matrix cores.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "dd.h"
#include "internal.h"
#include "mdgemm.h"

namespace mdg {
namespace {

constexpr int kTaylorNb = 64;  // QR panels and back-substitution blocks
constexpr int64_t kTaylorMaxN = int64_t{1} << 15;
constexpr int kTaylorMaxDegree = 1024;

__device__ inline dd tl_load(const double* P, int64_t plane, int64_t idx) { return {P[idx], P[plane + idx]}; }
__device__ inline void tl_store(double* P, int64_t plane, int64_t idx, dd v) {
  P[idx] = v.hi;
  P[plane + idx] = v.lo;
}

// dst[i][j] = src[i][j] for an h x w block of double-doubles; each operand has
// its own limb-plane stride and row stride.
__global__ void __launch_bounds__(256) tl_copy_kernel(int64_t h, int64_t w, const double* __restrict__ src,
                                                      int64_t splane, int64_t sld, double* __restrict__ dst,
                                                      int64_t dplane, int64_t dld) {
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < h * w;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / w, j = e - i * w;
    tl_store(dst, dplane, i * dld + j, tl_load(src, splane, i * sld + j));
  }
}

// dst = a - b (double-double difference) for an h x w block; dst may be a
// (each element read and written by one thread).
__global__ void __launch_bounds__(256) tl_sub_kernel(int64_t h, int64_t w, const double* a, int64_t aplane,
                                                     int64_t ald, const double* __restrict__ b, int64_t bplane,
                                                     int64_t bld, double* dst, int64_t dplane, int64_t dld) {
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < h * w;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / w, j = e - i * w;
    tl_store(dst, dplane, i * dld + j, dd_sub(tl_load(a, aplane, i * ald + j), tl_load(b, bplane, i * bld + j)));
  }
}

// The n x n identity into a block of row stride ld.
__global__ void __launch_bounds__(256) tl_identity_kernel(int64_t n, double* __restrict__ dst, int64_t dplane,
                                                          int64_t dld) {
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < n * n;
       e += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t i = e / n, j = e - i * n;
    tl_store(dst, dplane, i * dld + j, dd{i == j ? 1.0 : 0.0, 0.0});
  }
}

// Y <- R^-1 Y for an upper triangular jb x jb block R (jb <= kTaylorNb = 64)
// and a jb x w block Y, in place: one wave per column of Y, lane l holding row
// l, kTrsmWaves columns per workgroup.  Right-looking back substitution: for
// i = jb - 1 down to 0, lane i forms x_i = y_i / R(i, i), which every lane
// takes by a shuffle, and the lanes l < i subtract R(l, i) x_i from their y_l.
// R is staged transposed in LDS (lanes read consecutive entries).
constexpr int kTrsmWaves = 4;
__global__ void __launch_bounds__(64 * kTrsmWaves) tl_trsm_kernel(int jb, int64_t w, const double* __restrict__ R,
                                                                  int64_t rplane, int64_t rld,
                                                                  double* __restrict__ Y, int64_t yplane,
                                                                  int64_t yld) {
  static_assert(kTaylorNb == 64, "one lane per row of the diagonal block");
  __shared__ dd rt[kTaylorNb][kTaylorNb];  // rt[i][l] = R(l, i) for l <= i, else 0
  for (int e = threadIdx.x; e < jb * jb; e += blockDim.x) {
    const int i = e / jb, l = e - i * jb;
    rt[i][l] = l <= i ? tl_load(R, rplane, l * rld + i) : dd{0.0, 0.0};
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * kTrsmWaves + (threadIdx.x >> 6);
  if (c >= w) return;
  dd y = lane < jb ? tl_load(Y, yplane, lane * yld + c) : dd{0.0, 0.0};
  for (int i = jb - 1; i >= 0; --i) {
    const dd q = dd_div(y, rt[i][i]);  // meaningful on lane i
    const dd x = {__shfl(q.hi, i, 64), __shfl(q.lo, i, 64)};
    if (lane == i) y = x;
    else if (lane < i) y = dd_sub(y, dd_mul(rt[i][lane], x));
  }
  if (lane < jb) tl_store(Y, yplane, lane * yld + c, y);
}

inline unsigned grid_for(int64_t count) {
  return static_cast<unsigned>(std::min<int64_t>((count + 255) / 256, 65535));
}
inline size_t up256(size_t x) { return (x + 255) / 256 * 256; }

mdgemm_opts taylor_gemm_opts() {
  mdgemm_opts o;
  mdgemm_opts_init(&o);
  o.slice_bits = MDGEMM_SLICE_BITS_AUTO;
  return o;
}

// Workspace: Aug [2][n][2n] ([A_0 | I], then R and the vectors | Q^T, then M) |
// tau [2][2n] | M [2][n][n] | Acat [2][n][d n] | Xcat [2][d n][r] | Rp [2][nb][n] |
// Mp [2][n][n] | Pb [2][nb][n] | Rhs [2][n][r] | Pk [2][n][r] | QR workspace |
// product workspace.
struct TaylorLayout {
  size_t aug = 0, tau = 0, m = 0, acat = 0, xcat = 0, rp = 0, mp = 0, pb = 0, rhs = 0, pk = 0, qr = 0, gemm = 0,
         gemm_bytes = 0, total = 0;
};

bool taylor_layout(int64_t n, int64_t r, int d, TaylorLayout* L) {
  const size_t e = 2 * sizeof(double), un = static_cast<size_t>(n), ur = static_cast<size_t>(r);
  const size_t ud = static_cast<size_t>(d);
  size_t off = 0;
  auto take = [&](size_t* at, size_t bytes) {
    *at = off;
    off += up256(std::max<size_t>(bytes, 1));
  };
  take(&L->aug, e * un * 2 * un);
  take(&L->tau, e * 2 * un);
  take(&L->m, e * un * un);
  take(&L->acat, e * un * ud * un);
  take(&L->xcat, e * ud * un * ur);
  take(&L->rp, e * kTaylorNb * un);
  take(&L->mp, e * un * un);
  take(&L->pb, e * kTaylorNb * un);
  take(&L->rhs, e * un * ur);
  take(&L->pk, e * un * ur);
  const size_t qr = qr_core_workspace(n, n, 2 * n, kTaylorNb);
  if (qr == SIZE_MAX) return false;
  take(&L->qr, qr);
  // the largest workspace of the products: the back substitution's couplings,
  // the right-hand sides' P_k and the degrees' M (B_k - P_k)
  mdgemm_opts o = taylor_gemm_opts();
  size_t need = mdgemm_workspace_bytes(n, r, n, 2, &o);
  for (int64_t j0 = 0; j0 < n; j0 += kTaylorNb) {
    const int64_t jb = std::min<int64_t>(kTaylorNb, n - j0), rest = n - j0 - jb;
    if (rest > 0) need = std::max(need, mdgemm_workspace_bytes(jb, n, rest, 2, &o));
  }
  for (int k = 1; k <= d; ++k) need = std::max(need, mdgemm_workspace_bytes(n, r, static_cast<int64_t>(k) * n, 2, &o));
  if (need == SIZE_MAX) return false;
  take(&L->gemm, need);
  L->gemm_bytes = need;
  L->total = off;
  return true;
}

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + bbytes && y < x + abytes;
}

int taylor_impl(int64_t n, int64_t r, int d, const double* A, const double* B, double* X, void* workspace,
                size_t workspace_bytes, void* stream) {
  if (n < 1 || r < 1 || d < 0 || n > kTaylorMaxN || r > (int64_t{1} << 20) || d > kTaylorMaxDegree || !A || !B ||
      !X || !workspace)
    return MDGEMM_EINVAL;
  TaylorLayout L;
  if (!taylor_layout(n, r, d, &L)) return MDGEMM_EINVAL;
  if (workspace_bytes < L.total) return MDGEMM_EWORKSPACE;
  const size_t nd = static_cast<size_t>(d) + 1;
  const size_t sa = sizeof(double) * 2 * nd * n * n, sb = sizeof(double) * 2 * nd * n * r;
  if (overlaps(workspace, L.total, A, sa) || overlaps(workspace, L.total, B, sb) ||
      overlaps(workspace, L.total, X, sb) || overlaps(X, sb, A, sa) || overlaps(X, sb, B, sb))
    return MDGEMM_EINVAL;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  double* Aug = reinterpret_cast<double*>(ws + L.aug);
  double* tau = reinterpret_cast<double*>(ws + L.tau);
  double* M = reinterpret_cast<double*>(ws + L.m);
  double* Acat = reinterpret_cast<double*>(ws + L.acat);
  double* Xcat = reinterpret_cast<double*>(ws + L.xcat);
  double* Rp = reinterpret_cast<double*>(ws + L.rp);
  double* Mp = reinterpret_cast<double*>(ws + L.mp);
  double* Pb = reinterpret_cast<double*>(ws + L.pb);
  double* Rhs = reinterpret_cast<double*>(ws + L.rhs);
  double* Pk = reinterpret_cast<double*>(ws + L.pk);
  mdgemm_opts o = taylor_gemm_opts();
  o.stream = stream;
  o.workspace = ws + L.gemm;
  o.workspace_bytes = L.gemm_bytes;
  const int64_t n2 = 2 * n, pa = n * n2, pn = n * n, pr = n * r;
  auto ok = [] { return hipGetLastError() == hipSuccess; };

  // [A_0 | I], then its QR: R and the vectors on the left, Q^T on the right
  hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(pn)), dim3(256), 0, s, n, n, A, pn, n, Aug, pa, n2);
  hipLaunchKernelGGL(tl_identity_kernel, dim3(grid_for(pn)), dim3(256), 0, s, n, Aug + n, pa, n2);
  if (!ok()) return MDGEMM_EHIP;
  int st = qr_core(n, n, n2, kTaylorNb, Aug, tau, ws + L.qr, s);
  if (st != MDGEMM_OK) return st;

  // M = R^-1 Q^T in place of Q^T, block rows from the bottom
  double* Y = Aug + n;
  const int64_t last = (n - 1) / kTaylorNb * kTaylorNb;
  for (int64_t j0 = last; j0 >= 0; j0 -= kTaylorNb) {
    const int jb = static_cast<int>(std::min<int64_t>(kTaylorNb, n - j0));
    const int64_t c0 = j0 + jb, rest = n - c0;
    if (rest > 0) {
      // Y(j0:c0, :) -= R(j0:c0, c0:n) M(c0:n, :)
      const int64_t prp = jb * rest, pmp = rest * n, ppb = jb * n;
      hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(prp)), dim3(256), 0, s, int64_t{jb}, rest, Aug + j0 * n2 + c0,
                         pa, n2, Rp, prp, rest);
      hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(pmp)), dim3(256), 0, s, rest, n, Y + c0 * n2, pa, n2, Mp, pmp,
                         n);
      if (!ok()) return MDGEMM_EHIP;
      if ((st = mdgemm_ex(jb, n, rest, 2, Rp, Mp, Pb, &o)) != MDGEMM_OK) return st;
      hipLaunchKernelGGL(tl_sub_kernel, dim3(grid_for(ppb)), dim3(256), 0, s, int64_t{jb}, n, Y + j0 * n2, pa, n2, Pb,
                         ppb, n, Y + j0 * n2, pa, n2);
    }
    hipLaunchKernelGGL(tl_trsm_kernel, dim3(static_cast<unsigned>((n + kTrsmWaves - 1) / kTrsmWaves)),
                       dim3(64 * kTrsmWaves), 0, s, jb, n, Aug + j0 * n2 + j0, pa, n2, Y + j0 * n2, pa, n2);
    if (!ok()) return MDGEMM_EHIP;
  }
  hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(pn)), dim3(256), 0, s, n, n, Y, pa, n2, M, pn, n);
  if (!ok()) return MDGEMM_EHIP;

  // the degrees: X_k = M (B_k - [A_k ... A_1] [X_0; ...; X_{k-1}])
  for (int k = 0; k <= d; ++k) {
    const double* Bk = B + static_cast<int64_t>(k) * 2 * pr;
    double* Xk = X + static_cast<int64_t>(k) * 2 * pr;
    const double* rhs = Bk;
    if (k > 0) {
      const int64_t kn = static_cast<int64_t>(k) * n, pac = n * kn, pxc = kn * r;
      for (int i = 1; i <= k; ++i)  // A_i to column block k - i
        hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(pn)), dim3(256), 0, s, n, n,
                           A + static_cast<int64_t>(i) * 2 * pn, pn, n, Acat + static_cast<int64_t>(k - i) * n, pac,
                           kn);
      for (int j = 0; j < k; ++j)  // X_j to row block j
        hipLaunchKernelGGL(tl_copy_kernel, dim3(grid_for(pr)), dim3(256), 0, s, n, r,
                           X + static_cast<int64_t>(j) * 2 * pr, pr, r, Xcat + static_cast<int64_t>(j) * n * r, pxc,
                           r);
      if (!ok()) return MDGEMM_EHIP;
      if ((st = mdgemm_ex(n, r, kn, 2, Acat, Xcat, Pk, &o)) != MDGEMM_OK) return st;
      hipLaunchKernelGGL(tl_sub_kernel, dim3(grid_for(pr)), dim3(256), 0, s, n, r, Bk, pr, r, Pk, pr, r, Rhs, pr, r);
      if (!ok()) return MDGEMM_EHIP;
      rhs = Rhs;
    }
    if ((st = mdgemm_ex(n, r, n, 2, M, rhs, Xk, &o)) != MDGEMM_OK) return st;
  }
  return MDGEMM_OK;
}

}  // namespace
}  // namespace mdg

extern "C" {

size_t mdgemm_taylor_dd_workspace_bytes(int64_t n, int64_t r, int d) {
  if (n < 1 || r < 1 || d < 0 || n > mdg::kTaylorMaxN || r > (int64_t{1} << 20) || d > mdg::kTaylorMaxDegree)
    return SIZE_MAX;
  mdg::TaylorLayout L;
  return mdg::taylor_layout(n, r, d, &L) ? L.total : SIZE_MAX;
}

int mdgemm_taylor_dd(int64_t n, int64_t r, int d, const double* A, const double* B, double* X, void* workspace,
                     size_t workspace_bytes, void* stream) {
  ++mdg::log_depth;
  const int st = mdg::taylor_impl(n, r, d, A, B, X, workspace, workspace_bytes, stream);
  --mdg::log_depth;
  if (mdg::log_level() > mdg::log_depth)
    mdg::log_line("mdgemm_taylor_dd n=%lld r=%lld d=%d workspace=%zu stream=%p -> %s", static_cast<long long>(n),
                  static_cast<long long>(r), d, workspace_bytes, stream, mdgemm_status_string(st));
  return st;
}

}  // extern "C"

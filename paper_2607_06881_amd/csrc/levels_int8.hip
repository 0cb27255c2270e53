// Step a3 on the int8 matrix cores (the MDGEMM_INT8 option): the level
// products from the int8 digits, by the hand-written kernel of
// level_gemm_i8.hip or by hipBLASLt, whichever is faster for the shape.
//
// The level products of section 2 are exact integer sums, so any matrix unit
// that sums integer products exactly computes them.  With digits of at most 7
// bits (|d| <= 127) a product is below 2^14 and a level sum of pairs x k
// products stays below 2^31 when pairs k 127^2 < 2^31 (checked by the caller),
// so the int8 x int8 -> int32 matrix cores (5 POP/s on MI355X, 64 times the
// FP64 rate) form every level exactly.  Both routes give bit-identical planes.
//
// Layout (internal.h): rows of pitch ld = kI8Pad + S kp, A's digit p of row i at
// bytes kI8Pad + p kp .., B's digit q of column j at kI8Pad + (S-1-q) kp ...  The
// pairs (p, t - p), p = p0 .. p1, of level t are then the contiguous k range of
// length K = (p1 - p0 + 1) kp starting at p0 kp in every row of A's digits and
// at (S-1-t+p0) kp in every row of B's.  For hipBLASLt a level is one plain
// GEMM with both operands k-contiguous (column-major, the first one transposed):
//     G_t^T (n x m, ld n) = op_T(DBt + kI8Pad + (S-1-t+p0) kp: K x n, ld) . (DA + kI8Pad + p0 kp: K x m, ld)
// and G_t^T in column-major is the row-major plane G_t [m][n] that the
// accumulation reads.
//
// The route is chosen per shape (m, n, kp, S, T) on its first call: the
// hand-written kernel (all levels in one launch) and hipBLASLt's levels (each
// with the fastest of up to 32 hipBLASLt candidates, timed on that call) are
// timed (best of two runs each) on the call's stream, and the faster is kept
// for the process (the hand-written kernel unless hipBLASLt is more than 3%
// faster).  The environment variable MDGEMM_INT8_LEVELS = mfma | hipblaslt
// forces one route.  The hipBLASLt handle, the operation descriptor and the
// algorithms are created once per device and kept.  mdgemm_ex refuses int8 calls
// under graph capture; a capturing stream here would get the hand-written
// kernel (or hipBLASLt's first candidate), untimed.
#include <hipblaslt/hipblaslt.h>

#include <array>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <vector>

#include "internal.h"

namespace mdg {
namespace {

struct Blt {
  hipblasLtHandle_t handle = nullptr;
  hipblasLtMatmulDesc_t desc = nullptr;
  hipblasLtMatmulPreference_t pref = nullptr;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;  // for timing the candidates
  std::map<std::array<int64_t, 5>, hipblasLtMatmulAlgo_t> algos;  // (M, N, K, lda, ldb)
  std::map<std::array<int64_t, 5>, bool> own;                       // (m, n, kp, S, T): the hand-written kernel?
};

enum class Route { kAuto, kOwn, kBlas };
// read on every call, so that a process may switch routes
Route forced_route() {
  const char* e = std::getenv("MDGEMM_INT8_LEVELS");
  if (e && std::strcmp(e, "mfma") == 0) return Route::kOwn;
  if (e && std::strcmp(e, "hipblaslt") == 0) return Route::kBlas;
  return Route::kAuto;
}

struct BltState {
  std::mutex mu;
  std::vector<Blt*> dev;  // per device, created on first use and kept until the process ends
};

BltState& blt_state() {
  static BltState s;
  return s;
}

// The hipBLASLt objects of the current device (with blt_state().mu held).
Blt* blt_for_device() {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess) return nullptr;
  BltState& s = blt_state();
  if (static_cast<size_t>(d) >= s.dev.size()) s.dev.resize(d + 1, nullptr);
  if (s.dev[d]) return s.dev[d];
  Blt* b = new Blt;
  bool ok = hipblasLtCreate(&b->handle) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatmulDescCreate(&b->desc, HIPBLAS_COMPUTE_32I, HIP_R_32I) == HIPBLAS_STATUS_SUCCESS &&
            hipblasLtMatmulPreferenceCreate(&b->pref) == HIPBLAS_STATUS_SUCCESS &&
            hipEventCreate(&b->ev0) == hipSuccess && hipEventCreate(&b->ev1) == hipSuccess;
  if (ok) {
    const hipblasOperation_t opa = HIPBLAS_OP_T, opb = HIPBLAS_OP_N;
    const uint64_t ws = 0;  // no hipBLASLt workspace (split-k forms with one measured no faster)
    ok = hipblasLtMatmulDescSetAttribute(b->desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opa, sizeof opa) ==
             HIPBLAS_STATUS_SUCCESS &&
         hipblasLtMatmulDescSetAttribute(b->desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opb, sizeof opb) ==
             HIPBLAS_STATUS_SUCCESS &&
         hipblasLtMatmulPreferenceSetAttribute(b->pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof ws) ==
             HIPBLAS_STATUS_SUCCESS;
  }
  if (!ok) {
    if (b->ev0) (void)hipEventDestroy(b->ev0);
    if (b->ev1) (void)hipEventDestroy(b->ev1);
    if (b->pref) hipblasLtMatmulPreferenceDestroy(b->pref);
    if (b->desc) hipblasLtMatmulDescDestroy(b->desc);
    if (b->handle) hipblasLtDestroy(b->handle);
    delete b;
    return nullptr;
  }
  s.dev[d] = b;
  return b;
}

struct Layouts {
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, d = nullptr;
  ~Layouts() {
    if (a) hipblasLtMatrixLayoutDestroy(a);
    if (b) hipblasLtMatrixLayoutDestroy(b);
    if (d) hipblasLtMatrixLayoutDestroy(d);
  }
};

}  // namespace

namespace {

// One hipBLASLt GEMM per level (with blt_state().mu held).
hipError_t run_blas(Blt* b, int64_t m, int64_t n, int64_t kp, int S, int T, const int8_t* DA, const int8_t* DBt,
                    int32_t* G, hipStream_t stream) {
  const int32_t alpha = 1, beta = 0;
  for (int t = 0; t <= T; ++t) {
    const int p0 = t - (S - 1) > 0 ? t - (S - 1) : 0, p1 = t < S - 1 ? t : S - 1;
    const int64_t K = static_cast<int64_t>(p1 - p0 + 1) * kp;
    const int64_t ld = kI8Pad + static_cast<int64_t>(S) * kp;
    const int8_t* mat1 = DBt + kI8Pad + static_cast<int64_t>(S - 1 - t + p0) * kp;  // K x n, ld (used transposed)
    const int8_t* mat2 = DA + kI8Pad + static_cast<int64_t>(p0) * kp;               // K x m, ld
    int32_t* out = G + static_cast<int64_t>(t) * m * n;                              // n x m, ld n
    Layouts l;
    if (hipblasLtMatrixLayoutCreate(&l.a, HIP_R_8I, K, n, ld) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&l.b, HIP_R_8I, K, m, ld) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&l.d, HIP_R_32I, n, m, n) != HIPBLAS_STATUS_SUCCESS)
      return hipErrorInvalidValue;
    const std::array<int64_t, 5> key{n, m, K, ld, ld};
    auto it = b->algos.find(key);
    if (it == b->algos.end()) {
      constexpr int kCandidates = 32;
      hipblasLtMatmulHeuristicResult_t res[kCandidates];
      int nres = 0;
      if (hipblasLtMatmulAlgoGetHeuristic(b->handle, b->desc, l.a, l.b, l.d, l.d, b->pref, kCandidates, res,
                                          &nres) != HIPBLAS_STATUS_SUCCESS ||
          nres < 1)
        return hipErrorNotSupported;
      int best = 0;
      hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
      if (hipStreamIsCapturing(stream, &cap) != hipSuccess) return hipErrorUnknown;
      if (nres > 1 && cap == hipStreamCaptureStatusNone) {
        float best_ms = 0.0f;
        bool timed = false;
        for (int a = 0; a < nres; ++a) {
          auto run = [&]() {
            return hipblasLtMatmul(b->handle, b->desc, &alpha, mat1, l.a, mat2, l.b, &beta, out, l.d, out, l.d,
                                   &res[a].algo, nullptr, 0, stream) == HIPBLAS_STATUS_SUCCESS;
          };
          if (!run()) continue;  // warm-up; a candidate that fails is skipped
          if (hipEventRecord(b->ev0, stream) != hipSuccess || !run() || !run() ||
              hipEventRecord(b->ev1, stream) != hipSuccess || hipEventSynchronize(b->ev1) != hipSuccess)
            return hipErrorUnknown;
          float ms = 0.0f;
          if (hipEventElapsedTime(&ms, b->ev0, b->ev1) != hipSuccess) return hipErrorUnknown;
          if (!timed || ms < best_ms) {
            best_ms = ms;
            best = a;
            timed = true;
          }
        }
        if (!timed) return hipErrorLaunchFailure;
      }
      it = b->algos.emplace(key, res[best].algo).first;
    }
    if (hipblasLtMatmul(b->handle, b->desc, &alpha, mat1, l.a, mat2, l.b, &beta, out, l.d, out, l.d, &it->second,
                        nullptr, 0, stream) != HIPBLAS_STATUS_SUCCESS)
      return hipErrorLaunchFailure;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_levels_int8(int64_t m, int64_t n, int64_t kp, int S, int T, const int8_t* DA, const int8_t* DBt,
                              int32_t* G, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  if (S < 1 || T < 0 || T > 2 * S - 2 || kp <= 0 || kp % kI8Pad != 0) return hipErrorInvalidValue;
  const Route forced = forced_route();
  const bool fits = level_gemm_i8_fits(kp, S);
  if (forced == Route::kOwn && !fits) return hipErrorInvalidValue;
  if (forced == Route::kOwn) return launch_level_gemm_i8(m, n, kp, S, T, DA, DBt, G, stream);
  std::lock_guard<std::mutex> lock(blt_state().mu);
  Blt* b = blt_for_device();
  if (!b) return hipErrorNotInitialized;
  if (forced == Route::kBlas || !fits) return run_blas(b, m, n, kp, S, T, DA, DBt, G, stream);
  const std::array<int64_t, 5> key{m, n, kp, S, T};
  auto it = b->own.find(key);
  if (it != b->own.end())
    return it->second ? launch_level_gemm_i8(m, n, kp, S, T, DA, DBt, G, stream)
                      : run_blas(b, m, n, kp, S, T, DA, DBt, G, stream);
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cap) != hipSuccess) return hipErrorUnknown;
  if (cap != hipStreamCaptureStatusNone) return launch_level_gemm_i8(m, n, kp, S, T, DA, DBt, G, stream);
  // first call of the shape: time both routes (after one untimed run each, which
  // for hipBLASLt also picks its algorithms), keep the faster; both write the
  // same planes, so G holds the result whichever runs last
  float t_own = 0.0f, t_blas = 0.0f;
  // one untimed run, then the better of two timed ones
  auto timed = [&](auto&& fn, float* ms) -> hipError_t {
    hipError_t e = fn();
    if (e != hipSuccess) return e;
    for (int rep = 0; rep < 2; ++rep) {
      if (hipEventRecord(b->ev0, stream) != hipSuccess) return hipErrorUnknown;
      if ((e = fn()) != hipSuccess) return e;
      float t = 0.0f;
      if (hipEventRecord(b->ev1, stream) != hipSuccess || hipEventSynchronize(b->ev1) != hipSuccess ||
          hipEventElapsedTime(&t, b->ev0, b->ev1) != hipSuccess)
        return hipErrorUnknown;
      if (rep == 0 || t < *ms) *ms = t;
    }
    return hipSuccess;
  };
  hipError_t e = timed([&] { return launch_level_gemm_i8(m, n, kp, S, T, DA, DBt, G, stream); }, &t_own);
  if (e != hipSuccess) return e;
  e = timed([&] { return run_blas(b, m, n, kp, S, T, DA, DBt, G, stream); }, &t_blas);
  if (e != hipSuccess) {
    // hipBLASLt has no algorithm for a level shape (or one failed to launch):
    // keep the hand-written kernel, and recompute the planes with it
    (void)hipGetLastError();
    b->own.emplace(key, true);
    return launch_level_gemm_i8(m, n, kp, S, T, DA, DBt, G, stream);
  }
  b->own.emplace(key, t_own <= 1.03f * t_blas);  // ties (within 3%) go to the hand-written kernel
  return hipSuccess;
}

}  // namespace mdg

// Step a3 on the int8 matrix cores (the MDGEMM_INT8 option).
//
// The level products of section 2 are exact integer sums, so any matrix unit
// that sums integer products exactly computes them.  With digits of at most 7
// bits (|d| <= 127) a product is below 2^14 and a level sum of pairs x k
// products stays below 2^31 when pairs k 127^2 < 2^31 (checked by the caller),
// so the int8 x int8 -> int32 matrix cores (5 POP/s on MI355X, 64 times the
// FP64 rate) form every level exactly.
//
// Layouts: A's digits D_A [m][S][kp] (launch_split_int8), B's digits D_Bt
// [np][S kp] with digit q of column j at k range (S-1-q) kp .. (reverse order;
// launch_split_int8t).  The pairs (p, t - p) of level t, p = p0 .. p1, are then
// the contiguous k range of length K = (p1 - p0 + 1) kp starting at p0 kp in
// every row of D_A and at (S-1-t+p0) kp in every column of D_Bt, so a level is
// one plain GEMM with both operands k-contiguous (column-major, the first one
// transposed):
//     G_t^T (n x m, ld n) = op_T(D_Bt + (S-1-t+p0) kp: K x n, ld S kp) . (D_A + p0 kp: K x m, ld S kp)
// G_t^T in column-major is the row-major plane G_t [m][n] that the
// accumulation reads.  (With both operands k-contiguous hipBLASLt's int8 GEMMs
// ran at 2.2-2.8 POP/s on MI355X at these shapes, against 1.8-2.4 with B's
// digits n-contiguous.)
//
// The hipBLASLt handle, the operation descriptor and the algorithm per shape
// are created once per device and kept.  The algorithm of a shape is chosen on
// its first call: hipBLASLt's candidates (up to 32) are each timed on the call's
// stream (two runs into the level's own output plane, which the chosen one then
// overwrites) and the fastest is kept.  mdgemm_ex refuses int8 calls under graph
// capture; a capturing stream here would get the first candidate, untimed.
#include <hipblaslt/hipblaslt.h>

#include <array>
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
};

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

hipError_t launch_levels_int8(int64_t m, int64_t n, int64_t kp, int64_t np, int S, int T, const int8_t* DA,
                              const int8_t* DBt, int32_t* G, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  if (S < 1 || T < 0 || T > 2 * S - 2 || kp <= 0 || np < n) return hipErrorInvalidValue;
  std::lock_guard<std::mutex> lock(blt_state().mu);
  Blt* b = blt_for_device();
  if (!b) return hipErrorNotInitialized;
  const int32_t alpha = 1, beta = 0;
  for (int t = 0; t <= T; ++t) {
    const int p0 = t - (S - 1) > 0 ? t - (S - 1) : 0, p1 = t < S - 1 ? t : S - 1;
    const int64_t K = static_cast<int64_t>(p1 - p0 + 1) * kp;
    const int64_t ld = static_cast<int64_t>(S) * kp;
    const int8_t* mat1 = DBt + static_cast<int64_t>(S - 1 - t + p0) * kp;  // K x n, ld S kp (used transposed)
    const int8_t* mat2 = DA + static_cast<int64_t>(p0) * kp;               // K x m, ld S kp
    int32_t* out = G + static_cast<int64_t>(t) * m * n;                    // n x m, ld n
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

}  // namespace mdg

// Step a3 -- level GEMMs of the slice digits on the FP64 matrix cores.
//
// Section 2 (equation (3) and the rewritten product) multiplies the quarters
// pairwise and collects the products whose indices add up to the same level
// t = p + q.  Every digit is an integer with |d| <= 8191, every product is below
// 2^26, and every partial sum stays below 2^53 (the analogue of the bound
// (NBound) of section 2, checked on the host), so each level
//     G_t = sum over p + q = t of DA_p . DB_q
// is computed exactly by FP64 multiply-adds in any order and any blocking.
//
// The paper materializes Abar = [A_0 .. A_7] and a block-Toeplitz Bbar and runs
// one big FP64 GEMM.  Here nothing is materialized: one workgroup owns a
// 128 x 128 tile of one output plane and walks the K dimension of every pair of
// its level in turn, reading the digit planes in place.
//
// CDNA4 mapping: v_mfma_f64_16x16x4f64 (A 16x4, B 4x16, C/D 16x16 in FP64; lane
// l supplies A[l%16][l/16] and B[l/16][l%16]; register r of lane l holds
// D[4r + l/16][l%16]).  One instruction occupies the matrix pipe of a SIMD for
// 64 cycles, so four waves, one per SIMD, each with a 64 x 64 sub-tile (16
// independent accumulators) keep the pipes busy.  A and B tiles of 16 k-values
// are staged through LDS with double buffering: the global loads of step it+1
// are issued before the 64 MFMAs of step it and stored to the other buffer
// after them, one barrier per step.  LDS rows are padded (A: 17 doubles, B: 144)
// so that the fragment reads of a half-wave hit distinct banks.
//
// Work decomposition: grid.x = output tiles, grid.y = jobs (levels, heaviest
// first, or single pairs).  Tiles are renumbered so that each of the 8 XCDs
// (blocks are dealt to XCDs round-robin) works on a contiguous band of tiles
// that share rows of DA, which keeps those rows in that XCD's L2.
#include "internal.h"

namespace mdg {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 16;
constexpr int LDA = BK + 1;   // A tile in LDS: [BM][LDA]
constexpr int LDB = BN + 16;  // B tile in LDS: [BK][LDB]
constexpr int kThreads = 256;
constexpr int kALoads = BM * BK / kThreads;  // 8 doubles per thread
constexpr int kBLoads = BK * BN / kThreads;  // 8 doubles per thread
constexpr int kXcds = 8;

__global__ void __launch_bounds__(kThreads, 2) slice_gemm_kernel(int64_t m, int64_t n, int64_t k, int tiles_n,
                                                                 int ntiles, const double* __restrict__ DA,
                                                                 const double* __restrict__ DB,
                                                                 double* __restrict__ out, const JobTable jobs) {
  __shared__ double As[2][BM * LDA];
  __shared__ double Bs[2][BK * LDB];

  // XCD-aware renumbering: block b runs on XCD b % 8; give XCD x the tiles
  // [x * per, (x+1) * per) in row-major tile order.
  int tile = blockIdx.x;
  {
    const int per = ntiles / kXcds;
    if (tile < per * kXcds) tile = (tile % kXcds) * per + tile / kXcds;
  }
  const int64_t m0 = static_cast<int64_t>(tile / tiles_n) * BM;
  const int64_t n0 = static_cast<int64_t>(tile % tiles_n) * BN;
  const int job = blockIdx.y;
  const int p_first = jobs.p_first[job], q_first = jobs.q_first[job], npairs = jobs.npairs[job];
  const int64_t plane_a = m * k, plane_b = k * n;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;  // 2 x 2 waves, 64 x 64 each

  const int64_t nkb = (k + BK - 1) / BK;
  const int64_t niter = nkb * npairs;

  d4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};

  double ra[kALoads], rb[kBLoads];

  // Global -> registers for step (pair index pi, k-block kb); zero outside the matrices.
  auto load_tiles = [&](int pi, int64_t kb) {
    const double* a = DA + static_cast<int64_t>(p_first + pi) * plane_a;
    const double* b = DB + static_cast<int64_t>(q_first - pi) * plane_b;
    const int64_t k0 = kb * BK;
#pragma unroll
    for (int r = 0; r < kALoads; ++r) {
      const int idx = r * kThreads + tid;
      const int64_t gi = m0 + (idx >> 4), gk = k0 + (idx & 15);
      ra[r] = (gi < m && gk < k) ? a[gi * k + gk] : 0.0;
    }
#pragma unroll
    for (int r = 0; r < kBLoads; ++r) {
      const int idx = r * kThreads + tid;
      const int64_t gk = k0 + (idx >> 7), gj = n0 + (idx & 127);
      rb[r] = (gk < k && gj < n) ? b[gk * n + gj] : 0.0;
    }
  };
  auto store_tiles = [&](int buf) {
#pragma unroll
    for (int r = 0; r < kALoads; ++r) {
      const int idx = r * kThreads + tid;
      As[buf][(idx >> 4) * LDA + (idx & 15)] = ra[r];
    }
#pragma unroll
    for (int r = 0; r < kBLoads; ++r) {
      const int idx = r * kThreads + tid;
      Bs[buf][(idx >> 7) * LDB + (idx & 127)] = rb[r];
    }
  };

  int pi = 0;
  int64_t kb = 0;
  if (niter > 0) {
    load_tiles(0, 0);
    store_tiles(0);
  }
  __syncthreads();

  const int frag_row = lane & 15, frag_k = lane >> 4;
  for (int64_t it = 0; it < niter; ++it) {
    const int cur = static_cast<int>(it & 1);
    const bool more = it + 1 < niter;
    if (more) {
      if (++kb == nkb) {
        kb = 0;
        ++pi;
      }
      load_tiles(pi, kb);
    }
    const double* as = As[cur] + (wr * 64 + frag_row) * LDA + frag_k;
    const double* bs = Bs[cur] + frag_k * LDB + wc * 64 + frag_row;
#pragma unroll
    for (int kg = 0; kg < BK / 4; ++kg) {
      double af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = as[i * 16 * LDA + kg * 4];
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = bs[kg * 4 * LDB + j * 16];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_tiles(cur ^ 1);
    __syncthreads();
  }

  double* o = out + static_cast<int64_t>(jobs.out[job]) * m * n;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = m0 + wr * 64 + i * 16 + 4 * r + (lane >> 4);
        const int64_t gj = n0 + wc * 64 + j * 16 + (lane & 15);
        if (gi < m && gj < n) o[gi * n + gj] = acc[i][j][r];
      }
}

}  // namespace

hipError_t launch_slice_gemm(int64_t m, int64_t n, int64_t k, const double* DA, const double* DB, double* out,
                             const JobTable& jobs, hipStream_t stream) {
  if (m == 0 || n == 0 || jobs.njobs == 0) return hipSuccess;
  const int64_t tiles_m = (m + BM - 1) / BM, tiles_n = (n + BN - 1) / BN;
  const int64_t ntiles = tiles_m * tiles_n;
  if (ntiles > 0x7fffffff || jobs.njobs > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(slice_gemm_kernel, dim3(static_cast<unsigned>(ntiles), static_cast<unsigned>(jobs.njobs)),
                     dim3(kThreads), 0, stream, m, n, k, static_cast<int>(tiles_n), static_cast<int>(ntiles), DA, DB,
                     out, jobs);
  return hipGetLastError();
}

}  // namespace mdg

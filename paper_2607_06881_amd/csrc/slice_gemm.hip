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
// its level in turn, reading the digit panels in place.
//
// Operand layout ("panels", written by the split): both operands k-major and
// padded with zeros to whole tiles,
//     DAt [S][kp][mp]  (DAt[p][kk][i] = digit p of A[i][kk]),
//     DBp [S][kp][np]  (DBp[q][kk][j] = digit q of B[kk][j]),
// kp = k rounded up to 16, mp / np = m / n rounded up to 128.  A 16 x 128 slice
// of a panel is 16 rows of 1 KB, so the loads need no bounds checks.
//
// CDNA4 mapping:
// * v_mfma_f64_16x16x4f64 (A 16x4, B 4x16, C/D 16x16 in FP64; lane l supplies
//   A[l%16][l/16] and B[l/16][l%16]; register r of lane l holds
//   D[4r + l/16][l%16]).  One instruction occupies a SIMD's matrix pipe for 64
//   cycles; four waves (one per SIMD), each with a 64 x 64 sub-tile held in 16
//   independent accumulators, keep the pipes busy.
// * Tiles go global -> LDS directly with global_load_lds_dwordx4 (64 lanes x
//   16 bytes = one 1 KB panel row per wave instruction; no staging registers).
//   Two LDS stages, one barrier per step.  Within a step a wave first reads
//   all its fragments of the current stage (32 doubles), then issues the
//   copies of the next step into the other stage, then runs its 64 MFMAs:
//   since no LDS read follows a copy in flight, nothing waits for the copies
//   until the next step's barrier, and they land while the MFMAs run.
// * LDS rows are padded to 144 doubles so that the two 16-lane halves of a
//   fragment read (consecutive k rows) fall on different banks.
//
// Work decomposition: grid.x = output tiles, grid.y = jobs (levels, heaviest
// first, or single pairs).  Tiles are renumbered so that each of the 8 XCDs
// (blocks are dealt to XCDs round-robin) works on its own chunk of tiles, and
// the blocks resident on one XCD at a time cover an about 8 x 8 patch whose
// panel rows stay in that XCD's L2.
#include "internal.h"

namespace mdg {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int BM = kTileMN, BN = kTileMN, BK = kTileK;
constexpr int LDS_LD = BM + 16;  // doubles per LDS row
constexpr int kThreads = 256;
constexpr int kXcds = 8;
constexpr int kGroup = 8;  // tile-rows per group of the tile order
constexpr unsigned kWaitVmcnt0 = 0x0F70;  // s_waitcnt vmcnt(0)

static_assert(BM == 128 && BN == 128 && BK == 16, "the load mapping assumes 128 x 128 x 16 tiles and 4 waves");

__global__ void __launch_bounds__(kThreads, 2) slice_gemm_kernel(int64_t m, int64_t n, int64_t kp, int64_t mp,
                                                                 int64_t np, int tiles_n, int ntiles,
                                                                 const double* __restrict__ DAt,
                                                                 const double* __restrict__ DBp,
                                                                 double* __restrict__ out, const JobTable jobs) {
  __shared__ double As[2][BK * LDS_LD];
  __shared__ double Bs[2][BK * LDS_LD];

  // Tile order.  Block b runs on XCD b % 8 (round-robin dispatch); XCD x takes
  // the chunk [x * per, (x+1) * per) of an order that walks groups of kGroup
  // tile-rows column by column, so the ~64 blocks resident on one XCD at a time
  // form a near-square patch of tiles and share their panel rows in its L2.
  int t = blockIdx.x;
  {
    const int per = ntiles / kXcds;
    if (t < per * kXcds) t = (t % kXcds) * per + t / kXcds;
  }
  const int tiles_m = ntiles / tiles_n;
  const int gsz = kGroup * tiles_n, g = t / gsz, first = g * kGroup;
  const int rows_in = min(kGroup, tiles_m - first), within = t - g * gsz;
  const int64_t m0 = static_cast<int64_t>(first + within % rows_in) * BM;
  const int64_t n0 = static_cast<int64_t>(within / rows_in) * BN;
  const int job = blockIdx.y;
  const int p_first = jobs.p_first[job], q_first = jobs.q_first[job], npairs = jobs.npairs[job];
  const int64_t plane_a = kp * mp, plane_b = kp * np;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;  // 2 x 2 waves, 64 x 64 each

  const int64_t nkb = kp / BK;
  const int64_t niter = nkb * npairs;

  // Direct global -> LDS copies (global_load_lds_dwordx4, 1 KB panel row per wave
  // instruction); wave w copies rows 4w .. 4w+3 of the A and of the B tile.
  const int lane_off = 2 * lane;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  int lpi = 0;
  int64_t lkb = 0;  // the step the next copy fetches
  auto issue = [&](int stage) {
    const double* a = DAt + static_cast<int64_t>(p_first + lpi) * plane_a + (lkb * BK + 4 * wave_u) * mp + m0;
    const double* b = DBp + static_cast<int64_t>(q_first - lpi) * plane_b + (lkb * BK + 4 * wave_u) * np + n0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(a + r * mp + lane_off),
                                       (lds_void*)(&As[stage][(4 * wave_u + r) * LDS_LD]),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(b + r * np + lane_off),
                                       (lds_void*)(&Bs[stage][(4 * wave_u + r) * LDS_LD]),
                                       16, 0, 0);
    }
    if (++lkb == nkb) {
      lkb = 0;
      ++lpi;
    }
  };

  d4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};

  const int frag_col = lane & 15, frag_k = lane >> 4;
  if (niter > 0) issue(0);
  for (int64_t it = 0; it < niter; ++it) {
    const int cur = static_cast<int>(it & 1);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // this wave's copies of step it are in LDS
    __syncthreads();                     // everyone's are; everyone is done reading the other stage
    // all fragments of this step first, then the copies for the next step, then
    // the MFMAs: no LDS read follows a copy in flight, so nothing waits for it.
    const double* as = As[cur] + frag_k * LDS_LD + wr * 64 + frag_col;
    const double* bs = Bs[cur] + frag_k * LDS_LD + wc * 64 + frag_col;
    double af[4][4], bf[4][4];
#pragma unroll
    for (int kg = 0; kg < BK / 4; ++kg)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        af[kg][i] = as[kg * 4 * LDS_LD + i * 16];
        bf[kg][i] = bs[kg * 4 * LDS_LD + i * 16];
      }
    if (it + 1 < niter) issue(cur ^ 1);
#pragma unroll
    for (int kg = 0; kg < BK / 4; ++kg)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[kg][i], bf[kg][j], acc[i][j], 0, 0, 0);
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

hipError_t launch_slice_gemm(int64_t m, int64_t n, int64_t k, const double* DAt, const double* DBp, double* out,
                             const JobTable& jobs, hipStream_t stream) {
  if (m == 0 || n == 0 || jobs.njobs == 0) return hipSuccess;
  const int64_t mp = panel_mn(m), np = panel_mn(n), kp = panel_k(k);
  const int64_t tiles_n = np / BN;
  const int64_t ntiles = (mp / BM) * tiles_n;
  if (ntiles > 0x7fffffff || jobs.njobs > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(slice_gemm_kernel, dim3(static_cast<unsigned>(ntiles), static_cast<unsigned>(jobs.njobs)),
                     dim3(kThreads), 0, stream, m, n, kp, mp, np, static_cast<int>(tiles_n),
                     static_cast<int>(ntiles), DAt, DBp, out, jobs);
  return hipGetLastError();
}

}  // namespace mdg

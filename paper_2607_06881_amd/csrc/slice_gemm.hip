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
// * Tiles go global -> registers -> LDS in 16-byte pieces (a wave reads one
//   1 KB panel row per instruction).  Two LDS stages: the global loads of step
//   it+1 are issued before the 64 MFMAs of step it and written to the other
//   stage after them; one barrier per step.
// * LDS rows are padded to 144 doubles so that the two 16-lane halves of a
//   fragment read (consecutive k rows) fall on different banks.
// * Fragments of the next k-group are read from LDS while the current group's
//   MFMAs run (two register buffers).
//
// Work decomposition: grid.x = output tiles, grid.y = jobs (levels, heaviest
// first, or single pairs).  Tiles are renumbered so that each of the 8 XCDs
// (blocks are dealt to XCDs round-robin) works on a contiguous band of tiles
// that share rows of DAt, which keeps them in that XCD's L2.
#include "internal.h"

namespace mdg {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int BM = kTileMN, BN = kTileMN, BK = kTileK;
constexpr int LDS_LD = BM + 16;  // doubles per LDS row
constexpr int kThreads = 256;
constexpr int kXcds = 8;

static_assert(BM == 128 && BN == 128 && BK == 16, "the load mapping assumes 128 x 128 x 16 tiles and 4 waves");

__global__ void __launch_bounds__(kThreads, 2) slice_gemm_kernel(int64_t m, int64_t n, int64_t kp, int64_t mp,
                                                                 int64_t np, int tiles_n, int ntiles,
                                                                 const double* __restrict__ DAt,
                                                                 const double* __restrict__ DBp,
                                                                 double* __restrict__ out, const JobTable jobs) {
  __shared__ double As[2][BK * LDS_LD];
  __shared__ double Bs[2][BK * LDS_LD];

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
  const int64_t plane_a = kp * mp, plane_b = kp * np;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;  // 2 x 2 waves, 64 x 64 each

  const int64_t nkb = kp / BK;
  const int64_t niter = nkb * npairs;

  // Step copies: 16 panel rows x 128 doubles per operand = 1024 16-byte pieces,
  // four per thread; piece idx = r * 256 + tid covers row idx / 64, doubles
  // 2 (idx % 64) .. +1.  A wave reads 1 KB contiguous per instruction.
  typedef double d2 __attribute__((ext_vector_type(2)));
  d2 ra[4], rb[4];
  const int prow = tid >> 6, pcol = 2 * (tid & 63);
  auto load = [&](int pi, int64_t kb) {
    const double* a = DAt + static_cast<int64_t>(p_first + pi) * plane_a + (kb * BK + prow) * mp + m0 + pcol;
    const double* b = DBp + static_cast<int64_t>(q_first - pi) * plane_b + (kb * BK + prow) * np + n0 + pcol;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ra[r] = *reinterpret_cast<const d2*>(a + 4 * r * mp);
      rb[r] = *reinterpret_cast<const d2*>(b + 4 * r * np);
    }
  };
  auto store = [&](int stage) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      *reinterpret_cast<d2*>(&As[stage][(prow + 4 * r) * LDS_LD + pcol]) = ra[r];
      *reinterpret_cast<d2*>(&Bs[stage][(prow + 4 * r) * LDS_LD + pcol]) = rb[r];
    }
  };

  d4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};

  int pi = 0;
  int64_t kb = 0;
  if (niter > 0) {
    load(0, 0);
    store(0);
  }
  __syncthreads();

  const int frag_col = lane & 15, frag_k = lane >> 4;
  for (int64_t it = 0; it < niter; ++it) {
    const int cur = static_cast<int>(it & 1);
    const bool more = it + 1 < niter;
    if (more) {
      if (++kb == nkb) {
        kb = 0;
        ++pi;
      }
      load(pi, kb);  // in flight during this step's MFMAs
    }
    // 16 x 64 x 64 per wave: four k-groups of 16 MFMAs, the fragments of
    // group kg+1 read while group kg runs.
    const double* as = As[cur] + frag_k * LDS_LD + wr * 64 + frag_col;
    const double* bs = Bs[cur] + frag_k * LDS_LD + wc * 64 + frag_col;
    double af[2][4], bf[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[0][i] = as[i * 16];
      bf[0][i] = bs[i * 16];
    }
#pragma unroll
    for (int kg = 0; kg < BK / 4; ++kg) {
      const int c = kg & 1;
      if (kg + 1 < BK / 4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          af[c ^ 1][i] = as[(kg + 1) * 4 * LDS_LD + i * 16];
          bf[c ^ 1][i] = bs[(kg + 1) * 4 * LDS_LD + i * 16];
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[c][i], bf[c][j], acc[i][j], 0, 0, 0);
    }
    if (more) store(cur ^ 1);
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

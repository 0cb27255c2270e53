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
// first, single pairs, or the products of combinations of a Karatsuba
// schedule; each job lists its pairs in a device table, see schedule.h).  A
// job may cover one k chunk of its pairs (small products split k so that
// enough blocks fill the chip; the chunks' planes are added exactly later).  Tiles are renumbered so that each of the 8 XCDs
// (blocks are dealt to XCDs round-robin) works on its own chunk of tiles, and
// the blocks resident on one XCD at a time cover an about 8 x 8 patch whose
// panel rows stay in that XCD's L2.
#include <algorithm>

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
                                                                 double* __restrict__ out,
                                                                 const uint32_t* __restrict__ jobs,
                                                                 const uint32_t* __restrict__ pairs) {
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
  // the job's pairs (uniform: scalar loads); the pair after the one being
  // copied is fetched one pair ahead
  const int job = blockIdx.y;
  const uint32_t jw = jobs[3 * job], kw = jobs[3 * job + 2];
  const int pfirst = static_cast<int>(jw & 0xffffu), npairs = static_cast<int>(jw >> 16);
  const int64_t out_plane = jobs[3 * job + 1];
  // k chunk kw & 0xffff of kw >> 16: k steps [kb0, kb0 + nkb) of every pair (maybe none)
  const int64_t ksplit = kw >> 16, chunk = kw & 0xffffu;
  const int64_t plane_a = kp * mp, plane_b = kp * np;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;  // 2 x 2 waves, 64 x 64 each

  const int64_t nkb_all = kp / BK, csz = (nkb_all + ksplit - 1) / ksplit;
  const int64_t kb0 = min(chunk * csz, nkb_all), nkb = min(csz, nkb_all - kb0);
  const int64_t niter = nkb * npairs;

  // Direct global -> LDS copies (global_load_lds_dwordx4, 1 KB panel row per wave
  // instruction); wave w copies rows 4w .. 4w+3 of the A and of the B tile.
  const int lane_off = 2 * lane;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  int lpi = 0;
  int64_t lkb = 0;  // the step the next copy fetches
  uint32_t pr = pairs[pfirst];                             // pair lpi
  uint32_t pr_next = npairs > 1 ? pairs[pfirst + 1] : 0u;  // pair lpi + 1
  // this wave's first copy row of the pair's panels; advanced by one k step per copy
  const int64_t row_a = (kb0 * BK + 4 * wave_u) * mp + m0, row_b = (kb0 * BK + 4 * wave_u) * np + n0;
  const double* a = DAt + static_cast<int64_t>(pr & 0xffffu) * plane_a + row_a;
  const double* b = DBp + static_cast<int64_t>(pr >> 16) * plane_b + row_b;
  auto issue = [&](int stage) {
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
      pr = pr_next;
      if (lpi + 1 < npairs) pr_next = pairs[pfirst + lpi + 1];
      a = DAt + static_cast<int64_t>(pr & 0xffffu) * plane_a + row_a;
      b = DBp + static_cast<int64_t>(pr >> 16) * plane_b + row_b;
    } else {
      a += BK * mp;
      b += BK * np;
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

  double* o = out + out_plane * m * n;
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

// ---- the same product on FP32 panels ------------------------------------------
//
// Every digit and digit sum is an integer below 2^24 (checked on the host), so
// the panels hold it exactly as FP32: half the split's writes and half the
// GEMM's panel traffic.  The LDS footprint of a 16-deep FP64 step then holds a
// 32-deep FP32 step, so each barrier is followed by 128 MFMAs per wave instead
// of 64.  Each fragment value is widened back to FP64 (v_cvt_f64_f32, exact)
// right before its MFMAs.
//
// LDS rows are 128 floats without padding, so that one buffer_load_dwordx4 ...
// lds (64 lanes x 16 bytes) fills two rows in place; instead of padding, the 16-byte
// granules of row r are stored XOR-swizzled by (r & 3) << 2.  A fragment read
// (lanes 16h..16h+15 read row 4kg + h, 16 consecutive columns) then touches four
// different 16-bank groups for h = 0..3: conflict-free.  Panels are k-major and
// zero-padded to k multiple of 32, m / n multiple of 128.
//
// Outputs of at most 64 rows (the V^T X products of a blocked QR) take tiles of
// kRows = 64 rows: the same 128 columns and waves, each wave 32 x 64, A's LDS
// rows 64 floats (one copy instruction fills four), swizzled the same way.  A
// 128-row tile would spend half of its MFMAs on padding rows.
constexpr int BK32 = 32;
constexpr int ROW32 = 128;  // floats per LDS row of B (and of A for 128-row tiles)

// The k loop of slice_gemm32_kernel.  The two LDS stages (A0, B0 and A1, B1)
// are restrict parameters, so that the fragment reads of one stage carry alias
// scopes that exclude the copies in flight into the other: the compiler then
// makes no read wait for them, and the next step's copies go out right after
// the step's first fragment reads, a whole step (128 MFMAs per wave) ahead of
// their use.  The copies are buffer loads into LDS (counted on vmcnt only) from
// a resource based at the current pair's rows; the loop is unrolled by two so
// that each step's stages are fixed.  The four stage buffers must be distinct
// arrays for the scopes to hold (halves of one array were not told apart, and
// every read then waited for the copies).  Measured against the copies issued
// after the last read (32 MFMAs ahead): 1.7-1.9% less level-GEMM time on four
// workloads, the same bits; issuing them after the first two read groups
// instead of before them, another 0.3-0.6%.
template <int kRows>
__device__ __forceinline__ void gemm32_k_loop(float* __restrict__ A0, float* __restrict__ B0, float* __restrict__ A1,
                                              float* __restrict__ B1, const float* DAt, const float* DBp,
                                              const uint32_t* pairs, int pfirst, int npairs, int64_t nkb,
                                              int64_t plane_a, int64_t plane_b, int64_t mp, int64_t np,
                                              int64_t row_a, int64_t row_b, int wave_u,
                                              const int32_t (&off_a)[kRows / 32], const int32_t (&off_b)[4],
                                              const int (&fa)[kRows / 32], const int (&fb)[4],
                                              d4 (&acc)[kRows / 32][4]) {
  constexpr int kMI = kRows / 32, kRowsA = 256 / kRows;
  const int64_t niter = nkb * npairs;
  int lpi = 0;
  int64_t lkb = 0;
  // The pair word is read (scalar load) where the copies switch to the next pair
  // and used at once, so that no scalar load is pending while the fragment reads
  // are: the LDS counter then orders the reads alone and each group of MFMAs
  // waits for its own reads only.
  uint32_t pr = pairs[pfirst];
  const float* a = DAt + static_cast<int64_t>(pr & 0xffffu) * plane_a + row_a;
  const float* b = DBp + static_cast<int64_t>(pr >> 16) * plane_b + row_b;
  auto issue = [&](float* An, float* Bn) {
    // the largest record count: no range limit (the copies stay within the panels)
    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a), 0, 0xffffffff, kBufferWord3);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(b), 0, 0xffffffff, kBufferWord3);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < kMI)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(An + (8 * wave_u + kRowsA * q) * kRows), 16,
                                                 4 * off_a[q], 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(Bn + (8 * wave_u + 2 * q) * ROW32), 16,
                                               4 * off_b[q], 0, 0, 0);
    }
    if (++lkb == nkb) {
      lkb = 0;
      ++lpi;
      if (lpi < npairs) pr = pairs[pfirst + lpi];
      a = DAt + static_cast<int64_t>(pr & 0xffffu) * plane_a + row_a;
      b = DBp + static_cast<int64_t>(pr >> 16) * plane_b + row_b;
    } else {
      a += BK32 * mp;
      b += BK32 * np;
    }
  };
  auto step = [&](const float* as, const float* bs, float* An, float* Bn, bool more) {
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);  // this wave's copies of this step are in LDS
    __syncthreads();                          // everyone's are; everyone is done reading the other stage
    float af[BK32 / 4][kMI], bf[BK32 / 4][4];
    // fragments of k groups 2g and 2g + 1 (2 (kMI + 4) LDS instructions)
    auto read = [&](int g) {
#pragma unroll
      for (int kg = 2 * g; kg < 2 * g + 2; ++kg)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (i < kMI) af[kg][i] = as[kg * 4 * kRows + fa[i]];
          bf[kg][i] = bs[kg * 4 * ROW32 + fb[i]];
        }
    };
    auto mfma = [&](int kg) {
      double ad[kMI], bd[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (i < kMI) ad[i] = static_cast<double>(af[kg][i]);
        bd[i] = static_cast<double>(bf[kg][i]);
      }
#pragma unroll
      for (int i = 0; i < kMI; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(ad[i], bd[j], acc[i][j], 0, 0, 0);
    };
    // The reads go out in four groups, each one MFMA group ahead of its use, so
    // that at most 16 are outstanding and every wait is a partial one.
    // sched_barrier keeps the compiler from merging the groups back together.
    read(0);
    read(1);
    __builtin_amdgcn_sched_barrier(0);
    if (more) issue(An, Bn);
    __builtin_amdgcn_sched_barrier(0);
    mfma(0);
    mfma(1);
    __builtin_amdgcn_sched_barrier(0);
    read(2);
    __builtin_amdgcn_sched_barrier(0);
    mfma(2);
    mfma(3);
    __builtin_amdgcn_sched_barrier(0);
    read(3);
    __builtin_amdgcn_sched_barrier(0);
    mfma(4);
    mfma(5);
    mfma(6);
    mfma(7);
  };
  if (niter > 0) issue(A0, B0);
  for (int64_t it = 0; it < niter; it += 2) {
    step(A0, B0, A1, B1, it + 1 < niter);
    if (it + 1 < niter) step(A1, B1, A0, B0, it + 2 < niter);
  }
}

template <int kRows>
__global__ void __launch_bounds__(kThreads, 2) slice_gemm32_kernel(int64_t m, int64_t n, int64_t kp, int64_t mp,
                                                                   int64_t np, int tiles_n, int ntiles,
                                                                   const float* __restrict__ DAt,
                                                                   const float* __restrict__ DBp,
                                                                   double* __restrict__ out,
                                                                   const uint32_t* __restrict__ jobs,
                                                                   const uint32_t* __restrict__ pairs) {
  static_assert(kRows == 128 || kRows == 64, "tile rows");
  constexpr int kMI = kRows / 32;       // 16-row blocks per wave, and A copy instructions per wave and step
  constexpr int kRowsA = 256 / kRows;   // A rows filled by one copy instruction
  // the two LDS stages as four arrays (the k loop takes them as restrict pointers)
  __shared__ __attribute__((aligned(1024))) float A0s[BK32 * kRows];
  __shared__ __attribute__((aligned(1024))) float B0s[BK32 * ROW32];
  __shared__ __attribute__((aligned(1024))) float A1s[BK32 * kRows];
  __shared__ __attribute__((aligned(1024))) float B1s[BK32 * ROW32];

  // tile order as in slice_gemm_kernel
  int t = blockIdx.x;
  {
    const int per = ntiles / kXcds;
    if (t < per * kXcds) t = (t % kXcds) * per + t / kXcds;
  }
  const int tiles_m = ntiles / tiles_n;
  const int gsz = kGroup * tiles_n, g = t / gsz, first = g * kGroup;
  const int rows_in = min(kGroup, tiles_m - first), within = t - g * gsz;
  const int64_t m0 = static_cast<int64_t>(first + within % rows_in) * kRows;
  const int64_t n0 = static_cast<int64_t>(within / rows_in) * BN;
  const int job = blockIdx.y;
  const uint32_t jw = jobs[3 * job], kw = jobs[3 * job + 2];
  const int pfirst = static_cast<int>(jw & 0xffffu), npairs = static_cast<int>(jw >> 16);
  const int64_t out_plane = jobs[3 * job + 1];
  // k chunk kw & 0xffff of kw >> 16: k steps [kb0, kb0 + nkb) of every pair (maybe none)
  const int64_t ksplit = kw >> 16, chunk = kw & 0xffffu;
  const int64_t plane_a = kp * mp, plane_b = kp * np;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  const int64_t nkb_all = kp / BK32, csz = (nkb_all + ksplit - 1) / ksplit;
  const int64_t kb0 = min(chunk * csz, nkb_all), nkb = min(csz, nkb_all - kb0);

  // Copies: wave w fills rows 8w .. 8w+7 of each tile.  B: two rows per
  // instruction (q = 0..3); lane L lands at row 8w + 2q + L/32, granule L%32, and
  // fetches the panel granule (L%32) ^ (((2q + L/32) & 3) << 2) of that row.  A:
  // the same with kRows / 4 granules per row, kRowsA rows per instruction.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int half = lane >> 5, gran = lane & 31;
  const int row_in_a = lane / (kRows / 4), gran_a = lane % (kRows / 4);
  int32_t off_a[kMI], off_b[4];  // per-lane source offsets in floats, relative to the wave's first row
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = 2 * q + half;
    const int sg = gran ^ ((r & 3) << 2);
    if (kRows == 128) off_a[q % kMI] = static_cast<int32_t>(r * mp + 4 * sg);
    off_b[q] = static_cast<int32_t>(r * np + 4 * sg);
  }
  if (kRows == 64) {
#pragma unroll
    for (int q = 0; q < kMI; ++q) {
      const int r = kRowsA * q + row_in_a;
      off_a[q] = static_cast<int32_t>(r * mp + 4 * (gran_a ^ ((r & 3) << 2)));
    }
  }
  const int64_t row_a = (kb0 * BK32 + 8 * wave_u) * mp + m0, row_b = (kb0 * BK32 + 8 * wave_u) * np + n0;
  d4 acc[kMI][4];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = d4{0.0, 0.0, 0.0, 0.0};

  // Fragments: lane l = 16h + c reads row 4kg + h; the wave's column block
  // kMI * wr + i (16 floats each) lies at block (kMI * wr + i) ^ h after the
  // swizzle (for 128-row tiles that is wr * 64 + ((i ^ h) << 4): the swizzle
  // stays within the wave's 64 floats).
  const int h = lane >> 4, c = lane & 15;
  int fa[kMI], fb[4];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
    fa[i] = h * kRows + (kRows == 128 ? wr * 64 + ((i ^ h) << 4) : ((kMI * wr + i) ^ h) << 4) + c;
#pragma unroll
  for (int i = 0; i < 4; ++i) fb[i] = h * ROW32 + wc * 64 + ((i ^ h) << 4) + c;
  gemm32_k_loop<kRows>(A0s, B0s, A1s, B1s, DAt, DBp, pairs, pfirst, npairs, nkb, plane_a, plane_b, mp, np,
                       row_a, row_b, wave_u, off_a, off_b, fa, fb, acc);

  double* o = out + out_plane * m * n;
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = m0 + wr * (kRows / 2) + i * 16 + 4 * r + (lane >> 4);
        const int64_t gj = n0 + wc * 64 + j * 16 + (lane & 15);
        if (gi < m && gj < n) o[gi * n + gj] = acc[i][j][r];
      }
}

}  // namespace

hipError_t launch_slice_gemm(int64_t m, int64_t n, int64_t k, const double* DAt, const double* DBp, double* out,
                             const GemmJobs& jobs, hipStream_t stream) {
  if (m == 0 || n == 0 || jobs.njobs == 0) return hipSuccess;
  const int64_t mp = panel_mn(m), np = panel_mn(n), kp = panel_k(k);
  const int64_t tiles_n = np / BN;
  const int64_t ntiles = (mp / BM) * tiles_n;
  if (ntiles > 0x7fffffff || jobs.njobs > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(slice_gemm_kernel, dim3(static_cast<unsigned>(ntiles), static_cast<unsigned>(jobs.njobs)),
                     dim3(kThreads), 0, stream, m, n, kp, mp, np, static_cast<int>(tiles_n),
                     static_cast<int>(ntiles), DAt, DBp, out, jobs.jobs, jobs.pairs);
  return hipGetLastError();
}

hipError_t launch_slice_gemm32(int64_t m, int64_t n, int64_t k, const float* DAt, const float* DBp, double* out,
                               const GemmJobs& jobs, hipStream_t stream) {
  if (m == 0 || n == 0 || jobs.njobs == 0) return hipSuccess;
  const int64_t mp = panel_mn(m), np = panel_mn(n), kp = panel_k32(k);
  const int64_t tiles_n = np / BN;
  const bool skinny = m <= 64;  // one 64-row tile row (within the panel's 128 padded rows)
  const int64_t ntiles = (skinny ? 1 : mp / BM) * tiles_n;
  // per-lane copy offsets are 32-bit: 7 rows of a panel plus a row's width
  if (ntiles > 0x7fffffff || jobs.njobs > 65535 || mp > (1 << 27) || np > (1 << 27)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(ntiles), static_cast<unsigned>(jobs.njobs));
  if (skinny)
    hipLaunchKernelGGL(slice_gemm32_kernel<64>, grid, dim3(kThreads), 0, stream, m, n, kp, mp, np,
                       static_cast<int>(tiles_n), static_cast<int>(ntiles), DAt, DBp, out, jobs.jobs, jobs.pairs);
  else
    hipLaunchKernelGGL(slice_gemm32_kernel<128>, grid, dim3(kThreads), 0, stream, m, n, kp, mp, np,
                       static_cast<int>(tiles_n), static_cast<int>(ntiles), DAt, DBp, out, jobs.jobs, jobs.pairs);
  return hipGetLastError();
}

namespace {

constexpr int kUploadWords = 480;
struct WordChunk {
  uint32_t count;
  uint32_t w[kUploadWords];
};

__global__ void __launch_bounds__(256) upload_kernel(const WordChunk c, uint32_t* __restrict__ dst) {
  for (uint32_t i = threadIdx.x; i < c.count; i += blockDim.x) dst[i] = c.w[i];
}

constexpr int kComboChunk = 160;
struct ComboChunk {
  int count;
  uint16_t child[kComboChunk], p1[kComboChunk], p2[kComboChunk];
};

// panel child = panel p1 + panel p2 (integers below 2^24 for FP32 panels, below
// 2^53 for FP64: exact), two values per thread
template <class T>
__global__ void __launch_bounds__(256) combination_kernel(const ComboChunk c, T* __restrict__ D, int64_t plane) {
  const int e = blockIdx.y;
  const T* a = D + static_cast<int64_t>(c.p1[e]) * plane;
  const T* b = D + static_cast<int64_t>(c.p2[e]) * plane;
  T* d = D + static_cast<int64_t>(c.child[e]) * plane;
  for (int64_t i = 2 * (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x); i < plane;
       i += 2 * static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const T x0 = a[i], x1 = a[i + 1], y0 = b[i], y1 = b[i + 1];
    d[i] = x0 + y0;
    d[i + 1] = x1 + y1;
  }
}

// FP64 panels [S][kp_src][cp] -> FP32 panels [S][kp_dst][cp] (kp_dst >= kp_src, zero
// rows beyond kp_src); values are integers below 2^24, so the conversion is exact.
__global__ void __launch_bounds__(256) panel_to_f32_kernel(const double* __restrict__ src, float* __restrict__ dst,
                                                           int64_t kp_src, int64_t kp_dst, int64_t cp, int S) {
  const int64_t total = static_cast<int64_t>(S) * kp_dst * cp;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const int64_t s = i / (kp_dst * cp), r = (i / cp) % kp_dst, c = i % cp;
    dst[i] = r < kp_src ? static_cast<float>(src[(s * kp_src + r) * cp + c]) : 0.0f;
  }
}

}  // namespace

hipError_t launch_upload(const std::vector<uint32_t>& words, uint32_t* dst, hipStream_t stream) {
  for (size_t off = 0; off < words.size(); off += kUploadWords) {
    WordChunk c;
    c.count = static_cast<uint32_t>(std::min<size_t>(kUploadWords, words.size() - off));
    for (uint32_t i = 0; i < c.count; ++i) c.w[i] = words[off + i];
    hipLaunchKernelGGL(upload_kernel, dim3(1), dim3(256), 0, stream, c, dst + off);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

template <class T>
hipError_t combinations(const Schedule& s, bool a, T* D, int64_t plane, hipStream_t stream) {
  const std::vector<int>& depth = a ? s.depth_a : s.depth_b;
  const std::vector<int>& p1 = a ? s.par1_a : s.par1_b;
  const std::vector<int>& p2 = a ? s.par2_a : s.par2_b;
  int max_depth = 0;
  for (int d : depth) max_depth = std::max(max_depth, d);
  // panels are whole multiples of 16 x 128 values: an even count
  const unsigned gx = static_cast<unsigned>(std::min<int64_t>((plane / 2 + 255) / 256, 1024));
  for (int d = 1; d <= max_depth; ++d) {
    ComboChunk c;
    c.count = 0;
    auto flush = [&]() -> hipError_t {
      if (c.count == 0) return hipSuccess;
      hipLaunchKernelGGL(combination_kernel<T>, dim3(gx, static_cast<unsigned>(c.count)), dim3(256), 0, stream, c, D,
                         plane);
      c.count = 0;
      return hipGetLastError();
    };
    for (size_t i = 0; i < depth.size(); ++i) {
      if (depth[i] != d) continue;
      c.child[c.count] = static_cast<uint16_t>(i);
      c.p1[c.count] = static_cast<uint16_t>(p1[i]);
      c.p2[c.count] = static_cast<uint16_t>(p2[i]);
      if (++c.count == kComboChunk) {
        const hipError_t err = flush();
        if (err != hipSuccess) return err;
      }
    }
    const hipError_t err = flush();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

hipError_t launch_combinations(const Schedule& s, bool a, double* D, int64_t plane, hipStream_t stream) {
  return combinations<double>(s, a, D, plane, stream);
}

hipError_t launch_combinations32(const Schedule& s, bool a, float* D, int64_t plane, hipStream_t stream) {
  return combinations<float>(s, a, D, plane, stream);
}

hipError_t launch_panel_to_f32(const double* src, float* dst, int64_t kp_src, int64_t kp_dst, int64_t cp, int S,
                               hipStream_t stream) {
  const int64_t total = static_cast<int64_t>(S) * kp_dst * cp;
  if (total == 0) return hipSuccess;
  const unsigned g = static_cast<unsigned>(std::min<int64_t>((total + 255) / 256, 4096));
  hipLaunchKernelGGL(panel_to_f32_kernel, dim3(g), dim3(256), 0, stream, src, dst, kp_src, kp_dst, cp, S);
  return hipGetLastError();
}

}  // namespace mdg

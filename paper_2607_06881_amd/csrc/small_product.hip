// The whole product for small outputs in one launch: exponents, exact split,
// level products, exact accumulation and rounding (steps a1-a5) fused per
// 16 x 16 tile of C.
//
// For a small C the staged path is latency-bound: its level GEMM gives each
// 128 x 128 tile and level to one block (a 64 x 64 product leaves three
// quarters of every MFMA on padding, and its heaviest level runs all its pairs
// one after another in one block), and its seven launches each cost a few
// microseconds.  Here one block owns a 16 x 16 tile of C, the tile of the
// v_mfma_f64_16x16x4f64 instruction, and runs the five steps of the overview of
// section 2 itself:
//  1. the grid exponents of its 16 rows of A and 16 columns of B (section 3,
//     one power-of-two grid per line; the largest frexp exponent of the leading
//     limbs), the same reduction as the staged exponents kernels;
//  2. the exact split of those rows and columns into w-bit digits (section 2),
//     k chunk by k chunk, into LDS as FP32 values (integers below 2^24, exact);
//  3. the level products G_t = sum over p + q = t of DA_p . DB_q (section 2,
//     equation (3) and the rewritten product): every level belongs to one of
//     the eight waves, two per SIMD (the host balances the pair counts of the
//     SIMDs and of the two waves within each), which sums its pairs for the
//     chunk in one FP64 accumulator and adds it to the level's plane in LDS;
//     every partial sum is an integer below 2^53, so the result is exact and
//     equal to the staged path's;
//  4.-5. the exact sum of the levels in increasing significance and the greedy
//     rounding into L limbs, one thread per output element, from LDS.
// The digits, levels and limbs are those of the staged kernels bit for bit
// (the same device arithmetic, digits.h).
#include <mutex>

#include "digits.h"
#include "internal.h"

namespace mdg {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 16;
constexpr int kThreads = 64 * kSmallWaves;  // two waves per SIMD
constexpr int kPhases = kThreads / kTile;    // row phases of the column exponents
constexpr int kBatch = 4;  // elements whose limbs a thread loads before splitting them

// The S digits of one element (limbs xs, grid exponent g) to out[s * stride],
// FP32.  Digit windows of at most 128 bits (w S <= 128: double-double at 13-bit
// digits and the adaptive widths) take the 128-bit integer floor, windows of at
// most 256 bits (triple- and quad-double) the 256-bit one, the others the
// general one (the same digits).
template <int NW, int ML>
__device__ inline void split_into(const double (&xs)[ML], int L, int g, int S, int w, float* __restrict__ out,
                                  int64_t stride) {
  if (w * S <= 128) {
    uint64_t I[2];
    const bool neg = floor_on_grid_128<ML>(xs, L, g, I);
    store_digits<2, float>(I, S, w, neg, out, stride);
  } else if (w * S <= 256) {
    uint64_t I[4];
    const bool neg = floor_on_grid_256<ML>(xs, L, g, I);
    store_digits<4, float>(I, S, w, neg, out, stride);
  } else {
    uint64_t I[NW];
    const bool neg = floor_on_grid<NW, ML>(xs, L, g, I);
    store_digits<NW, float>(I, S, w, neg, out, stride);
  }
}

__device__ inline int wave_max_i(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
  return v;
}

// LDS: digits of A [S][16][kc + 1] and of B [S][kc][16] (FP32), levels [T+1][256]
// (FP64), exponents and partial column maxima.
template <int NWS, int NWA, int ML>
__global__ void __launch_bounds__(kThreads) small_product_kernel(int64_t m, int64_t n, int64_t k, int L, int S, int T,
                                                                 int w, int kc, SmallLevelOwners owners,
                                                                 const double* __restrict__ A,
                                                                 const double* __restrict__ B, double* __restrict__ C) {
  extern __shared__ double lds_d[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t i0 = static_cast<int64_t>(blockIdx.y) * kTile, j0 = static_cast<int64_t>(blockIdx.x) * kTile;
  const int lda = kc + 1;  // odd row pitch of A's digits: the 16 rows of a fragment read fall on distinct banks
  double* G = lds_d;                                          // [T+1][256]
  float* sA = reinterpret_cast<float*>(G + (T + 1) * kTile * kTile);  // [S][16][lda]
  float* sB = sA + S * kTile * lda;                           // [S][kc][16]
  __shared__ int eA[kTile], eB[kTile], part[kPhases][kTile];

  // 1. grid exponents of the tile's rows of A (wave w: rows R w .. R w + R - 1,
  //    R = 16 / waves, their loads issued together) and columns of B (kPhases
  //    phases of rows)
  {
    constexpr int R = kTile / kSmallWaves;
    int best[R];
#pragma unroll
    for (int r = 0; r < R; ++r) best[r] = kNoExp;
    for (int64_t kk = lane; kk < k; kk += 64) {
      double v[R];
#pragma unroll
      for (int r = 0; r < R; ++r) v[r] = i0 + R * wave + r < m ? A[(i0 + R * wave + r) * k + kk] : 0.0;
#pragma unroll
      for (int r = 0; r < R; ++r) best[r] = max(best[r], frexp_exp_or_min(v[r]));
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int b = wave_max_i(best[r]);
      if (lane == 0) eA[R * wave + r] = b == kNoExp ? 0 : b;
    }
  }
  {
    const int col = tid & 15, phase = tid >> 4;
    int best = kNoExp;
    if (j0 + col < n) {
#pragma unroll 4
      for (int64_t kk = phase; kk < k; kk += kPhases) best = max(best, frexp_exp_or_min(B[kk * n + j0 + col]));
    }
    part[phase][col] = best;
  }
  for (int t = tid; t < (T + 1) * kTile * kTile; t += kThreads) G[t] = 0.0;
  __syncthreads();
  if (tid < kTile) {
    int best = kNoExp;
    for (int ph = 0; ph < kPhases; ++ph) best = max(best, part[ph][tid]);
    eB[tid] = best == kNoExp ? 0 : best;
  }
  __syncthreads();

  const int64_t planeA = m * k, planeB = k * n;
  for (int64_t k0 = 0; k0 < k; k0 += kc) {
    const int kn = static_cast<int>(k - k0 < kc ? k - k0 : kc);  // valid k of this chunk
    const int kn4 = (kn + 3) & ~3;                                   // rounded up to the MFMA depth
    // 2. digits of the chunk: A's 16 x kn4 elements (consecutive threads on
    //    consecutive k) and B's kn4 x 16 (consecutive threads on consecutive
    //    columns); the limbs of a thread's kBatch elements are loaded before any
    //    of them is split
    for (int e0 = 0; e0 < kTile * kn4; e0 += kThreads * kBatch) {
      double xs[kBatch][ML];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int e = e0 + b * kThreads + tid, row = e / kn4, kk = e - row * kn4;
        const bool ok = e < kTile * kn4 && i0 + row < m && kk < kn;
        const int64_t idx = ok ? (i0 + row) * k + k0 + kk : 0;
        load_limbs<ML>(A, planeA, ok ? L : 0, idx, xs[b]);
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int e = e0 + b * kThreads + tid, row = e / kn4, kk = e - row * kn4;
        if (e >= kTile * kn4) break;
        float* out = sA + row * lda + kk;
        split_into<NWS, ML>(xs[b], L, eA[row] - w * S, S, w, out, kTile * lda);  // zero limbs: zero digits
      }
    }
    for (int e0 = 0; e0 < kn4 * kTile; e0 += kThreads * kBatch) {
      double xs[kBatch][ML];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int e = e0 + b * kThreads + tid, kk = e >> 4, col = e & 15;
        const bool ok = e < kn4 * kTile && j0 + col < n && kk < kn;
        const int64_t idx = ok ? (k0 + kk) * n + j0 + col : 0;
        load_limbs<ML>(B, planeB, ok ? L : 0, idx, xs[b]);
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int e = e0 + b * kThreads + tid, kk = e >> 4, col = e & 15;
        if (e >= kn4 * kTile) break;
        float* out = sB + kk * kTile + col;
        split_into<NWS, ML>(xs[b], L, eB[col] - w * S, S, w, out, kc * kTile);
      }
    }
    __syncthreads();
    // 3. this wave's levels: lane l supplies A[l%16][l/16] and B[l/16][l%16] of
    //    each 16 x 4 by 4 x 16 step; register r of lane l holds D[4r + l/16][l%16]
    const int fi = lane & 15, fk = lane >> 4;
    for (int t = 0; t <= T; ++t) {
      if (owners.wave[t] != wave) continue;
      // four independent accumulators (16-deep steps) so that the matrix pipe
      // never waits on one chain; their sums are integers below 2^53: exact
      d4 acc[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[c] = d4{0.0, 0.0, 0.0, 0.0};
      const int p0 = t - (S - 1) > 0 ? t - (S - 1) : 0, p1 = t < S - 1 ? t : S - 1;
      for (int p = p0; p <= p1; ++p) {
        const float* a = sA + (p * kTile + fi) * lda + fk;
        const float* b = sB + ((t - p) * kc + fk) * kTile + fi;
        int kk = 0;
        for (; kk + 16 <= kn4; kk += 16) {
          float av[4], bv[4];
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            av[c] = a[kk + 4 * c];
            bv[c] = b[(kk + 4 * c) * kTile];
          }
#pragma unroll
          for (int c = 0; c < 4; ++c)
            acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(static_cast<double>(av[c]), static_cast<double>(bv[c]),
                                                          acc[c], 0, 0, 0);
        }
        for (; kk < kn4; kk += 4)
          acc[0] = __builtin_amdgcn_mfma_f64_16x16x4f64(static_cast<double>(a[kk]),
                                                        static_cast<double>(b[kk * kTile]), acc[0], 0, 0, 0);
      }
      const d4 sum = (acc[0] + acc[1]) + (acc[2] + acc[3]);
      double* g = G + t * kTile * kTile + fk * kTile + fi;
#pragma unroll
      for (int r = 0; r < 4; ++r) g[4 * r * kTile] += sum[r];  // this wave alone owns level t
    }
    __syncthreads();  // the next chunk overwrites the digits; after the last, the levels are complete
  }

  // 4.-5. exact accumulation and greedy rounding, one thread per output element
  const int i = tid >> 4, j = tid & 15;
  if (tid < kTile * kTile && i0 + i < m && j0 + j < n) {
    uint64_t N[NWA];
#pragma unroll
    for (int q = 0; q < NWA; ++q) N[q] = 0;
    CarryChain<NWA> chain;
    const uint64_t mask = (1ull << w) - 1ull;
    for (int t = T; t >= 0; --t) chain.step(N, static_cast<int64_t>(G[t * kTile * kTile + tid]), w, mask);
    chain.finish(N, w, T);
    const int scale = eA[i] + eB[j] - 2 * w - w * T;
    round_limbs<NWA>(N, L, scale, C, m * n, (i0 + i) * n + j0 + j);
  }
}

}  // namespace

size_t small_product_lds(int S, int T, int kc) {
  return sizeof(double) * static_cast<size_t>(T + 1) * kTile * kTile +
         sizeof(float) * static_cast<size_t>(S) * kTile * (kc + 1) +
         sizeof(float) * static_cast<size_t>(S) * kc * kTile;
}

hipError_t launch_small_product(int64_t m, int64_t n, int64_t k, int L, int S, int T, int w, int kc,
                                const SmallLevelOwners& owners, const double* A, const double* B, double* C,
                                hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  if (L < 1 || L > kSmallMaxLimbs || S < 1 || w < 1 || w > 24 || T < 0 || T > 2 * S - 2 ||
      T + 1 > kSmallMaxLevels || kc < 4 || kc % 4 != 0 || k < 1 || w * S + 52 > 64 * kSmallSplitWords ||
      w * T + 55 > 64 * kSmallAccumWords)
    return hipErrorInvalidValue;
  const size_t lds = small_product_lds(S, T, kc);
  if (lds > kSmallMaxLds) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>((n + kTile - 1) / kTile), static_cast<unsigned>((m + kTile - 1) / kTile));
  // dynamic LDS beyond 64 KB: allowed once for the kernel (a failure here shows
  // up as a launch error below)
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute(
        reinterpret_cast<const void*>(&small_product_kernel<kSmallSplitWords, kSmallAccumWords, kSmallMaxLimbs>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kSmallMaxLds));
    (void)hipGetLastError();
  });
  hipLaunchKernelGGL((small_product_kernel<kSmallSplitWords, kSmallAccumWords, kSmallMaxLimbs>), grid,
                     dim3(kThreads), lds, stream, m, n, k, L, S, T, w, kc, owners, A, B, C);
  return hipGetLastError();
}

}  // namespace mdg

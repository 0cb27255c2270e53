// Step a3 on the int8 matrix cores, hand-written: every level product of
// section 2 in one launch.
//
// The level G_t = sum over p + q = t of DA_p . DB_q is an integer sum of
// products of digits of at most 7 bits; the caller has checked that it stays
// below 2^31, so the int8 x int8 -> int32 matrix instruction forms it exactly
// in any order and blocking.
//
// Operands (written by the int8 splits): the digits of row i of A and of
// column j of B, k-contiguous, in rows of pitch ld = kI8Pad + S kp bytes:
//     DA  [mp][ld]: bytes kI8Pad + p kp + kk hold digit p of A[i][kk],
//     DBt [np][ld]: bytes kI8Pad + (S-1-q) kp + kk hold digit q of B[kk][j],
// zeros in the first kI8Pad bytes of every row and for kk >= k; kp is a
// multiple of 128, mp and np are m and n rounded up to 256 (rows beyond m or n
// only feed outputs that are not stored).  The pairs of level t are then one
// contiguous k range of length K = (p1 - p0 + 1) kp, starting at p0 kp in every
// row of DA and at (S-1-t+p0) kp in every row of DBt.  When K / 128 is odd the
// range starts one 128-byte stage early: that stage is the zero pad of A's row
// (p0 = 0) or of B's row (p0 > 0 means t >= S, so B's range starts at its pad),
// and adds nothing.  (Levels are split into chunks of pairs only when a pair is
// an even number of stages, so a chunk never needs that.)
//
// CDNA4 mapping:
// * v_mfma_i32_16x16x64_i8: lane l supplies 16 bytes of row l%16 of the A block
//   and of column l%16 of the B block, at k granule l/16 (any k order works as
//   long as A and B agree); register r of lane l holds D[4 (l/16) + r][l%16].
// * One workgroup, eight waves (two per SIMD), owns a 256 x 256 output tile;
//   each wave holds a 128 x 64 sub-tile in 32 accumulator blocks (128 AGPRs,
//   220 registers in all, so two waves fit a SIMD: one issues while the other
//   waits; four waves of 128 x 128 ran 1-9% slower).  The MFMAs are issued as
//   inline instructions with AGPR accumulators: left to itself the register
//   allocator permutes accumulators between AGPRs and VGPRs across the loop,
//   dozens of copies per step that stall behind the MFMAs writing them.
// * k advances in stages of 128 bytes, two LDS stages (64 KB each: the A tile
//   then the B tile, 128-byte rows).  Copies go global -> LDS directly with
//   buffer_load_dwordx4 ... lds (counted on vmcnt only; the FLAT form would make
//   the compiler wait for every LDS read).  A ds_read_b128 is served 16 lanes at
//   a time over 64 banks, lanes 8a .. 8a+7 together with 32+8a .. 32+8a+7 (the
//   grouping that the bank-conflict counter confirms: a swizzle conflict-free
//   for 16 consecutive lanes still doubled every read).  A fragment read meets
//   8 rows twice there, at granules g and g ^ 2, so the 16-byte granules of LDS
//   row R are XOR-swizzled by swz(R) = bit1(R) | (bit0(R) ^ bit3(R)) << 1 |
//   bit2(R) << 2, which keeps all 16 accesses on distinct bank groups (and 16
//   consecutive lanes too).
// * A stage is two sub-steps of 32 MFMAs per wave; the fragments of the next
//   sub-step are read (four groups of three ds_read_b128) while the current one
//   runs.  The barrier sits before a stage's last sub-step: it certifies the
//   next stage's copies and frees the current buffer, whose next copies (two
//   stages ahead) are then issued one pair after every eighth MFMA: a burst of
//   copies blocks the wave's in-order issue and starves the matrix pipe.
//
// Work decomposition: grid.x = output tiles (renumbered per XCD, as in the
// FP64 kernel, in patches of `group` tile-rows), grid.y = jobs, heaviest first
// (a table in the kernel arguments): whole levels, or, for small outputs whose
// grid would hold few blocks, chunks of a level's pairs that add their partial
// sums into zeroed planes with int32 atomics (exact in any order).
#include <type_traits>

#include "internal.h"

namespace mdg {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTile = 256;                 // output tile edge
constexpr int kStage = 128;                // bytes of k per LDS stage
constexpr int kBuf = 2 * kTile * kStage;   // one LDS stage: A tile then B tile
constexpr int kXcds = 8;
constexpr unsigned kWaitVmLgkm0 = 0x0070;  // s_waitcnt vmcnt(0) lgkmcnt(0)
static_assert(kI8Pad == kStage, "the zero pad is one stage");

// the jobs of one launch, heaviest first: level t[y], its pairs first[y] ..
// first[y] + count[y] - 1 (indices into the level's pair range)
struct Jobs {
  uint8_t t[128], first[128], count[128];
};

// the granule swizzle of LDS row r (depends on r mod 16 only)
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 1) | ((((r & 1) ^ ((r >> 3) & 1))) << 1) | (r & 4); }

struct Frag {
  v4i a[8], b[4];
};

__device__ __forceinline__ void mfma(v4i& acc, const v4i& a, const v4i& b) {
  asm volatile("v_mfma_i32_16x16x64_i8 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// The k loop of one tile.  The buffers are restrict parameters so that the
// LDS reads of one carry alias scopes that exclude the copies in flight into
// the other (the compiler then waits for neither).
__device__ __forceinline__ void tile_loop(int8_t* __restrict__ P0, int8_t* __restrict__ P1, const int8_t* a,
                                          const int8_t* b, uint32_t na, uint32_t nb, int nst, uint32_t qs,
                                          uint32_t lo0, uint32_t lo1, int fa0, int fa1, int fb0, int fb1, int wave,
                                          v4i (&acc)[8][4]) {
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a), 0, na, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(b), 0, nb, kBufferWord3);
  // copy q (0..3) of stage s into buffer P: tile rows 32 wave + 8q .. +7 of A and of B
  auto copy = [&](int8_t* P, int s, int q) {
    const uint32_t so = static_cast<uint32_t>(s) * kStage + static_cast<uint32_t>(q) * qs;
    const uint32_t lo = (q & 1) ? lo1 : lo0;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(P + (32 * wave + 8 * q) * kStage), 16, lo, so, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(P + kTile * kStage + (32 * wave + 8 * q) * kStage), 16,
                                             lo, so, 0, 0);
  };
  auto read = [&](const int8_t* P, int h, Frag& f, int g) {
    const int oa = h ? fa1 : fa0, ob = h ? fb1 : fb0;
#pragma unroll
    for (int i = 2 * g; i < 2 * g + 2; ++i) f.a[i] = *reinterpret_cast<const v4i*>(P + oa + i * 16 * kStage);
    f.b[g] = *reinterpret_cast<const v4i*>(P + kTile * kStage + ob + g * 16 * kStage);
  };
  // rows 2g, 2g + 1 of the 8 x 4 blocks; with copies, copy pair g into P after the eighth MFMA
  auto run = [&](const Frag& f, int g, auto with_copies, int8_t* P, int s) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = 2 * g + (e >> 2), j = e & 3;
      mfma(acc[i][j], f.a[i], f.b[j]);
      if constexpr (decltype(with_copies)::value) {
        if (e == 7) {
          __builtin_amdgcn_sched_barrier(0);
          copy(P, s, g);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };
  // sub-step: the next fragments (buffer Q, half h) into nxt while cur runs
  auto step = [&](const int8_t* Q, int h, Frag& nxt, const Frag& cur, auto with_copies, int8_t* P, int s) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      read(Q, h, nxt, g);
      __builtin_amdgcn_sched_barrier(0);
      run(cur, g, with_copies, P, s);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  Frag x, y;
  // stage s in buffer P (sub-step 0 in x), stage s + 1 in Q
  auto stage = [&](int8_t* P, int8_t* Q, int s) {
    step(P, 1, y, x, std::false_type{}, P, 0);
    __builtin_amdgcn_s_waitcnt(kWaitVmLgkm0);  // this wave's copies of stage s + 1 are in LDS, its reads of P done
    __syncthreads();                            // everyone's
    __builtin_amdgcn_sched_barrier(0);
    step(Q, 0, x, y, std::true_type{}, P, min(s + 2, nst - 1));  // copies of stage s + 2 (the last again near the end)
  };
#pragma unroll
  for (int q = 0; q < 4; ++q) copy(P0, 0, q);
#pragma unroll
  for (int q = 0; q < 4; ++q) copy(P1, 1, q);
  __builtin_amdgcn_s_waitcnt(kWaitVmLgkm0);
  __syncthreads();
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < 4; ++g) read(P0, 0, x, g);
  for (int s = 0; s < nst; s += 2) {
    stage(P0, P1, s);
    stage(P1, P0, s + 1);
  }
  // the last MFMAs' results settle before the accumulators are read
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

__global__ void __launch_bounds__(512, 1) level_gemm_i8_kernel(int64_t m, int64_t n, int64_t kp, int S, int tiles_n,
                                                               int ntiles, int group, const int8_t* __restrict__ DA,
                                                               const int8_t* __restrict__ DBt,
                                                               int32_t* __restrict__ G, Jobs jobs, int split) {
  __shared__ __attribute__((aligned(1024))) int8_t P0[kBuf];
  __shared__ __attribute__((aligned(1024))) int8_t P1[kBuf];

  // tile order: block b runs on XCD b % 8; XCD x takes the chunk [x per, (x+1) per)
  // of an order that walks patches of `group` tile-rows column by column
  int tt = blockIdx.x;
  {
    const int per = ntiles / kXcds;
    if (tt < per * kXcds) tt = (tt % kXcds) * per + tt / kXcds;
  }
  const int tiles_m = ntiles / tiles_n;
  const int gsz = group * tiles_n, g = tt / gsz, first = g * group;
  const int rows_in = min(group, tiles_m - first), within = tt - g * gsz;
  const int64_t m0 = static_cast<int64_t>(first + within % rows_in) * kTile;
  const int64_t n0 = static_cast<int64_t>(within / rows_in) * kTile;
  const int t = jobs.t[blockIdx.y];
  const int p0 = (t - (S - 1) > 0 ? t - (S - 1) : 0) + jobs.first[blockIdx.y];
  const int64_t ld = kI8Pad + static_cast<int64_t>(S) * kp;
  int nst = static_cast<int>(jobs.count[blockIdx.y] * kp / kStage);
  const int odd = nst & 1;  // start one (zero) stage early
  nst += odd;
  const int64_t oa = kI8Pad + p0 * kp - odd * kStage, ob = kI8Pad + (S - 1 - t + p0) * kp - odd * kStage;

  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wr = wave >> 2, wc = wave & 3;
  // copies: lane L of instruction q lands at tile row 32 wave + 8q + L/8 (= 8 (q&1) + L/8
  // mod 16), granule L%8, and fetches logical granule (L%8) ^ swz(row) of that row
  const int lr = 32 * wave + (lane >> 3);
  const uint32_t lo0 = static_cast<uint32_t>(lr * ld + (((lane & 7) ^ swz(lane >> 3)) << 4));
  const uint32_t lo1 = static_cast<uint32_t>(lr * ld + (((lane & 7) ^ swz(8 + (lane >> 3))) << 4));
  // fragments: lane l reads row 16 i + l%16 of the wave's 128 rows of A (64 columns of B),
  // logical granule 4h + l/16
  int fa[2], fb[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int l = lane & 15, gl = 4 * h + (lane >> 4);
    const int sw = ((gl ^ swz(l)) << 4) + l * kStage;
    fa[h] = wr * 128 * kStage + sw;
    fb[h] = wc * 64 * kStage + sw;
  }
  v4i acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4i{0, 0, 0, 0};
  const int8_t* a = DA + m0 * ld + oa;
  const int8_t* b = DBt + n0 * ld + ob;
  tile_loop(P0, P1, a, b, static_cast<uint32_t>(kTile * ld - oa), static_cast<uint32_t>(kTile * ld - ob), nst,
            static_cast<uint32_t>(8 * ld), lo0, lo1, fa[0], fa[1], fb[0], fb[1], wave, acc);

  int32_t* o = G + static_cast<int64_t>(t) * m * n;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t gi = m0 + wr * 128 + i * 16 + 4 * (lane >> 4) + r;
        const int64_t gj = n0 + wc * 64 + j * 16 + (lane & 15);
        if (gi < m && gj < n) {
          if (split)
            atomicAdd(o + gi * n + gj, acc[i][j][r]);  // exact: the level's bound covers every partial sum
          else
            o[gi * n + gj] = acc[i][j][r];
        }
      }
}

__global__ void __launch_bounds__(256) zero_i32_kernel(int32_t* __restrict__ p, int64_t count) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = 0;
}

}  // namespace

bool level_gemm_i8_fits(int64_t kp, int S) {
  const int64_t ld = kI8Pad + static_cast<int64_t>(S) * kp;
  return S >= 1 && S <= kI8MaxSlices && kp > 0 && kp % kStage == 0 &&
         static_cast<int64_t>(kTile) * ld < (int64_t{1} << 31);
}

hipError_t launch_level_gemm_i8(int64_t m, int64_t n, int64_t kp, int S, int T, const int8_t* DA, const int8_t* DBt,
                                int32_t* G, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  if (T < 0 || T > 2 * S - 2 || !level_gemm_i8_fits(kp, S)) return hipErrorInvalidValue;
  const int64_t tiles_m = (m + kTile - 1) / kTile, tiles_n = (n + kTile - 1) / kTile;
  const int64_t ntiles = tiles_m * tiles_n;
  if (ntiles > 0x7fffffff) return hipErrorInvalidValue;
  // Jobs: every level whole, or, when the grid would hold few blocks (small
  // outputs) and every pair is an even number of stages, each level split into
  // chunks of at most c pairs that add their sums into zeroed planes; heaviest
  // first (ties in level order).
  auto pairs_of = [&](int t) {
    const int p0 = t - (S - 1) > 0 ? t - (S - 1) : 0, p1 = t < S - 1 ? t : S - 1;
    return p1 - p0 + 1;
  };
  int chunk = S;
  const bool even = (kp / kStage) % 2 == 0;
  if (even && ntiles * (T + 1) < 512) {
    chunk = (S + 1) / 2;  // halves: on c1 (1024^2, S = 15) +11%; thirds and quarters lose to the atomics
    for (;; ++chunk) {
      int njobs = 0;
      for (int t = 0; t <= T; ++t) njobs += (pairs_of(t) + chunk - 1) / chunk;
      if (njobs <= 128) break;
    }
  }
  const bool split = chunk < S;
  Jobs jobs{};
  int cnt = 0;
  for (int size = chunk; size >= 1; --size)
    for (int t = 0; t <= T; ++t)
      for (int f = 0; f < pairs_of(t); f += chunk) {
        const int c = pairs_of(t) - f < chunk ? pairs_of(t) - f : chunk;
        if (c != size) continue;
        if (cnt == 128) return hipErrorInvalidValue;
        jobs.t[cnt] = static_cast<uint8_t>(t);
        jobs.first[cnt] = static_cast<uint8_t>(f);
        jobs.count[cnt] = static_cast<uint8_t>(c);
        ++cnt;
      }
  if (!split && cnt != T + 1) return hipErrorInvalidValue;
  if (split) {
    const int64_t count = static_cast<int64_t>(T + 1) * m * n;
    const int64_t blocks = (count + 255) / 256 < 4096 ? (count + 255) / 256 : 4096;
    hipLaunchKernelGGL(zero_i32_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, G, count);
  }
  // patches of 2 tile-rows for large outputs, 4 otherwise (measured on MI355X)
  const int group = ntiles >= 1024 ? 2 : 4;
  hipLaunchKernelGGL(level_gemm_i8_kernel, dim3(static_cast<unsigned>(ntiles), static_cast<unsigned>(cnt)),
                     dim3(512), 0, stream, m, n, kp, S, static_cast<int>(tiles_n), static_cast<int>(ntiles), group,
                     DA, DBt, G, jobs, split ? 1 : 0);
  return hipGetLastError();
}

}  // namespace mdg

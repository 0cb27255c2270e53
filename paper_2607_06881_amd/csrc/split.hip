// Step a2 -- exact split of multiple doubles into 13-bit integer digits.
//
// Section 2 cuts the 52-bit fraction of a double into four 13-bit quarters
// whose exponents lie on the grid 0, -13, -26, -39; products of two quarters
// keep at least 26 trailing zero bits, so long inner products of them are
// exact.  Section 3 puts numbers that are multiplied together on one balanced
// grid and moves a unit of 2^-52 between a high and a low double of opposite
// signs so that both parts get the same sign.
//
// Here every element x (L limbs, exact value V) of a row of A or a column of B
// is read on the grid of its line's exponent E with unit u = 2^(E - w S):
//     D = floor(|V| / u),   digit_s = sign(V) * (w-bit field s of D),
// which for w = 13 are the truncated 13-bit quarters of the exact value; a limb
// of opposite sign lowers D by the floor, which is the borrow of section 3.
// Wider digits (w up to 26, the adaptive width) are the same cut with fewer,
// longer fields; the level sums stay exact while pairs k (2^w - 1)^2 < 2^53.
//
// The floor is formed exactly in 64-bit integer words: |V| / u is accumulated
// as a fixed-point integer with 52 fraction bits.  For a normalized multiple
// double every limb whose top bit is at or above u has its ulp at or above
// 2^-52 u, so those limbs add exactly; the first limb entirely below u (and
// everything after it, of smaller magnitude) only decides the floor through its
// sign, when the fraction of the accumulated part is exactly zero.  For digit
// windows of up to 256 bits (multiple doubles of up to four limbs at the
// default digits) the panel kernel uses the equivalent integer-only form
// without fraction bits (floor_on_grid_128 / _256: by nonoverlap only the first
// limb with bits below u acts below it), in 128-bit arithmetic.
//
// Two output layouts share this arithmetic: row-major digit planes (one thread
// per element, consecutive threads on consecutive columns, so limb loads and
// digit stores of a wave are contiguous 512-byte rows), and the k-major padded
// panels the level GEMM reads (see split_panel_kernel and split_tile_kernel).
#include <type_traits>

#include "digits.h"
#include "internal.h"

namespace mdg {
namespace {

// The combinations c = S .. C-1 of the Karatsuba schedule (sums of digits of
// this element, digit set masks[c] as two 32-bit words) to out[c * stride]:
// every digit of a combination carries sign(V), so a combination is sign(V)
// times the sum of the digits' w-bit fields of D, below 64 * 2^26 (exact).
template <int NW, class OutT>
__device__ inline void store_combos(const uint64_t (&I)[NW], int S, int C, int w, bool neg,
                                    const uint32_t* __restrict__ masks, OutT* __restrict__ out, int64_t stride) {
  const uint64_t fmask = (1ull << w) - 1ull;
  for (int c = S; c < C; ++c) {
    uint64_t m = static_cast<uint64_t>(masks[2 * c]) | (static_cast<uint64_t>(masks[2 * c + 1]) << 32);
    uint64_t sum = 0;
    while (m) {
      const int p = __builtin_ctzll(m);
      m &= m - 1;
      const int o = w * (S - 1 - p);  // digit p: bits o .. o + w - 1 of D
      const int wi = o >> 6, b = o & 63;
      uint64_t f = word_or_zero<NW>(I, wi) >> b;
      if (b + w > 64) f |= word_or_zero<NW>(I, wi + 1) << (64 - b);
      sum += f & fmask;
    }
    const double v = static_cast<double>(sum);  // below 2^32: exact
    out[static_cast<int64_t>(c) * stride] = static_cast<OutT>(sum == 0 ? 0.0 : (neg ? -v : v));
  }
}

// Row-major output: D [S][rows][cols], the layout of the input planes.
template <int NW, int ML>
__global__ void __launch_bounds__(256) split_kernel(int64_t rows, int64_t cols, int L, int S, int w, int axis,
                                                    const double* __restrict__ X, const int32_t* __restrict__ E,
                                                    double* __restrict__ D) {
  const int64_t plane = rows * cols;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const int64_t idx = r * cols + c;
    const int e = axis == 0 ? E[r] : E[c];
    double xs[ML];
    load_limbs<ML>(X, plane, L, idx, xs);
    uint64_t I[NW];
    const bool neg = floor_on_grid<NW, ML>(xs, L, e - w * S, I);
    store_digits<NW, double>(I, S, w, neg, D + idx, plane);
  }
}

// Panel output for the level GEMM: both operands k-major and padded,
//   axis 0 (A, rows = m, cols = k):  D [S][kp][mp],  D[s][kk][i] = digit s of A[i][kk]
//   axis 1 (B, rows = k, cols = n):  D [S][kp][np],  D[s][kk][j] = digit s of B[kk][j]
// with kp, mp, np rounded up to the GEMM tile (16 and 128) and zeros in the padding.
// A block covers 64 lines (c) x 4 RPT k, each thread RPT elements of one line:
// with RPT = 4 its reads of A touch 64 full 128-byte lines; RPT = 1 gives four
// times the blocks for panels too small to fill the GPU otherwise (the split of
// a long multiple double is integer work, bound by latency at low occupancy).
// Stores are rows of 64 consecutive panel values.
// With C > S, panels S .. C-1 receive the combinations of the Karatsuba
// schedule (store_combos), computed from the same integer as the digits.
// OutT = float for FP32 panels (the host checks that every value is below 2^24,
// so the conversion is exact; kp is then a multiple of 32).
template <int NW, int ML, class OutT, int RPT>
__global__ void __launch_bounds__(256) split_panel_kernel(int64_t rows, int64_t cols, int L, int S, int w, int axis,
                                                          int64_t kp, int64_t cp, const double* __restrict__ X,
                                                          const int32_t* __restrict__ E, OutT* __restrict__ D,
                                                          const uint32_t* __restrict__ masks, int C) {
  const int64_t plane = rows * cols, pplane = kp * cp;
  const int64_t K = axis == 0 ? cols : rows;   // reduction length
  const int64_t Cn = axis == 0 ? rows : cols;  // lines (rows of A or columns of B)
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 64 + (threadIdx.x & 63);
  if (c >= cp) return;
  const int64_t cc = c < Cn ? c : 0;  // clamped line for the unconditional loads
  const int e = E[cc];
  // the limbs of kBatch of this thread's RPT elements are loaded before any of
  // them is split (fewer at a time for long multiple doubles, to stay in registers)
  constexpr int kBatchL = ML <= 4 ? 4 : (ML <= 8 ? 2 : 1);
  constexpr int kBatch = kBatchL < RPT ? kBatchL : RPT;
  constexpr int kRows = 4 * RPT;  // k rows per block
  for (int64_t kb = blockIdx.y; kb * kRows < kp; kb += gridDim.y) {
#pragma unroll
    for (int r0 = 0; r0 < RPT; r0 += kBatch) {
      double xs[kBatch][ML];
      bool valid[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int64_t kk = kb * kRows + (threadIdx.x >> 6) + 4 * (r0 + b);
        valid[b] = c < Cn && kk < K;
        const int64_t kc = kk < K ? kk : 0;
        load_limbs<ML>(X, plane, L, axis == 0 ? cc * cols + kc : kc * cols + cc, xs[b]);
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int64_t kk = kb * kRows + (threadIdx.x >> 6) + 4 * (r0 + b);
        OutT* out = D + kk * cp + c;
        if (valid[b]) {
          uint64_t I[NW];
          const bool neg = floor_on_grid<NW, ML>(xs[b], L, e - w * S, I);
          store_digits<NW, OutT>(I, S, w, neg, out, pplane);
          if (C > S) store_combos<NW, OutT>(I, S, C, w, neg, masks, out, pplane);
        } else {
          for (int s = 0; s < (C > S ? C : S); ++s) out[static_cast<int64_t>(s) * pplane] = OutT(0);
        }
      }
    }
  }
}

// The panel layout of split_panel_kernel for multiple doubles of up to four
// limbs, by tiles of 64 lines x 16 k values; a block takes the tiles of its 64
// lines at k steps of gridDim.y tiles (up to four), each in two phases:
//  - load: the tile's limbs go through LDS, so that every global load of a wave
//    reads whole 128-byte lines whichever operand it is (A's lines are rows, 16
//    consecutive k values of a row per 16 lanes; B's lines are columns, 64
//    consecutive columns per wave), the padding positions loading +0.0; the
//    next tile's loads are issued before the current tile is split;
//  - split: each thread takes 4 consecutive lines of one k value, so that every
//    digit store is one 16-byte vector (a wave writes 256 bytes of each of four
//    FP32 panel rows).
// kFast selects floor_on_grid_128 (digit windows w S <= 128, NW = 2) or
// floor_on_grid_256 (w S <= 256, NW = 4); otherwise floor_on_grid with NW
// words.  The digit fields are read upward from bit 0 in a two-word window as
// in store_digits; the window position is the same for all four elements (and
// all lanes), so only the words differ.
constexpr int kTileLines = 64, kTileK = 16, kTilePitch = kTileLines + 4;  // LDS row pitch in doubles

__host__ __device__ constexpr size_t split_tile_lds(int L) {
  return sizeof(double) * static_cast<size_t>(L) * kTileK * kTilePitch;
}

template <class OutT>
__device__ inline OutT digit_value(uint64_t f, uint64_t mask, bool neg);
template <>
__device__ inline float digit_value<float>(uint64_t f, uint64_t mask, bool neg) {
  const uint32_t d = static_cast<uint32_t>(f & mask);  // below 2^24 for FP32 panels: exact
  const uint32_t b = __float_as_uint(static_cast<float>(d));
  return __uint_as_float(b | ((neg && d) ? 0x80000000u : 0u));  // zero digits are +0.0
}
template <>
__device__ inline double digit_value<double>(uint64_t f, uint64_t mask, bool neg) {
  return signed_digit(static_cast<uint32_t>(f & mask), neg);
}

__device__ inline void store4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ inline void store4(double* p, const double (&v)[4]) {
  reinterpret_cast<double2*>(p)[0] = make_double2(v[0], v[1]);
  reinterpret_cast<double2*>(p)[1] = make_double2(v[2], v[3]);
}

template <int NW, int ML, class OutT, bool kFast>
__global__ void __launch_bounds__(256) split_tile_kernel(int64_t rows, int64_t cols, int L, int S, int w, int axis,
                                                         int64_t kp, int64_t cp, const double* __restrict__ X,
                                                         const int32_t* __restrict__ E, OutT* __restrict__ D) {
  static_assert(!kFast || NW == 2 || NW == 4, "the fast floors fill two or four words");
  extern __shared__ double tile[];  // [L][kTileK][kTilePitch]
  const int64_t plane = rows * cols, pplane = kp * cp;
  const int64_t K = axis == 0 ? cols : rows;   // reduction length
  const int64_t Cn = axis == 0 ? rows : cols;  // lines
  const int t = threadIdx.x;
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kTileLines;
  const int qk = t >> 4, qc = 4 * (t & 15);  // split phase: lines qc .. qc + 3 of k row qk
  int e[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) e[i] = c0 + qc + i < Cn ? E[c0 + qc + i] : 0;
  const uint64_t mask = (1ull << w) - 1ull;
  // load-phase positions (fixed per thread) and the tile's limbs in registers
  int lk[4], lc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    lk[i] = axis == 0 ? (t & 15) : (t >> 6) + 4 * i;
    lc[i] = axis == 0 ? (t >> 4) + 16 * i : (t & 63);
  }
  double v[ML][4];
  auto load_tile = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t c = c0 + lc[i], kk = k0 + lk[i];
      const bool ok = c < Cn && kk < K;
      const int64_t idx = ok ? (axis == 0 ? c * cols + kk : kk * cols + c) : 0;
#pragma unroll
      for (int l = 0; l < ML; ++l) v[l][i] = (ok && l < L) ? X[static_cast<int64_t>(l) * plane + idx] : 0.0;
    }
  };
  int64_t kb = blockIdx.y;
  if (kb * kTileK < kp) load_tile(kb * kTileK);
  for (; kb * kTileK < kp; kb += gridDim.y) {
    const int64_t k0 = kb * kTileK;
    __syncthreads();  // the previous tile's readers are done
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int l = 0; l < ML; ++l)
        if (l < L) tile[(l * kTileK + lk[i]) * kTilePitch + lc[i]] = v[l][i];
    __syncthreads();
    if ((kb + gridDim.y) * kTileK < kp) load_tile((kb + gridDim.y) * kTileK);
    uint64_t I[4][NW];
    bool neg[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      double xs[ML];
#pragma unroll
      for (int l = 0; l < ML; ++l) xs[l] = l < L ? tile[(l * kTileK + qk) * kTilePitch + qc + i] : 0.0;
      if constexpr (kFast && NW == 2)
        neg[i] = floor_on_grid_128<ML>(xs, L, e[i] - w * S, I[i]);
      else if constexpr (kFast)
        neg[i] = floor_on_grid_256<ML>(xs, L, e[i] - w * S, I[i]);
      else
        neg[i] = floor_on_grid<NW, ML>(xs, L, e[i] - w * S, I[i]);
    }
    OutT* out = D + (k0 + qk) * cp + c0 + qc + static_cast<int64_t>(S - 1) * pplane;
    uint64_t cur[4], nxt[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      cur[i] = I[i][0];
      nxt[i] = NW > 1 ? I[i][1] : 0ull;
    }
    int b = 0, wi = 0;  // the window: word wi of every I, next unread bit b
    for (int j = 0; j < S; ++j) {
      OutT d[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint64_t f = cur[i] >> b;
        if (b + w > 64) f |= nxt[i] << (64 - b);
        d[i] = digit_value<OutT>(f, mask, neg[i]);
      }
      store4(out - static_cast<int64_t>(j) * pplane, d);
      b += w;
      if (b >= 64) {
        b -= 64;
        ++wi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cur[i] = nxt[i];
          nxt[i] = word_or_zero<NW>(I[i], wi + 1);
        }
      }
    }
  }
}

// A's digits for the int8 level products (digits of at most 7 bits), rows of
// pitch kI8Pad + S kp: D[i][kI8Pad + s kp + kk] = digit s of A[i][kk], zeros for
// kk >= k and in the first kI8Pad bytes.  A level's pairs (p, t - p), p
// ascending, are then one contiguous k range of every row.  One thread per
// element of the padded grid [m][kp], consecutive threads on consecutive kk:
// limb loads and digit stores of a wave are contiguous.
template <int NW, int ML>
__global__ void __launch_bounds__(256) split_int8_kernel(int64_t rows, int64_t cols, int64_t kp, int L, int S, int w,
                                                         const double* __restrict__ X,
                                                         const int32_t* __restrict__ E, int8_t* __restrict__ D) {
  const int64_t plane = rows * cols;
  const int64_t ld = kI8Pad + static_cast<int64_t>(S) * kp;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (c >= kp) return;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    int8_t* row = D + r * ld;
    if (c < kI8Pad) row[c] = 0;
    int8_t* out = row + kI8Pad + c;
    if (c < cols) {
      double xs[ML];
      load_limbs<ML>(X, plane, L, r * cols + c, xs);
      uint64_t I[NW];
      const bool neg = floor_on_grid<NW, ML>(xs, L, E[r] - w * S, I);
      store_digits<NW, int8_t>(I, S, w, neg, out, kp);
    } else {
      for (int q = 0; q < S; ++q) out[static_cast<int64_t>(q) * kp] = 0;
    }
  }
}

// B's int8 digits straight into the k-contiguous layout of the int8 level
// products, rows of pitch kI8Pad + S kp: Dt[j][kI8Pad + (S-1-q) kp + kk] = digit q
// of B[kk][j], zeros for j >= n, kk >= k and in the first kI8Pad bytes.  Lanes
// take consecutive kk, so every digit store of a wave is 64
// contiguous bytes; a block covers 64 kk x 16 columns (each wave 4 columns), so
// the 16 consecutive doubles of a row of B that one 128-byte line holds are all
// read by the same block.
template <int NW, int ML>
__global__ void __launch_bounds__(256) split_int8t_kernel(int64_t rows, int64_t cols, int64_t kp, int64_t np, int L,
                                                          int S, int w, const double* __restrict__ X,
                                                          const int32_t* __restrict__ E, int8_t* __restrict__ Dt) {
  const int64_t plane = rows * cols;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t ld = kI8Pad + static_cast<int64_t>(S) * kp;
  for (int64_t by = blockIdx.y; by * 16 < np; by += gridDim.y) {
    const int64_t kk = static_cast<int64_t>(blockIdx.x) * 64 + lane;
    if (kk >= kp) continue;
#pragma unroll 1
    for (int r = 0; r < 4; ++r) {
      const int64_t j = by * 16 + 4 * wave + r;
      if (j >= np) break;
      if (kk < kI8Pad) Dt[j * ld + kk] = 0;
      int8_t* out = Dt + j * ld + kI8Pad + static_cast<int64_t>(S - 1) * kp + kk;
      if (kk < rows && j < cols) {
        double xs[ML];
        load_limbs<ML>(X, plane, L, kk * cols + j, xs);
        uint64_t I[NW];
        const bool neg = floor_on_grid<NW, ML>(xs, L, E[j] - w * S, I);
        store_digits<NW, int8_t>(I, S, w, neg, out, -kp);
      } else {
        for (int q = 0; q < S; ++q) out[-static_cast<int64_t>(q) * kp] = 0;
      }
    }
  }
}

// Grouped panels (section 3: numbers grouped by sign and by the exponent of
// their leading part, each group multiplied separately).  Every element belongs
// to one of G = (sign ? 2 : 1) Ge groups: exponent class c = 0 for a zero
// element, else min(Ge - 1, floor((E - e) / w)) where e is the frexp exponent of
// its leading limb (the class of elements whose leading digit falls c digits
// below the line's grid), and sign group 1 for a negative element with sign
// grouping, else 0; g = sign group * Ge + c.  Its S digits are taken on the
// class grid E - c w (so the element keeps its leading bits) and written to
// panels g S .. g S + S - 1; the S digits of the other G - 1 groups are zero.
// (e <= E - c w, so |V| < 2^(E - c w): the split's precondition holds.)
// One element per thread, the panel layout of split_panel_kernel.
template <int NW, int ML, class OutT>
__global__ void __launch_bounds__(256) split_groups_kernel(int64_t rows, int64_t cols, int L, int S, int w, int axis,
                                                           int64_t kp, int64_t cp, int Ge, int G,
                                                           const double* __restrict__ X,
                                                           const int32_t* __restrict__ E, OutT* __restrict__ D) {
  const int64_t plane = rows * cols, pplane = kp * cp;
  const int64_t K = axis == 0 ? cols : rows;
  const int64_t Cn = axis == 0 ? rows : cols;
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 64 + (threadIdx.x & 63);
  if (c >= cp) return;
  const int64_t cc = c < Cn ? c : 0;
  const int e = E[cc];
  for (int64_t kb = blockIdx.y; kb * 4 < kp; kb += gridDim.y) {
    const int64_t kk = kb * 4 + (threadIdx.x >> 6);
    OutT* out = D + kk * cp + c;
    const bool valid = c < Cn && kk < K;
    const int64_t kc = kk < K ? kk : 0;
    double xs[ML];
    load_limbs<ML>(X, plane, valid ? L : 0, axis == 0 ? cc * cols + kc : kc * cols + cc, xs);
    int g = 0, cls = 0;
    if (xs[0] != 0.0) {
      const int fe = frexp_exp_or_min(xs[0]);
      cls = (e - fe) / w;
      cls = cls < Ge - 1 ? cls : Ge - 1;
      g = (G > Ge && xs[0] < 0.0 ? Ge : 0) + cls;
    }
    uint64_t I[NW];
    const bool neg = floor_on_grid<NW, ML>(xs, L, e - cls * w - w * S, I);
    for (int h = 0; h < G; ++h) {
      OutT* o = out + static_cast<int64_t>(h) * S * pplane;
      if (h == g) {
        store_digits<NW, OutT>(I, S, w, neg, o, pplane);
      } else {
        for (int q = 0; q < S; ++q) o[static_cast<int64_t>(q) * pplane] = OutT(0);
      }
    }
  }
}

template <int NW, int ML>
hipError_t launch_nw(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X, const int32_t* E,
                     void* D, bool panel, bool f32, const uint32_t* masks, int C, hipStream_t stream) {
  if (!panel) {
    const unsigned gx = static_cast<unsigned>((cols + 255) / 256);
    const unsigned gy = static_cast<unsigned>(rows < 65535 ? rows : 65535);
    hipLaunchKernelGGL((split_kernel<NW, ML>), dim3(gx, gy), dim3(256), 0, stream, rows, cols, L, S, w, axis, X, E,
                       static_cast<double*>(D));
    return hipGetLastError();
  }
  const int64_t K = axis == 0 ? cols : rows, Cn = axis == 0 ? rows : cols;
  const int64_t kp = f32 ? panel_k32(K) : panel_k(K), cp = panel_mn(Cn);
  const unsigned gx = static_cast<unsigned>(cp / 64);
  // four elements per thread while that still gives 2048 blocks (8 per CU),
  // one per thread below (kp is a multiple of 16)
  const bool wide = (cp / 64) * (kp / 16) >= 2048;
  const int64_t nkb = kp / (wide ? 16 : 4);
  const unsigned gy = static_cast<unsigned>(nkb < 65535 ? nkb : 65535);
  const dim3 grid(gx, gy);
  if constexpr (ML == 4) {
    // tiles of 64 lines x 16 k through LDS, 16-byte digit stores (the panel base
    // must be 16-byte aligned; kp is a multiple of 16 and cp of 64)
    if (wide && C == S && (reinterpret_cast<uintptr_t>(D) & 15u) == 0) {
      const size_t lds = split_tile_lds(L);
      // up to four tiles per block (each block's next loads overlap its split)
      // while at least 2048 blocks remain
      int64_t tiles = kp / kTileK, per = 1;
      while (per < 4 && gx * ((tiles + 2 * per - 1) / (2 * per)) >= 2048) per *= 2;
      const int64_t gyt = (tiles + per - 1) / per;
      const dim3 grid(gx, static_cast<unsigned>(gyt < 65535 ? gyt : 65535));
      auto go = [&](auto kernel, auto* out) {
        hipLaunchKernelGGL(kernel, grid, dim3(256), lds, stream, rows, cols, L, S, w, axis, kp, cp, X, E, out);
        return hipGetLastError();
      };
      const int bits = w * S;
      if (f32) {
        float* out = static_cast<float*>(D);
        if (bits <= 128) return go(split_tile_kernel<2, 4, float, true>, out);
        if (bits <= 256) return go(split_tile_kernel<4, 4, float, true>, out);
        return go(split_tile_kernel<NW, 4, float, false>, out);
      }
      double* out = static_cast<double*>(D);
      if (bits <= 128) return go(split_tile_kernel<2, 4, double, true>, out);
      if (bits <= 256) return go(split_tile_kernel<4, 4, double, true>, out);
      return go(split_tile_kernel<NW, 4, double, false>, out);
    }
  }
  if (f32) {
    if (wide)
      hipLaunchKernelGGL((split_panel_kernel<NW, ML, float, 4>), grid, dim3(256), 0, stream, rows, cols, L, S, w, axis,
                         kp, cp, X, E, static_cast<float*>(D), masks, C);
    else
      hipLaunchKernelGGL((split_panel_kernel<NW, ML, float, 1>), grid, dim3(256), 0, stream, rows, cols, L, S, w, axis,
                         kp, cp, X, E, static_cast<float*>(D), masks, C);
  } else {
    if (wide)
      hipLaunchKernelGGL((split_panel_kernel<NW, ML, double, 4>), grid, dim3(256), 0, stream, rows, cols, L, S, w,
                         axis, kp, cp, X, E, static_cast<double*>(D), masks, C);
    else
      hipLaunchKernelGGL((split_panel_kernel<NW, ML, double, 1>), grid, dim3(256), 0, stream, rows, cols, L, S, w,
                         axis, kp, cp, X, E, static_cast<double*>(D), masks, C);
  }
  return hipGetLastError();
}

// Word counts instantiated for w S up to 908 digit bits (960 bits).
template <int ML>
hipError_t split_words(int words, int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X,
                       const int32_t* E, void* D, bool panel, bool f32, const uint32_t* masks, int C,
                       hipStream_t stream) {
  if (words <= 2) return launch_nw<2, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 3) return launch_nw<3, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 4) return launch_nw<4, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 5) return launch_nw<5, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 6) return launch_nw<6, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 8) return launch_nw<8, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 10) return launch_nw<10, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 14) return launch_nw<14, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (words <= 15) return launch_nw<15, ML>(rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  return hipErrorInvalidValue;
}

template <int ML>
hipError_t split_int8t_words(int words, int64_t rows, int64_t cols, int64_t kp, int64_t np, int L, int S, int w,
                             const double* X, const int32_t* E, int8_t* Dt, hipStream_t stream) {
  const int64_t gy = (np + 15) / 16;
  const dim3 grid(static_cast<unsigned>((kp + 63) / 64), static_cast<unsigned>(gy < 65535 ? gy : 65535));
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, rows, cols, kp, np, L, S, w, X, E, Dt);
    return hipGetLastError();
  };
  if (words <= 2) return go(split_int8t_kernel<2, ML>);
  if (words <= 3) return go(split_int8t_kernel<3, ML>);
  if (words <= 4) return go(split_int8t_kernel<4, ML>);
  if (words <= 6) return go(split_int8t_kernel<6, ML>);
  if (words <= 8) return go(split_int8t_kernel<8, ML>);
  return hipErrorInvalidValue;
}

template <int ML>
hipError_t split_int8_words(int words, int64_t rows, int64_t cols, int64_t kp, int L, int S, int w, const double* X,
                            const int32_t* E, int8_t* D, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>((kp + 255) / 256), static_cast<unsigned>(rows < 65535 ? rows : 65535));
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid, dim3(256), 0, stream, rows, cols, kp, L, S, w, X, E, D);
    return hipGetLastError();
  };
  // w <= 7 and S <= 64: w S + 52 <= 500 bits, at most 8 words
  if (words <= 2) return go(split_int8_kernel<2, ML>);
  if (words <= 3) return go(split_int8_kernel<3, ML>);
  if (words <= 4) return go(split_int8_kernel<4, ML>);
  if (words <= 6) return go(split_int8_kernel<6, ML>);
  if (words <= 8) return go(split_int8_kernel<8, ML>);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_split(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X, const int32_t* E,
                        void* D, bool panel, hipStream_t stream, const uint32_t* masks, int combos, bool f32) {
  if (f32 && !panel) return hipErrorInvalidValue;
  const int C = (panel && masks && combos > S) ? combos : S;
  if (rows == 0 || cols == 0) return hipSuccess;
  // The accumulator holds |V| / u < 2^(w S) with 52 fraction bits: w S + 52 bits,
  // in the next word count instantiated (extra words stay zero).
  const int words = (w * S + 52 + 63) / 64;
  if (L <= 4) return split_words<4>(words, rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  if (L <= 8) return split_words<8>(words, rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
  return split_words<16>(words, rows, cols, L, S, w, axis, X, E, D, panel, f32, masks, C, stream);
}

hipError_t launch_split_groups(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X,
                               const int32_t* E, void* D, bool f32, int Ge, bool sign, hipStream_t stream) {
  if (L < 1 || L > 4 || Ge < 1 || (w * S + 52 + 63) / 64 > kGroupSplitWords) return hipErrorInvalidValue;
  if (rows == 0 || cols == 0) return hipSuccess;
  const int G = (sign ? 2 : 1) * Ge;
  const int64_t K = axis == 0 ? cols : rows, Cn = axis == 0 ? rows : cols;
  const int64_t kp = f32 ? panel_k32(K) : panel_k(K), cp = panel_mn(Cn);
  const int64_t nkb = kp / 4;
  const dim3 grid(static_cast<unsigned>(cp / 64), static_cast<unsigned>(nkb < 65535 ? nkb : 65535));
  if (f32)
    hipLaunchKernelGGL((split_groups_kernel<kGroupSplitWords, 4, float>), grid, dim3(256), 0, stream, rows, cols, L, S,
                       w, axis, kp, cp, Ge, G, X, E, static_cast<float*>(D));
  else
    hipLaunchKernelGGL((split_groups_kernel<kGroupSplitWords, 4, double>), grid, dim3(256), 0, stream, rows, cols, L,
                       S, w, axis, kp, cp, Ge, G, X, E, static_cast<double*>(D));
  return hipGetLastError();
}

hipError_t launch_split_int8(int64_t rows, int64_t cols, int L, int S, int w, const double* X, const int32_t* E,
                             int8_t* D, int64_t kp, hipStream_t stream) {
  if (w < 1 || w > 7 || S < 1 || S > kI8MaxSlices || kp < cols || kp % kI8Pad != 0) return hipErrorInvalidValue;
  if (rows == 0 || kp == 0) return hipSuccess;
  const int words = (w * S + 52 + 63) / 64;
  if (L <= 4) return split_int8_words<4>(words, rows, cols, kp, L, S, w, X, E, D, stream);
  if (L <= 8) return split_int8_words<8>(words, rows, cols, kp, L, S, w, X, E, D, stream);
  return split_int8_words<16>(words, rows, cols, kp, L, S, w, X, E, D, stream);
}

hipError_t launch_split_int8t(int64_t rows, int64_t cols, int L, int S, int w, const double* X, const int32_t* E,
                              int8_t* Dt, int64_t kp, int64_t np, hipStream_t stream) {
  if (w < 1 || w > 7 || S < 1 || S > kI8MaxSlices || kp < rows || np < cols || kp % kI8Pad != 0)
    return hipErrorInvalidValue;
  if (kp == 0 || np == 0) return hipSuccess;
  const int words = (w * S + 52 + 63) / 64;
  if (L <= 4) return split_int8t_words<4>(words, rows, cols, kp, np, L, S, w, X, E, Dt, stream);
  if (L <= 8) return split_int8t_words<8>(words, rows, cols, kp, np, L, S, w, X, E, Dt, stream);
  return split_int8t_words<16>(words, rows, cols, kp, np, L, S, w, X, E, Dt, stream);
}

}  // namespace mdg

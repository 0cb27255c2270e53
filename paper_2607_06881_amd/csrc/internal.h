// Internal launch interface shared by the HIP translation units of libmdgemm.
// Every launcher enqueues its kernels on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "schedule.h"

namespace mdg {

constexpr int kSliceBits = 13;
constexpr int kDigitMax = (1 << kSliceBits) - 1;  // 8191
constexpr int kMaxSlices = 68;  // the 66 default digits of a hexa double, and a little room
constexpr int kMaxLimbs = 16;   // hexa double
constexpr int kMaxLevels = 2 * kMaxSlices - 1;
constexpr int kZWords = 28;     // 64-bit words of an exact level sum (w (levels - 1) + 55 bits <= 1792)
constexpr int kMaxJobs = 65535;  // jobs of one level-GEMM launch (grid.y)
constexpr int kMaxSliceBits = 26;                  // widest digit: products of two stay below 2^52
constexpr int kMaxDigitBits = 64 * 15 - 52;  // w S + 52 <= 960: the split's integer fits 15 words
constexpr int kTileMN = 128;  // level-GEMM tile rows / columns
constexpr int kTileK = 16;    // level-GEMM k step

// Panel dimensions of the level-GEMM operands: k rounded up to the k step,
// m / n rounded up to the tile.
inline int64_t panel_k(int64_t k) { return (k + kTileK - 1) / kTileK * kTileK; }
// FP32 panels (every digit and digit sum below 2^24) use 32-deep k steps.
constexpr int kTileK32 = 32;
// Word 3 of the raw buffer descriptors of the buffer-to-LDS copies (the level
// GEMM kernels): the DATA_FORMAT field (bits 15-18) set to 4, 32-bit elements.
constexpr int kBufferWord3 = 0x00020000;
inline int64_t panel_k32(int64_t k) { return (k + kTileK32 - 1) / kTileK32 * kTileK32; }
inline int64_t panel_mn(int64_t x) { return (x + kTileMN - 1) / kTileMN * kTileMN; }

// Slice-pair jobs of the level GEMM, read from a device table in the format of
// ScheduleTable (schedule.h): `jobs` holds three words per job (first pair |
// pair count << 16, output plane, k chunk | k chunks << 16), `pairs` one word
// per pair (combination of A | combination of B << 16).  Job j sums the
// products of its pairs over its k chunk into plane out[j].
struct GemmJobs {
  const uint32_t* jobs = nullptr;
  const uint32_t* pairs = nullptr;
  int njobs = 0;
};

// a1: per-row (axis 0) or per-column (axis 1) grid exponents of a [rows][cols] plane.
// MDGEMM_LOG (environment, read once): 0 or unset, silent; 1, one stderr line per
// call of mdgemm_ex, mdgemm_ex_noalloc and mdgemm_qr_dd; 2, also the products a
// QR makes.  log_depth is the nesting of the calling thread (the QR raises it).
int log_level();
extern thread_local int log_depth;
void log_line(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

hipError_t launch_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, hipStream_t stream);
// The exponents of A's rows (EA) and of B's columns (EB) in one pass over both
// leading limbs; scratch (cy n int32 partial maxima, cy <= ceil(k / 64)) is
// device memory that is free until the pass ends (too small: the two launches above).
hipError_t launch_exponents_ab(int64_t m, int64_t k, int64_t n, const double* A0, const double* B0, int32_t* EA,
                               int32_t* EB, void* scratch, size_t scratch_bytes, hipStream_t stream);

// Exponent spread of every line: E as launch_exponents, spread = E - (smallest
// frexp exponent of a nonzero entry of the line), 0 for an all-zero line.
hipError_t launch_line_spread(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, int32_t* spread,
                              hipStream_t stream);

// a2: w-bit digits of X [L][rows][cols] on the grid exponents E, either row-major
// D [S][rows][cols] (panel == false) or as a level-GEMM panel (panel == true):
// axis 0: D [S][panel_k(cols)][panel_mn(rows)] (transposed), axis 1:
// D [S][panel_k(rows)][panel_mn(cols)], zeros in the padding.
// With panel == true and masks (the schedule's combination digit sets, two
// words per combination, in device memory) and combos > S, panels S .. combos-1
// receive the schedule's combinations (sums of digits) as well.  D is double*,
// or float* with f32 (panels only: panel_k32 rows, every value below 2^24).
hipError_t launch_split(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X, const int32_t* E,
                        void* D, bool panel, hipStream_t stream, const uint32_t* masks = nullptr,
                        int combos = 0, bool f32 = false);

// a2 for grouped products (section 3's grouping by sign and by exponent class):
// panels as launch_split (panel == true), G = (sign ? 2 : 1) Ge groups of S
// panels each; element in group g = sign group * Ge + class, class c =
// min(Ge - 1, floor((E - e) / w)) (e: the frexp exponent of its leading limb, 0
// for a zero element), split on the grid E - c w into panels g S .. g S + S - 1,
// zeros in the other groups' panels.  Up to 4 limbs and w S + 52 <= 384 bits.
constexpr int kGroupSplitWords = 6;
hipError_t launch_split_groups(int64_t rows, int64_t cols, int L, int S, int w, int axis, const double* X,
                               const int32_t* E, void* D, bool f32, int Ge, bool sign, hipStream_t stream);

// Layout of the int8 digits: rows of pitch kI8Pad + S kp bytes (kp = k rounded
// up to 128), the first kI8Pad bytes of every row zero, A's rows m rounded up to
// 256, B's (columns of B) n rounded up to 256 (those extra rows are never
// stored and only feed outputs that are not kept).
constexpr int kI8Pad = 128;
constexpr int kI8MaxSlices = 64;  // int8 digits per element (w S + 52 <= 500 bits at w <= 7)
inline int64_t i8_kp(int64_t k) { return (k + 127) / 128 * 128; }
inline int64_t i8_rows(int64_t x) { return (x + 255) / 256 * 256; }

// a2 for the int8 level products: A's digits (at most 7 bits) as int8,
// D[i][kI8Pad + s kp + kk] = digit s of A[i][kk] (rows = m, cols = k), zeros for
// kk >= k and in the pad.
hipError_t launch_split_int8(int64_t rows, int64_t cols, int L, int S, int w, const double* X, const int32_t* E,
                             int8_t* D, int64_t kp, hipStream_t stream);

// a2 for the int8 level products, B (rows = k, cols = n) straight into the
// k-contiguous layout: Dt[j][kI8Pad + (S-1-q) kp + kk] = digit q of B[kk][j], for
// the np rows j (zeros for j >= n, kk >= k and in the pad).
hipError_t launch_split_int8t(int64_t rows, int64_t cols, int L, int S, int w, const double* X, const int32_t* E,
                              int8_t* Dt, int64_t kp, int64_t np, hipStream_t stream);

// a3 on the int8 matrix cores: levels t = 0..T into int32 planes G [T+1][m][n],
// from A's digits (launch_split_int8, i8_rows(m) rows) and B's (launch_split_int8t,
// i8_rows(n) rows), all levels in one launch of the hand-written kernel of
// level_gemm_i8.hip; every level sum must stay below 2^31 (checked by the caller).
// level_gemm_i8_fits tells whether a digit layout fits that kernel.
bool level_gemm_i8_fits(int64_t kp, int S);
hipError_t launch_level_gemm_i8(int64_t m, int64_t n, int64_t kp, int S, int T, const int8_t* DA, const int8_t* DBt,
                                int32_t* G, hipStream_t stream);

// a3: products of the combination panels DAt [*][panel_k(k)][panel_mn(m)] and
// DBp [*][panel_k(k)][panel_mn(n)] (combinations 0..S-1 are the digits); one
// job per grid row, outputs [*][m][n].
hipError_t launch_slice_gemm(int64_t m, int64_t n, int64_t k, const double* DAt, const double* DBp, double* out,
                             const GemmJobs& jobs, hipStream_t stream);

// a3 on FP32 panels DAt [*][panel_k32(k)][panel_mn(m)], DBp [*][panel_k32(k)][panel_mn(n)]
// whose values are integers below 2^24 (exact in FP32); same jobs and outputs.
hipError_t launch_slice_gemm32(int64_t m, int64_t n, int64_t k, const float* DAt, const float* DBp, double* out,
                               const GemmJobs& jobs, hipStream_t stream);

// The fused small-product kernel (small_product.hip): one block per 16 x 16
// tile of C runs all five steps.  Limits: up to 4 limbs, digits below 2^24
// (held in LDS as FP32), w S + 52 <= 320 bits
// (the split's integer in 5 words), w T + 55 <= 448 bits (the level sum in 7
// words), up to 32 levels; its dynamic LDS holds the levels of the tile and the
// digits of one k chunk of kc (a multiple of 4).  wave[t] is the wave (0..7)
// that forms level t; waves w and w + 4 share a SIMD.
constexpr int kSmallWaves = 8;
constexpr int kSmallMaxLimbs = 4;
constexpr int kSmallSplitWords = 5;
constexpr int kSmallAccumWords = 7;
constexpr int kSmallMaxLevels = 32;
constexpr size_t kSmallMaxLds = 150 * 1024;
struct SmallLevelOwners {
  int8_t wave[kSmallMaxLevels];
};
size_t small_product_lds(int S, int T, int kc);
hipError_t launch_small_product(int64_t m, int64_t n, int64_t k, int L, int S, int T, int w, int kc,
                                const SmallLevelOwners& owners, const double* A, const double* B, double* C,
                                hipStream_t stream);

// Copies `words` into the device array dst (stream-ordered kernel launches that
// carry the words as arguments, so that no host memory is read later).
hipError_t launch_upload(const std::vector<uint32_t>& words, uint32_t* dst, hipStream_t stream);

// The combinations c >= S of one operand (mask/parents of the schedule, `a`
// selects A's or B's): panel c = panel par1[c] + panel par2[c], whole panels of
// `plane` doubles, in order of depth.
hipError_t launch_combinations(const Schedule& s, bool a, double* D, int64_t plane, hipStream_t stream);
hipError_t launch_combinations32(const Schedule& s, bool a, float* D, int64_t plane, hipStream_t stream);

// FP64 panels [S][kp_src][cp] -> FP32 panels [S][kp_dst][cp], rows kp_src .. kp_dst-1
// zero; every value an integer below 2^24.
hipError_t launch_panel_to_f32(const double* src, float* dst, int64_t kp_src, int64_t kp_dst, int64_t cp, int S,
                               hipStream_t stream);

// a4: exact accumulation of `levels` planes of w-bit digit products (weights
// 2^(-w t)) into kZWords-word integers Z [kZWords][m][n].
hipError_t launch_accumulate(int64_t m, int64_t n, int levels, int w, const double* G, int64_t* Z,
                             hipStream_t stream);

// a4 + a5: exact accumulation and greedy rounding into L limbs, scaled by 2^(EA+EB-2w).
hipError_t launch_accum_renorm(int64_t m, int64_t n, int L, int levels, int w, const double* G, const int32_t* EA,
                               const int32_t* EB, double* C, hipStream_t stream);

// a4 + a5 from int32 level planes (the int8 level products).
hipError_t launch_accum_renorm_i32(int64_t m, int64_t n, int L, int levels, int w, const int32_t* G,
                                   const int32_t* EA, const int32_t* EB, double* C, hipStream_t stream);

// a4 + a5 for a schedule whose planes enter several levels: level t =
// sum of coef * plane over the entries (chunk_first / chunks of ScheduleTable;
// chunks 8-byte aligned), formed exactly in 64-bit integers, then accumulated
// and rounded as launch_accum_renorm (C != nullptr), or written as
// integer-valued doubles Gout [levels][m][n] (C == nullptr).
hipError_t launch_plan_accum(int64_t m, int64_t n, int L, int levels, int w, int planes, const double* P,
                             const uint32_t* chunk_first, const uint32_t* chunks, const int32_t* EA,
                             const int32_t* EB, double* C, double* Gout, hipStream_t stream);

// 64-bit words of the exact sum of `levels` levels of w-bit digits (sign included).
int accum_words(int levels, int w);

// Utilities: fill `count` doubles with +0.0; zero/set a device flag; scan for inf/nan.
hipError_t launch_zero_f64(double* p, int64_t count, hipStream_t stream);
hipError_t launch_nonfinite_scan(const double* X, int64_t count, int32_t* flag, hipStream_t stream);
hipError_t launch_set_i32(int32_t* p, int64_t count, int32_t value, hipStream_t stream);

// Householder QR in double-double of the first nf columns of A [2][m][n]
// (limb-major, nf <= m), with the reflections applied to the columns nf .. n - 1
// as well, which then hold Q^T times their input; tau [2][n] (entries 0 .. nf - 1
// written).  Panels of nb <= 64 columns.  qr_core_workspace gives the bytes of
// the workspace qr_core takes (SIZE_MAX for invalid sizes); qr_core checks no
// overlaps and returns an mdgemm status.
size_t qr_core_workspace(int64_t m, int64_t nf, int64_t n, int nb);
int qr_core(int64_t m, int64_t nf, int64_t n, int nb, double* A, double* tau, void* workspace, hipStream_t s);

}  // namespace mdg

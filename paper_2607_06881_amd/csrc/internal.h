// Internal launch interface shared by the HIP translation units of libmdgemm.
// Every launcher enqueues its kernels on `stream` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mdg {

constexpr int kSliceBits = 13;
constexpr int kDigitMax = (1 << kSliceBits) - 1;  // 8191
constexpr int kMaxSlices = 16;
constexpr int kMaxLimbs = 4;
constexpr int kZWords = 8;

// Slice-pair jobs of the level GEMM: job j multiplies the pairs
// (p_first + i, q_first - i) for i < npairs into output plane out[j].
struct JobTable {
  int njobs;
  uint8_t p_first[256];
  uint8_t q_first[256];
  uint8_t npairs[256];
  uint8_t out[256];
};

// a1: per-row (axis 0) or per-column (axis 1) grid exponents of a [rows][cols] plane.
hipError_t launch_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, hipStream_t stream);

// a2: digits [S][rows][cols] of X [L][rows][cols] on the grid exponents E.
hipError_t launch_split(int64_t rows, int64_t cols, int L, int S, int axis, const double* X, const int32_t* E,
                        double* D, hipStream_t stream);

// a3: level or pair products; `jobs` lists the pair groups, outputs are [*][m][n].
hipError_t launch_slice_gemm(int64_t m, int64_t n, int64_t k, const double* DA, const double* DB, double* out,
                             const JobTable& jobs, hipStream_t stream);

// a4: exact accumulation of `levels` planes into 8-word integers Z [8][m][n].
hipError_t launch_accumulate(int64_t m, int64_t n, int levels, const double* G, int64_t* Z, hipStream_t stream);

// a4 + a5: exact accumulation and greedy rounding into L limbs, scaled by 2^(EA+EB-26).
hipError_t launch_accum_renorm(int64_t m, int64_t n, int L, int levels, const double* G, const int32_t* EA,
                               const int32_t* EB, double* C, hipStream_t stream);

// Utilities: fill `count` doubles with +0.0; zero/set a device flag; scan for inf/nan.
hipError_t launch_zero_f64(double* p, int64_t count, hipStream_t stream);
hipError_t launch_nonfinite_scan(const double* X, int64_t count, int32_t* flag, hipStream_t stream);
hipError_t launch_set_i32(int32_t* p, int64_t count, int32_t value, hipStream_t stream);

}  // namespace mdg

// Step a1 -- balancing exponents, plus small utility kernels.
//
// Section 3 balances numbers by grouping them on a common exponent grid; here
// the group is one row of A or one column of B, and its grid exponent E is the
// largest frexp exponent (x = f 2^E, 1/2 <= |f| < 1) among the leading limbs of
// the line, so every element satisfies |x| < 2^E.  An all-zero line gets E = 0
// (section 3: a zero needs nothing).  The exponent convention is the one of the
// worked example of section 2, whose quarters have exponents 0, -13, -26, -39.
//
// Rows (axis 0): one wave64 per row reads the row with 8-byte coalesced loads
// and reduces with cross-lane max.  Columns (axis 1): lanes span 64 consecutive
// columns (coalesced 512-byte rows), the four waves of a block and the blocks
// of grid.y split the rows, partial maxima meet in LDS and then in global
// memory through a vector atomic max; a last pass maps "no nonzero" to 0.
#include <climits>

#include "digits.h"
#include "internal.h"

namespace mdg {
namespace {

__device__ inline int wave_max(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
  return v;
}

__global__ void __launch_bounds__(256) row_exponents_kernel(int64_t rows, int64_t cols, const double* __restrict__ X0,
                                                            int32_t* __restrict__ E) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;  // whole wave leaves together
  const double* r = X0 + row * cols;
  int best = kNoExp;
  int64_t c = lane;
  // four independent loads per lane in flight, then the tail
  for (; c + 192 < cols; c += 256) {
    const double x0 = r[c], x1 = r[c + 64], x2 = r[c + 128], x3 = r[c + 192];
    best = max(best, max(max(frexp_exp_or_min(x0), frexp_exp_or_min(x1)),
                         max(frexp_exp_or_min(x2), frexp_exp_or_min(x3))));
  }
  for (; c < cols; c += 64) best = max(best, frexp_exp_or_min(r[c]));
  best = wave_max(best);
  if (lane == 0) E[row] = (best == kNoExp) ? 0 : best;
}

__global__ void __launch_bounds__(256) col_exponents_kernel(int64_t rows, int64_t cols, const double* __restrict__ X0,
                                                            int32_t* __restrict__ E) {
  __shared__ int part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  int best = kNoExp;
  if (col < cols) {
    const int64_t stride = static_cast<int64_t>(gridDim.y) * 4;
    for (int64_t r = static_cast<int64_t>(blockIdx.y) * 4 + wave; r < rows; r += stride)
      best = max(best, frexp_exp_or_min(X0[r * cols + col]));
  }
  part[wave][lane] = best;
  __syncthreads();
  if (wave == 0 && col < cols) {
    best = max(max(part[0][lane], part[1][lane]), max(part[2][lane], part[3][lane]));
    if (best != kNoExp) atomicMax(E + col, best);
  }
}

// Both operands in one launch, without an initial fill or a final pass over
// atomics: blocks [0, ra) take four rows of A each (one wave per row); blocks
// [ra, ra + cx cy) take 64 columns of B over one chunk of chunk_rows rows (lanes
// on consecutive columns, the four waves on interleaved rows) and write the
// chunk's maxima to P[chunk][column] (kNoExp where the chunk has no nonzero), or,
// with a single chunk (cy = 1), the final exponents straight to EB.  Every lane
// issues its loads in predicated batches of eight before reducing them; with
// kVec, A's rows are read as 16-byte pairs (k even and A 16-byte aligned).
template <bool kVec>
__global__ void __launch_bounds__(256) exponents_ab_kernel(int64_t m, int64_t k, int64_t n,
                                                           const double* __restrict__ A0,
                                                           const double* __restrict__ B0, int32_t* __restrict__ EA,
                                                           int32_t* __restrict__ EB, int32_t* __restrict__ P,
                                                           int64_t ra, int64_t cx, int64_t cy, int64_t chunk_rows) {
  __shared__ int part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t b = blockIdx.x;
  if (b < ra) {  // block-uniform: A's rows
    const int64_t row = b * 4 + wave;
    if (row >= m) return;
    int best = kNoExp;
    if constexpr (kVec) {
      const double2* r = reinterpret_cast<const double2*>(A0 + row * k);
      const int64_t k2 = k / 2;
      for (int64_t c = lane; c < k2; c += 64 * 8) {
        double2 x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = c + 64 * j < k2 ? r[c + 64 * j] : make_double2(0.0, 0.0);
#pragma unroll
        for (int j = 0; j < 8; ++j) best = max(best, max(frexp_exp_or_min(x[j].x), frexp_exp_or_min(x[j].y)));
      }
    } else {
      const double* r = A0 + row * k;
      for (int64_t c = lane; c < k; c += 64 * 8) {
        double x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = c + 64 * j < k ? r[c + 64 * j] : 0.0;
#pragma unroll
        for (int j = 0; j < 8; ++j) best = max(best, frexp_exp_or_min(x[j]));
      }
    }
    best = wave_max(best);
    if (lane == 0) EA[row] = best == kNoExp ? 0 : best;
    return;
  }
  const int64_t bb = b - ra, chunk = bb / cx;
  const int64_t col = (bb - chunk * cx) * 64 + lane;
  int best = kNoExp;
  if (col < n) {
    const int64_t r1 = min(k, (chunk + 1) * chunk_rows);
    for (int64_t r = chunk * chunk_rows + wave; r < r1; r += 4 * 8) {
      double x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = r + 4 * j < r1 ? B0[(r + 4 * j) * n + col] : 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j) best = max(best, frexp_exp_or_min(x[j]));
    }
  }
  part[wave][lane] = best;
  __syncthreads();
  if (wave == 0 && col < n) {
    best = max(max(part[0][lane], part[1][lane]), max(part[2][lane], part[3][lane]));
    if (cy == 1)
      EB[col] = best == kNoExp ? 0 : best;
    else
      P[chunk * n + col] = best;
  }
}

// EB[j] = the largest of the cy chunk maxima of column j, 0 for a zero column.
__global__ void __launch_bounds__(256) reduce_col_chunks_kernel(int64_t n, int64_t cy, const int32_t* __restrict__ P,
                                                                int32_t* __restrict__ EB) {
  const int64_t col = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (col >= n) return;
  int best = kNoExp;
  for (int64_t c = 0; c < cy; c += 8) {
    int v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = c + j < cy ? P[(c + j) * n + col] : kNoExp;
#pragma unroll
    for (int j = 0; j < 8; ++j) best = max(best, v[j]);
  }
  EB[col] = best == kNoExp ? 0 : best;
}

// Smallest frexp exponent of a nonzero entry of every row (one wave per row) or
// column (64 columns per block, as col_exponents_kernel, vector atomic min);
// INT_MAX for a line without a nonzero entry.
__device__ inline int frexp_exp_or_max(double x) {
  const int e = frexp_exp_or_min(x);
  return e == kNoExp ? INT_MAX : e;
}

__device__ inline int wave_min(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, 64));
  return v;
}

__global__ void __launch_bounds__(256) row_min_exponents_kernel(int64_t rows, int64_t cols,
                                                                const double* __restrict__ X0,
                                                                int32_t* __restrict__ Emin) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const double* r = X0 + row * cols;
  int best = INT_MAX;
  for (int64_t c = lane; c < cols; c += 64) best = min(best, frexp_exp_or_max(r[c]));
  best = wave_min(best);
  if (lane == 0) Emin[row] = best;
}

__global__ void __launch_bounds__(256) col_min_exponents_kernel(int64_t rows, int64_t cols,
                                                                const double* __restrict__ X0,
                                                                int32_t* __restrict__ Emin) {
  __shared__ int part[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t col = static_cast<int64_t>(blockIdx.x) * 64 + lane;
  int best = INT_MAX;
  if (col < cols) {
    const int64_t stride = static_cast<int64_t>(gridDim.y) * 4;
    for (int64_t r = static_cast<int64_t>(blockIdx.y) * 4 + wave; r < rows; r += stride)
      best = min(best, frexp_exp_or_max(X0[r * cols + col]));
  }
  part[wave][lane] = best;
  __syncthreads();
  if (wave == 0 && col < cols) {
    best = min(min(part[0][lane], part[1][lane]), min(part[2][lane], part[3][lane]));
    if (best != INT_MAX) atomicMin(Emin + col, best);
  }
}

// spread = E - Emin, 0 for a line without a nonzero entry (in place over Emin).
__global__ void spread_kernel(int64_t count, const int32_t* __restrict__ E, int32_t* __restrict__ spread) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < count) spread[i] = spread[i] == INT_MAX ? 0 : E[i] - spread[i];
}

__global__ void finalize_exponents_kernel(int64_t count, int32_t* __restrict__ E) {
  int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < count && E[i] == kNoExp) E[i] = 0;
}

__global__ void set_i32_kernel(int32_t* __restrict__ p, int64_t count, int32_t value) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = value;
}

__global__ void zero_f64_kernel(double* __restrict__ p, int64_t count) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = 0.0;
}

__global__ void nonfinite_scan_kernel(const double* __restrict__ X, int64_t count, int32_t* __restrict__ flag) {
  bool bad = false;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    uint64_t b = static_cast<uint64_t>(__double_as_longlong(X[i]));
    bad |= ((b >> 52) & 0x7ff) == 0x7ff;
  }
  if (bad) *flag = 1;  // every writer stores the same value
}

inline unsigned grid_for(int64_t count, int block, int64_t cap = 65536) {
  int64_t g = (count + block - 1) / block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return static_cast<unsigned>(g);
}

}  // namespace

hipError_t launch_exponents(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, hipStream_t stream) {
  if (axis == 0) {
    if (rows == 0) return hipSuccess;
    if (cols == 0) return launch_set_i32(E, rows, 0, stream);
    unsigned g = static_cast<unsigned>((rows + 3) / 4);
    hipLaunchKernelGGL(row_exponents_kernel, dim3(g), dim3(256), 0, stream, rows, cols, X0, E);
    return hipGetLastError();
  }
  if (cols == 0) return hipSuccess;
  hipError_t err = launch_set_i32(E, cols, kNoExp, stream);
  if (err != hipSuccess) return err;
  if (rows > 0) {
    // enough blocks to cover the chip; each block walks rows / (4 * gy) rows of 64 columns
    int64_t gx = (cols + 63) / 64;
    int64_t gy = (2048 + gx - 1) / gx;
    int64_t max_gy = (rows + 63) / 64;  // keep at least ~64 rows per block row
    if (gy > max_gy) gy = max_gy;
    if (gy < 1) gy = 1;
    if (gy > 65535) gy = 65535;
    hipLaunchKernelGGL(col_exponents_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)), dim3(256),
                       0, stream, rows, cols, X0, E);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(finalize_exponents_kernel, dim3(grid_for(cols, 256, 1ll << 30)), dim3(256), 0, stream, cols, E);
  return hipGetLastError();
}

hipError_t launch_exponents_ab(int64_t m, int64_t k, int64_t n, const double* A0, const double* B0, int32_t* EA,
                               int32_t* EB, void* scratch, size_t scratch_bytes, hipStream_t stream) {
  const int64_t ra = (m + 3) / 4, cx = (n + 63) / 64;
  // 16 column chunks: a wave of B's blocks then reads 64 columns x k / 64 rows,
  // as many elements as a wave of A's rows (both kinds of blocks take about the
  // same time); chunks of at least 64 rows
  int64_t cy = 16;
  const int64_t max_cy = (k + 63) / 64;
  if (cy > max_cy) cy = max_cy;
  if (cy < 1) cy = 1;
  if (cy > 1 && static_cast<size_t>(cy) * static_cast<size_t>(n) * sizeof(int32_t) > scratch_bytes) {
    hipError_t err = launch_exponents(m, k, 0, A0, EA, stream);
    return err != hipSuccess ? err : launch_exponents(k, n, 1, B0, EB, stream);
  }
  const int64_t chunk_rows = cy > 1 ? (k + cy - 1) / cy : (k > 0 ? k : 1);
  const int64_t blocks = ra + cx * cy;
  if (blocks == 0) return hipSuccess;
  if (blocks > INT_MAX) return hipErrorInvalidValue;
  int32_t* P = static_cast<int32_t*>(scratch);
  const bool vec = k % 2 == 0 && (reinterpret_cast<uintptr_t>(A0) & 15u) == 0;
  if (vec)
    hipLaunchKernelGGL(exponents_ab_kernel<true>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, m, k, n,
                       A0, B0, EA, EB, P, ra, cx, cy, chunk_rows);
  else
    hipLaunchKernelGGL(exponents_ab_kernel<false>, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, m, k, n,
                       A0, B0, EA, EB, P, ra, cx, cy, chunk_rows);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || cy == 1 || n == 0) return err;
  hipLaunchKernelGGL(reduce_col_chunks_kernel, dim3(grid_for(n, 256, 1ll << 30)), dim3(256), 0, stream, n, cy, P, EB);
  return hipGetLastError();
}

hipError_t launch_line_spread(int64_t rows, int64_t cols, int axis, const double* X0, int32_t* E, int32_t* spread,
                              hipStream_t stream) {
  hipError_t err = launch_exponents(rows, cols, axis, X0, E, stream);
  if (err != hipSuccess) return err;
  const int64_t lines = axis == 0 ? rows : cols;
  if (lines == 0) return hipSuccess;
  err = launch_set_i32(spread, lines, INT_MAX, stream);
  if (err != hipSuccess) return err;
  if (rows > 0 && cols > 0) {
    if (axis == 0) {
      hipLaunchKernelGGL(row_min_exponents_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream,
                         rows, cols, X0, spread);
    } else {
      int64_t gx = (cols + 63) / 64;
      int64_t gy = (2048 + gx - 1) / gx;
      int64_t max_gy = (rows + 63) / 64;
      if (gy > max_gy) gy = max_gy;
      if (gy < 1) gy = 1;
      if (gy > 65535) gy = 65535;
      hipLaunchKernelGGL(col_min_exponents_kernel, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy)),
                         dim3(256), 0, stream, rows, cols, X0, spread);
    }
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  hipLaunchKernelGGL(spread_kernel, dim3(grid_for(lines, 256, 1ll << 30)), dim3(256), 0, stream, lines, E, spread);
  return hipGetLastError();
}

hipError_t launch_set_i32(int32_t* p, int64_t count, int32_t value, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(set_i32_kernel, dim3(grid_for(count, 256)), dim3(256), 0, stream, p, count, value);
  return hipGetLastError();
}

hipError_t launch_zero_f64(double* p, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_f64_kernel, dim3(grid_for(count, 256)), dim3(256), 0, stream, p, count);
  return hipGetLastError();
}

hipError_t launch_nonfinite_scan(const double* X, int64_t count, int32_t* flag, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(nonfinite_scan_kernel, dim3(grid_for(count, 256, 4096)), dim3(256), 0, stream, X, count, flag);
  return hipGetLastError();
}

}  // namespace mdg

// Calibration kernels: the rates the level GEMM and the HBM-bound stages are
// measured against, taken on the same device in the same process.
//
// mfma_f64_probe_kernel keeps the FP64 matrix pipes of every SIMD busy with
// independent v_mfma_f64_16x16x4f64 chains (eight accumulators per wave, no
// memory traffic inside the loop), so its rate is the sustainable FP64 MFMA
// throughput of the chip at its current clock.  copy_probe_kernel streams a
// buffer through 32-byte loads and stores, the sustainable HBM rate of a
// read-plus-write stream; stream_probe_kernel the rate of a plain stream with
// the read/write mix of one of the memory-bound stages.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "mdgemm.h"

namespace mdg {
namespace {

typedef double d4 __attribute__((ext_vector_type(4)));
constexpr int kProbeChains = 8;
constexpr int kProbeThreads = 256;

__global__ __launch_bounds__(kProbeThreads) void mfma_f64_probe_kernel(int64_t iters, double* sink) {
  d4 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) acc[c] = d4{0.0, 0.0, 0.0, 0.0};
  // operands that depend on the lane, so that nothing folds
  const double a = 1.0 + static_cast<double>(threadIdx.x) * 0x1p-20;
  const double b = 1.0 - static_cast<double>(threadIdx.x) * 0x1p-20;
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) acc[c] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[c], 0, 0, 0);
  }
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  sink[static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x] = s;
}

// Each block copies kCopyUnroll x 256 consecutive 32-byte vectors: every thread
// issues all its loads before its stores, so that enough bytes are in flight.
constexpr int kCopyUnroll = 4;

__global__ __launch_bounds__(256) void copy_probe_kernel(const d4* __restrict__ src, d4* __restrict__ dst,
                                                         int64_t count4) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * (256 * kCopyUnroll) + threadIdx.x;
  d4 v[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u)
    if (base + u * 256 < count4) v[u] = __builtin_nontemporal_load(&src[base + u * 256]);
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u)
    if (base + u * 256 < count4) __builtin_nontemporal_store(v[u], &dst[base + u * 256]);
}

// A plain stream with a given mix: every element i reads `reads` planes and
// writes `writes` planes (plane stride count), loads issued in batches of eight.
// Timed at a stage's own size and read/write mix it gives the rate a simple
// streaming kernel reaches for that traffic, next to the published peak.
__global__ __launch_bounds__(256) void stream_probe_kernel(const double* __restrict__ src, int reads,
                                                           double* __restrict__ dst, int writes, int64_t count) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < count;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    double s = 0.0;
    for (int r0 = 0; r0 < reads; r0 += 8) {
      double v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = r0 + j < reads ? src[static_cast<int64_t>(r0 + j) * count + i] : 0.0;
#pragma unroll
      for (int j = 0; j < 8; ++j) s += v[j];
    }
    for (int w = 0; w < writes; ++w) dst[static_cast<int64_t>(w) * count + i] = s + static_cast<double>(w);
  }
}

}  // namespace
}  // namespace mdg

extern "C" {

int mdgemm_probe_stream(const double* src, int reads, double* dst, int writes, int64_t count, void* stream) {
  if (reads < 1 || reads > 256 || writes < 0 || writes > 256 || count < 0 || count > (int64_t{1} << 40))
    return MDGEMM_EINVAL;
  if (count == 0) return MDGEMM_OK;
  if (!src || (writes > 0 && !dst)) return MDGEMM_EINVAL;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  const uintptr_t sbytes = static_cast<uintptr_t>(count) * reads * sizeof(double);
  const uintptr_t dbytes = static_cast<uintptr_t>(count) * writes * sizeof(double);
  if (writes > 0 && s0 < d0 + dbytes && d0 < s0 + sbytes) return MDGEMM_EINVAL;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, int64_t{1} << 20);
  hipLaunchKernelGGL(mdg::stream_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), src, reads, dst, writes, count);
  return hipGetLastError() == hipSuccess ? MDGEMM_OK : MDGEMM_EHIP;
}

int64_t mdgemm_probe_mfma_f64(int64_t blocks, int64_t iters, double* sink, void* stream) {
  if (blocks < 1 || blocks > (int64_t{1} << 24) || iters < 1 || !sink) return MDGEMM_EINVAL;
  hipLaunchKernelGGL(mdg::mfma_f64_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(mdg::kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), iters, sink);
  if (hipGetLastError() != hipSuccess) return MDGEMM_EHIP;
  // 2 * 16 * 16 * 4 flops per instruction, kProbeChains per iteration per wave
  return blocks * (mdg::kProbeThreads / 64) * iters * mdg::kProbeChains * 2048;
}

int mdgemm_probe_copy(const double* src, double* dst, int64_t count, void* stream) {
  if (count < 0 || count % 4 != 0 || (count > 0 && (!src || !dst))) return MDGEMM_EINVAL;
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 31u) return MDGEMM_EINVAL;
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  const uintptr_t bytes = static_cast<uintptr_t>(count) * sizeof(double);
  if (count > 0 && s0 < d0 + bytes && d0 < s0 + bytes) return MDGEMM_EINVAL;
  if (count == 0) return MDGEMM_OK;
  const int64_t count4 = count / 4;
  const int64_t blocks = (count4 + 256 * mdg::kCopyUnroll - 1) / (256 * mdg::kCopyUnroll);
  if (blocks > 0x7fffffff) return MDGEMM_EINVAL;
  hipLaunchKernelGGL(mdg::copy_probe_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), reinterpret_cast<const mdg::d4*>(src),
                     reinterpret_cast<mdg::d4*>(dst), count4);
  return hipGetLastError() == hipSuccess ? MDGEMM_OK : MDGEMM_EHIP;
}

}  // extern "C"

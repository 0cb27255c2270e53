// Steps a4 and a5 -- exact accumulation of the level products and rounding
// into nonoverlapping limbs.
//
// Section 2 (steps 4 and 5 of the overview) extracts the parts of the product
// and adds them into a multiple double on the regular cores, a massively
// parallel summation of the levels of every output element.  Section 1
// (renormalization) requires the result to be a sum of nonoverlapping doubles.
//
// Level t of an output element is an integer G_t, |G_t| < 2^53, of weight
// 2^(-w t) (times the grid scale 2^(EA + EB - 2w)); w = 13 for the digits of
// section 2, up to 26 for the adaptive width.  Their sum is formed exactly, in
// increasing significance (t = T down to 0), as the two's-complement integer
// N = sum_t G_t 2^(w (T - t)) held in NW 64-bit words in registers (a base-2^w
// carry chain: one int64 add, mask and shift per level); the value is
// Z = N 2^(-w T).  The L limbs are then peeled off greedily with
// round-to-nearest-even: c_0 = RN(Z), c_1 = RN(Z - c_0), ..., each taken from
// the 53 leading bits of the remaining magnitude with the round bit and the
// sticky bits below it; when a limb rounds up, the remainder changes sign.  The
// result is the canonical nonoverlapping representation, |c_{l+1}| <= ulp(c_l)/2.
//
// One thread per output element; consecutive threads take consecutive columns,
// so the T + 1 level loads and the L limb stores are contiguous 512-byte rows.
#include <type_traits>

#include "digits.h"
#include "internal.h"

namespace mdg {
namespace {

// The chain over levels read from G [levels][m][n] (integer-valued doubles, or
// int32 planes of the int8 level products).  Loads are issued eight levels at a
// time before any of them is used, so a thread keeps up to eight independent
// loads in flight.
template <int NW, class PT = double>
__device__ inline void accumulate_levels(uint64_t (&N)[NW], const PT* __restrict__ G, int levels, int w,
                                         int64_t plane, int64_t idx) {
#pragma unroll
  for (int i = 0; i < NW; ++i) N[i] = 0;
  const int T = levels - 1;
  const uint64_t mask = (1ull << w) - 1ull;
  CarryChain<NW> chain;
  for (int t0 = T; t0 >= 0; t0 -= 8) {
    // unconditional loads (levels below 0 re-read level 0 and are discarded),
    // so that the eight loads go out back to back
    PT g[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int t = t0 - u;
      g[u] = G[static_cast<int64_t>(t >= 0 ? t : 0) * plane + idx];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (t0 - u < 0) break;
      chain.step(N, static_cast<int64_t>(g[u]), w, mask);  // exact: |G_t| < 2^53
    }
  }
  chain.finish(N, w, T);
}

template <int NW, class PT>
__global__ void __launch_bounds__(256) accum_renorm_kernel(int64_t m, int64_t n, int L, int levels, int w,
                                                           const PT* __restrict__ G,
                                                           const int32_t* __restrict__ EA,
                                                           const int32_t* __restrict__ EB, double* __restrict__ C) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int64_t plane = m * n;
  const int ebj = EB[j];
  for (int64_t i = blockIdx.y; i < m; i += gridDim.y) {
    const int64_t idx = i * n + j;
    uint64_t N[NW];
    accumulate_levels<NW, PT>(N, G, levels, w, plane, idx);
    const int scale = EA[i] + ebj - 2 * w - w * (levels - 1);
    round_limbs<NW>(N, L, scale, C, plane, idx);
  }
}

template <int NW>
__global__ void __launch_bounds__(256) accumulate_kernel(int64_t m, int64_t n, int levels, int w,
                                                         const double* __restrict__ G, int64_t* __restrict__ Z) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= n) return;
  const int64_t plane = m * n;
  for (int64_t i = blockIdx.y; i < m; i += gridDim.y) {
    const int64_t idx = i * n + j;
    uint64_t N[NW];
    accumulate_levels<NW>(N, G, levels, w, plane, idx);
    const uint64_t ext = (N[NW - 1] >> 63) ? ~0ull : 0ull;
    for (int w = 0; w < kZWords; ++w)
      Z[static_cast<int64_t>(w) * plane + idx] = static_cast<int64_t>(w < NW ? word_at<NW>(N, w) : ext);
  }
}

// Levels from the output planes of a Karatsuba schedule: each plane enters a
// few levels with small integer coefficients.  Every thread keeps its levels
// as 64-bit integers in LDS (level t of thread x at lv[t * blockDim.x + x], one
// more slot t = T + 1 takes the padding entries), reads each plane once (a
// batch of 8 loads in flight while the previous batch is applied) and adds
// coef * plane to the levels of the plane's entries.
// The entries come four at a time (one 8-byte scalar load); the levels of one
// plane are distinct, so the four old values are read before any is written
// and the four read-modify-writes overlap.  Plane values are integers below
// 2^53 and the level sums are the exact G_t (|G_t| < 2^53), so no step rounds.
// Then the carry chain and rounding of accum_renorm_kernel, or (C == nullptr)
// the levels written out as doubles.
constexpr int kBatch = 8;

template <int NW>
__global__ void __launch_bounds__(256) plan_accum_kernel(int64_t m, int64_t n, int L, int levels, int w, int planes,
                                                         const double* __restrict__ P,
                                                         const uint32_t* __restrict__ chunk_first,
                                                         const uint2* __restrict__ chunks,
                                                         const int32_t* __restrict__ EA,
                                                         const int32_t* __restrict__ EB, double* __restrict__ C,
                                                         double* __restrict__ Gout) {
  extern __shared__ int64_t lv[];
  const int bd = blockDim.x;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * bd + threadIdx.x;
  if (j >= n) return;  // no barriers below: every thread owns its own LDS slots
  int64_t* my = lv + threadIdx.x;
  const int64_t plane = m * n;
  const int T = levels - 1;
  const uint64_t mask = (1ull << w) - 1ull;
  const int ebj = C ? EB[j] : 0;
  for (int64_t i = blockIdx.y; i < m; i += gridDim.y) {
    const int64_t idx = i * n + j;
    for (int t = 0; t <= levels; ++t) my[t * bd] = 0;
    // planes in batches of kBatch: the next batch's loads are in flight while
    // the current batch's entries are applied
    double cur[kBatch], nxt[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) cur[u] = P[static_cast<int64_t>(u < planes ? u : planes - 1) * plane + idx];
    for (int p0 = 0; p0 < planes; p0 += kBatch) {
      if (p0 + kBatch < planes) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
          const int pl = p0 + kBatch + u < planes ? p0 + kBatch + u : planes - 1;
          nxt[u] = P[static_cast<int64_t>(pl) * plane + idx];
        }
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int pl = p0 + u;
        if (pl >= planes) break;
        const int64_t v = static_cast<int64_t>(cur[u]);  // exact: integer below 2^53
        const uint32_t c1 = chunk_first[pl + 1];
        for (uint32_t c = chunk_first[pl]; c < c1; ++c) {
          const uint2 ch = chunks[c];
          const uint32_t e[4] = {ch.x & 0xffffu, ch.x >> 16, ch.y & 0xffffu, ch.y >> 16};
          int64_t* a[4];
          int64_t old[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            a[q] = my + static_cast<int>(e[q] & 0xffu) * bd;
            old[q] = *a[q];
          }
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *a[q] = old[q] + static_cast<int64_t>(static_cast<int8_t>(e[q] >> 8)) * v;
        }
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) cur[u] = nxt[u];
    }
    if (!C) {
      for (int t = 0; t < levels; ++t) Gout[static_cast<int64_t>(t) * plane + idx] = static_cast<double>(my[t * bd]);
      continue;
    }
    uint64_t N[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) N[q] = 0;
    CarryChain<NW> chain;
    for (int t = T; t >= 0; --t) chain.step(N, my[t * bd], w, mask);
    chain.finish(N, w, T);
    const int scale = EA[i] + ebj - 2 * w - w * T;
    round_limbs<NW>(N, L, scale, C, plane, idx);
  }
}

}  // namespace

// Words for |N| < 2^(w T + 54) plus a sign bit.
int accum_words(int levels, int w) {
  const int bits = w * (levels - 1) + 55;
  return (bits + 63) / 64;
}

namespace {

inline dim3 elem_grid(int64_t m, int64_t n) {
  return dim3(static_cast<unsigned>((n + 255) / 256), static_cast<unsigned>(m < 65535 ? m : 65535));
}

template <int NW>
using Words = std::integral_constant<int, NW>;

// Calls f(Words<NW>{}) for the smallest instantiated NW >= words (levels up to
// 2 * 64 - 1 need 27 words).
template <class F>
hipError_t with_words(int words, F&& f) {
  if (words <= 2) f(Words<2>{});
  else if (words <= 3) f(Words<3>{});
  else if (words <= 4) f(Words<4>{});
  else if (words <= 5) f(Words<5>{});
  else if (words <= 6) f(Words<6>{});
  else if (words <= 7) f(Words<7>{});
  else if (words <= 8) f(Words<8>{});
  else if (words <= 10) f(Words<10>{});
  else if (words <= 12) f(Words<12>{});
  else if (words <= 14) f(Words<14>{});
  else if (words <= 15) f(Words<15>{});  // sixteen limbs at the default digits: 13 x 65 + 55 bits
  else if (words <= 20) f(Words<20>{});
  else if (words <= kZWords) f(Words<kZWords>{});
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_accum_renorm(int64_t m, int64_t n, int L, int levels, int w, const double* G, const int32_t* EA,
                               const int32_t* EB, double* C, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  const dim3 grid = elem_grid(m, n);
  // the next word count instantiated (the extra words hold the sign extension)
  return with_words(accum_words(levels, w), [&](auto nw) {
    hipLaunchKernelGGL((accum_renorm_kernel<decltype(nw)::value, double>), grid, dim3(256), 0, stream, m, n, L,
                       levels, w, G, EA, EB, C);
  });
}

hipError_t launch_accum_renorm_i32(int64_t m, int64_t n, int L, int levels, int w, const int32_t* G,
                                   const int32_t* EA, const int32_t* EB, double* C, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  const dim3 grid = elem_grid(m, n);
  return with_words(accum_words(levels, w), [&](auto nw) {
    hipLaunchKernelGGL((accum_renorm_kernel<decltype(nw)::value, int32_t>), grid, dim3(256), 0, stream, m, n, L,
                       levels, w, G, EA, EB, C);
  });
}

hipError_t launch_plan_accum(int64_t m, int64_t n, int L, int levels, int w, int planes, const double* P,
                             const uint32_t* chunk_first, const uint32_t* chunks, const int32_t* EA,
                             const int32_t* EB, double* C, double* Gout, hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  // (levels + 1) x threads x 8 bytes of LDS: at most 32 KB up to 63 levels, 64 KB for 127
  const int bd = levels < 16 ? 256 : (levels < 32 ? 128 : 64);
  const dim3 grid(static_cast<unsigned>((n + bd - 1) / bd), static_cast<unsigned>(m < 65535 ? m : 65535));
  const size_t lds = sizeof(int64_t) * static_cast<size_t>(levels + 1) * bd;
  const uint2* ch = reinterpret_cast<const uint2*>(chunks);
  if (!C) {
    hipLaunchKernelGGL(plan_accum_kernel<2>, grid, dim3(bd), lds, stream, m, n, L, levels, w, planes, P,
                       chunk_first, ch, EA, EB, C, Gout);
    return hipGetLastError();
  }
  return with_words(accum_words(levels, w), [&](auto nw) {
    hipLaunchKernelGGL(plan_accum_kernel<decltype(nw)::value>, grid, dim3(bd), lds, stream, m, n, L, levels, w,
                       planes, P, chunk_first, ch, EA, EB, C, Gout);
  });
}

hipError_t launch_accumulate(int64_t m, int64_t n, int levels, int w, const double* G, int64_t* Z,
                             hipStream_t stream) {
  if (m == 0 || n == 0) return hipSuccess;
  const dim3 grid = elem_grid(m, n);
  return with_words(accum_words(levels, w), [&](auto nw) {
    hipLaunchKernelGGL(accumulate_kernel<decltype(nw)::value>, grid, dim3(256), 0, stream, m, n, levels, w, G, Z);
  });
}

}  // namespace mdg

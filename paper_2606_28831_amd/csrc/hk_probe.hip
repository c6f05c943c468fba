// Rate probes behind the rooflines of the score passes (measurement only, not part of the
// method): the issue rate of the hardware exponential and the bf16 MFMA rate, each from a
// kernel that keeps enough independent chains in flight to be throughput- rather than
// latency-bound, and whether a SIMD overlaps MFMA and VALU work within a wave or across
// waves.
#include "hk_internal.h"

namespace hk {

constexpr int PROBE_NT = 256;

// Eight independent chains x <- 2^(-x) per thread (the negation is a source modifier, so
// the chain is one v_exp_f32 per step); the values stay in (0, 1].
__global__ __launch_bounds__(PROBE_NT) void probe_exp_kernel(int iters, float* __restrict__ out) {
  float x[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = 0.125f * (float)(c + 1) + 1e-6f * (float)threadIdx.x;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) x[c] = __builtin_amdgcn_exp2f(-x[c]);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c) s += x[c];
  out[(size_t)blockIdx.x * PROBE_NT + threadIdx.x] = s;
}

// Four independent 32x32x16 bf16 MFMA accumulation chains per wave.
__global__ __launch_bounds__(PROBE_NT) void probe_mfma_kernel(int iters, float* __restrict__ out) {
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)((threadIdx.x + e) & 7));
    b[e] = (__bf16)(0.002f * (float)((threadIdx.x * 3 + e) & 7));
  }
  f32x16 acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(size_t)blockIdx.x * PROBE_NT + threadIdx.x] = s;
}

// The score passes' per-element VALU work beside their MFMAs, alone and together.  One
// step is what a score wave does per MFMA: one 32x32x16 bf16 MFMA and, for two (row, key)
// values, an fma, an exponential and an add (a pass's tile is 8 MFMAs and 16 values per
// lane).  Four MFMA chains and eight exponential chains per wave keep both units fed; a and
// b come from the host, so the fma cannot fold into the exponential's source modifier.
//   MIX    every wave runs iters x 4 steps with both kinds of work interleaved, one step
//          per scheduling region (as the score passes issue them);
//   SPLIT  the same total work with the kinds in different waves of each SIMD: even waves
//          the MFMAs, odd waves the VALU work, 2 iters x 4 steps each;
//   VALU   only the VALU part of MIX;  MFMA4  only the MFMA part of MIX.
template <bool DO_M, bool DO_V>
__device__ __forceinline__ void probe_steps(int iters, float a, float b, bf16x8 qa, bf16x8 qb,
                                            f32x16 (&acc)[4], float (&x)[8], float (&sum)[2]) {
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if constexpr (DO_M) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, qb, acc[c], 0, 0, 0);
      if constexpr (DO_V) {
        x[2 * c] = __builtin_amdgcn_exp2f(fmaf(x[2 * c], a, b));
        x[2 * c + 1] = __builtin_amdgcn_exp2f(fmaf(x[2 * c + 1], a, b));
        sum[0] += x[2 * c];
        sum[1] += x[2 * c + 1];
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

template <int KIND>
__global__ __launch_bounds__(PROBE_NT) void probe_mix_kernel(int iters, float a, float b,
                                                             float* __restrict__ out) {
  bf16x8 qa, qb;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    qa[e] = (__bf16)(0.001f * (float)((threadIdx.x + e) & 7));
    qb[e] = (__bf16)(0.002f * (float)((threadIdx.x * 3 + e) & 7));
  }
  f32x16 acc[4];
  float x[8], sum[2] = {0.f, 0.f};
#pragma unroll
  for (int c = 0; c < 4; ++c) acc[c] = f32x16{};
#pragma unroll
  for (int c = 0; c < 8; ++c) x[c] = 0.125f * (float)(c + 1) + 1e-6f * (float)threadIdx.x;
  const bool even = ((threadIdx.x >> 6) & 1) == 0;
  if constexpr (KIND == HK_PROBE_MIX) probe_steps<true, true>(iters, a, b, qa, qb, acc, x, sum);
  else if constexpr (KIND == HK_PROBE_VALU) probe_steps<false, true>(iters, a, b, qa, qb, acc, x, sum);
  else if constexpr (KIND == HK_PROBE_MFMA4) probe_steps<true, false>(iters, a, b, qa, qb, acc, x, sum);
  else if (even) probe_steps<true, false>(2 * iters, a, b, qa, qb, acc, x, sum);
  else probe_steps<false, true>(2 * iters, a, b, qa, qb, acc, x, sum);
  float s = sum[0] + sum[1];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  out[(size_t)blockIdx.x * PROBE_NT + threadIdx.x] = s;
}

}  // namespace hk

using namespace hk;

hipError_t hk_launch_probe(int kind, int blocks, int iters, float* out, hipStream_t st) {
  const dim3 g(blocks), b(PROBE_NT);
  // x <- 2^(1e-7 - x) keeps every exponential chain in [0.5, 1]
  const float fa = -1.0f, fb = 1e-7f;
  switch (kind) {
    case HK_PROBE_EXP: hipLaunchKernelGGL(probe_exp_kernel, g, b, 0, st, iters, out); break;
    case HK_PROBE_MFMA: hipLaunchKernelGGL(probe_mfma_kernel, g, b, 0, st, iters, out); break;
    case HK_PROBE_MIX: hipLaunchKernelGGL(probe_mix_kernel<HK_PROBE_MIX>, g, b, 0, st, iters, fa, fb, out); break;
    case HK_PROBE_SPLIT: hipLaunchKernelGGL(probe_mix_kernel<HK_PROBE_SPLIT>, g, b, 0, st, iters, fa, fb, out); break;
    case HK_PROBE_VALU: hipLaunchKernelGGL(probe_mix_kernel<HK_PROBE_VALU>, g, b, 0, st, iters, fa, fb, out); break;
    default: hipLaunchKernelGGL(probe_mix_kernel<HK_PROBE_MFMA4>, g, b, 0, st, iters, fa, fb, out); break;
  }
  return hipGetLastError();
}

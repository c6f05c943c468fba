// Rate probes behind the rooflines of the score passes (measurement only, not part of the
// method): the issue rate of the hardware exponential and the bf16 MFMA rate, each from a
// kernel that keeps enough independent chains in flight to be throughput- rather than
// latency-bound.
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

}  // namespace hk

using namespace hk;

hipError_t hk_launch_probe(int kind, int blocks, int iters, float* out, hipStream_t st) {
  if (kind == HK_PROBE_EXP)
    hipLaunchKernelGGL(probe_exp_kernel, dim3(blocks), dim3(PROBE_NT), 0, st, iters, out);
  else
    hipLaunchKernelGGL(probe_mfma_kernel, dim3(blocks), dim3(PROBE_NT), 0, st, iters, out);
  return hipGetLastError();
}

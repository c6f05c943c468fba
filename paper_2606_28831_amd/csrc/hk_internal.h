// Internal helpers shared by the HIP kernels of libhardkv (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "hardkv.h"

#define HK_PAGE 16
#define HK_WAVE 64

namespace hk {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Hardware base-2 exponential and logarithm (v_exp_f32 / v_log_f32, ~1 ulp).  Unlike the
// library exp2f/log2f they skip the denormal range fix-ups: results below 2^-126 come out
// as 0 and log of a denormal input as -inf, which is harmless where they are used (sums of
// probabilities whose terms below 2^-126 carry no weight).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// bf16 bits -> fp32 (exact)
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Wave-wide reductions on DPP lane moves (no LDS round trip): pairs within quads, the
// two halves of each 8-lane group, of each 16-lane row, then rows 0->1, 2->3 and 1->2,3
// by row broadcasts; lane 63 ends with the total, which is read back as a scalar so every
// lane returns it.  `id` is the identity filled into the rows a broadcast does not reach.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v, uint32_t id) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, CTRL, ROW_MASK, 0xf, false);
}
template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, uint32_t id, Op op) {
  v = op(v, dpp_u32<0xb1>(v, id));          // quad_perm [1,0,3,2]
  v = op(v, dpp_u32<0x4e>(v, id));          // quad_perm [2,3,0,1]
  v = op(v, dpp_u32<0x141>(v, id));         // row_half_mirror
  v = op(v, dpp_u32<0x140>(v, id));         // row_mirror
  v = op(v, dpp_u32<0x142, 0xa>(v, id));    // row_bcast:15
  v = op(v, dpp_u32<0x143, 0xc>(v, id));    // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ float wave_max(float v) {
  return __uint_as_float(wave_reduce_u32(__float_as_uint(v), 0xff800000u, [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }));
}
__device__ __forceinline__ float wave_sum(float v) {
  return __uint_as_float(wave_reduce_u32(__float_as_uint(v), 0u, [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}
__device__ __forceinline__ int wave_sum_i(int v) {
  return (int)wave_reduce_u32((uint32_t)v, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#define HK_U64_STEP(CTRL, RM)                                                                     \
  {                                                                                               \
    const unsigned long long t = ((unsigned long long)dpp_u32<CTRL, RM>(hi, 0u) << 32) |          \
                                 dpp_u32<CTRL, RM>(lo, 0u);                                       \
    const unsigned long long r = (((unsigned long long)hi << 32) | lo) + t;                       \
    lo = (uint32_t)r;                                                                             \
    hi = (uint32_t)(r >> 32);                                                                     \
  }
  HK_U64_STEP(0xb1, 0xf)
  HK_U64_STEP(0x4e, 0xf)
  HK_U64_STEP(0x141, 0xf)
  HK_U64_STEP(0x140, 0xf)
  HK_U64_STEP(0x142, 0xa)
  HK_U64_STEP(0x143, 0xc)
#undef HK_U64_STEP
  lo = (uint32_t)__builtin_amdgcn_readlane((int)lo, 63);
  hi = (uint32_t)__builtin_amdgcn_readlane((int)hi, 63);
  return ((unsigned long long)hi << 32) | lo;
}

// Block-wide reductions for blockDim.x = NT threads (multiple of 64).  `red` is LDS
// scratch of at least NT/64 elements; every thread gets the result.
template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, red[i]);
  return r;
}
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float r = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r += red[i];
  return r;
}
template <int NT>
__device__ __forceinline__ unsigned long long block_sum_u64(unsigned long long v,
                                                            unsigned long long* red) {
  v = wave_sum_u64(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  unsigned long long r = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r += red[i];
  return r;
}
template <int NT>
__device__ __forceinline__ int block_sum_int(int v, int* red) {
  v = wave_sum_i(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  int r = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) r += red[i];
  return r;
}

// Candidate predicate: slot j of a head is a candidate when j < cand_len and its page
// mask bit is set (mask row may be null: all slots valid).
__device__ __forceinline__ bool is_cand(const uint16_t* mask_row, int cand_len, int j) {
  if (j >= cand_len) return false;
  if (mask_row == nullptr) return true;
  return (mask_row[j >> 4] >> (j & 15)) & 1;
}

__device__ __forceinline__ int dense_pages(int L_dense) { return (L_dense + HK_PAGE - 1) / HK_PAGE; }

// Raise a kernel's dynamic-LDS limit above the 64 KB default.  The attribute is set only
// when a launch asks for more than any earlier one, so repeated launches (including ones a
// caller records into a graph) make no further API calls.
template <auto Kernel>
inline void allow_dynamic_lds(size_t bytes) {
  static std::atomic<size_t> granted{65536};
  size_t g = granted.load(std::memory_order_relaxed);
  if (bytes <= g) return;
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(Kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  while (g < bytes && !granted.compare_exchange_weak(g, bytes)) {
  }
}

// Records HIP events around one kernel launch on its stream while kernel timing is on
// (hk_timing_enable); construct right before the launch, let it go out of scope after.
class TimedLaunch {
 public:
  TimedLaunch(int kernel, hipStream_t st);
  ~TimedLaunch();
  TimedLaunch(const TimedLaunch&) = delete;
  TimedLaunch& operator=(const TimedLaunch&) = delete;

 private:
  int kernel_;
  hipStream_t st_;
  bool active_;
};

}  // namespace hk

// ---------------------------------------------------------------- launchers
// Each returns hipGetLastError() of its launches; arguments are validated by the C ABI.
struct hk_score_args {
  const void* q_obs;
  const hk_paged_kv* kv;
  int NS, Hq, Hkv, D, W;
  int L_dense;
  float sm_scale;
  const float* row_lse_in;
  float* row_lse_out;
  float* s_attn;
  int32_t* cand_len;
  const int32_t* ref_slots;
  int n_ref;
  float* x_red;
  void* ws;
};
hipError_t hk_launch_score(const hk_score_args& a, hipStream_t st);
size_t hk_score_ws(int NS, int Hq, int Hkv, int D, int W, int max_pages);
size_t hk_score_lds_bytes(int R, int D, int esize, bool redundancy);
hipError_t hk_launch_score_rows(int NS, int Hq, int Hkv, int D, int W, const void* q_obs,
                                const hk_paged_kv* kv, int L_dense, float sm_scale,
                                const float* row_lse, float* a_rows, hipStream_t st);

hipError_t hk_launch_vote_topp(int n_heads, int R, int S_max, const int32_t* cand_len,
                               const uint16_t* mask, const float* a_rows, int p_q, uint16_t* votes,
                               int32_t* row_k, uint32_t* row_sel, int32_t* status, hipStream_t st);
hipError_t hk_launch_budget_plan(int n_heads, int max_pages, const int32_t* n_pages,
                                 const uint16_t* mask, int L_dense, int L_lower, int L_upper,
                                 int32_t* head_mode, int32_t* k_cap, hipStream_t st);
hipError_t hk_launch_budget_select(int n_heads, int S_max, const int32_t* cand_len,
                                   const uint16_t* mask, const uint16_t* votes, const float* c,
                                   const uint32_t* sel_in, const int32_t* head_mode,
                                   const int32_t* k_cap, int n_sink, uint32_t* sel_out,
                                   int32_t* k_out, hipStream_t st);

hipError_t hk_launch_calibrate(int n_heads, int S_max, const int32_t* cand_len,
                               const uint16_t* mask, int n_metrics, const float* x0,
                               const float* x1, const float* T0, const float* T1, float w0,
                               float w1, float* c_out, float* lse_out, hipStream_t st);
hipError_t hk_launch_topp(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                          const float* c, int p_q, int k_min, int k_max, uint32_t* sel_bits,
                          int32_t* k_out, float* sel_mass, int32_t* status, hipStream_t st);
hipError_t hk_launch_calib_topp(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                                int n_metrics, const float* x0, const float* x1, const float* T0,
                                const float* T1, float w0, float w1, int p_q, int k_min, int k_max,
                                float* c_out, float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                                float* sel_mass, int32_t* status, hipStream_t st);
// the multi-workgroup selector (n_metrics = 0: Top-p of c_in alone)
size_t hk_select_wide_ws(int n_heads, int S_max);
hipError_t hk_launch_select_wide(int n_heads, int S_max, const int32_t* cand_len,
                                 const uint16_t* mask, int n_metrics, const float* x0,
                                 const float* x1, const float* T0, const float* T1, float w0,
                                 float w1, const float* c_in, int p_q, int k_min, int k_max,
                                 float* c_out, float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                                 float* sel_mass, int32_t* status, void* ws, hipStream_t st);
hipError_t hk_launch_pool_max(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                              const float* x, int radius, float* out, hipStream_t st);
hipError_t hk_launch_solve_T_gd(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                                const float* x, const int32_t* k, const float* target, float T_init,
                                float lr, int iters, float tol, float* T_out, float* loss_out,
                                hipStream_t st);
hipError_t hk_launch_solve_T(int n_heads, int S_max, const int32_t* cand_len,
                             const uint16_t* mask, const float* x, const int32_t* k,
                             const float* target, float T_lo, float T_hi, int iters,
                             float* T_out, hipStream_t st);

hipError_t hk_launch_compact(int n_heads, int D, const hk_paged_kv* kv, const uint32_t* sel_bits,
                             int L_dense, int L_sparse, const int32_t* head_mode,
                             const hk_allocator* alloc, int32_t* status, void* ws, hipStream_t st);
size_t hk_compact_ws(int n_heads, int max_pages);
hipError_t hk_launch_probe(int kind, int blocks, int iters, float* out, hipStream_t st);
hipError_t hk_launch_alloc_init(int32_t* free_ids, int32_t* free_top, int first_free, int n,
                                hipStream_t st);

hipError_t hk_launch_decode(int NS, int Hq, int Hkv, int D, const void* q, const hk_paged_kv* kv,
                            float sm_scale, float* o, float* lse, void* ws, hipStream_t st,
                            bool timed = true);
// the static scratch of hk_decode_attn_noalloc: its size, this device's address of it, and
// the bytes one call needs (the split partial states of the actual split)
#define HK_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
hipError_t hk_noalloc_scratch(void** ptr);
size_t hk_decode_noalloc_bytes(int NS, int Hq, int Hkv, int D, int max_pages);
size_t hk_decode_ws(int NS, int Hq, int Hkv, int D, int max_pages);
void hk_decode_split_plan(int n_heads, int max_pages, int* pps_out, int* n_split_out);

hipError_t hk_launch_append(int NS, int Hkv, int D, const hk_paged_kv* kv, const void* k_new,
                            const void* v_new, const hk_allocator* alloc, int32_t* status,
                            void* ws, hipStream_t st);
size_t hk_append_ws(int NS, int Hkv);

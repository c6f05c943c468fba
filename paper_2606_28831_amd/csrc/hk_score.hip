// a1: importance scoring of cached keys against the observation window (MFMA, gfx950).
//
// s[h][j] = log( (1/R) sum_r exp(z[r][j] - LSE_r) ),  z = sm_scale * q_r . k_j,
// LSE_r = log sum_{j valid} exp z[r][j]  (App. F attention; Reduce step of App. E applied
// to the raw attention distribution of Problem 1, Sec. 3.2).
//
// Two passes over K (pass 1 is skipped when the caller supplies the row LSEs, e.g. the
// decode step's own LSEs):
//   pass 1  per (head, page chunk): C[key][query] = K Q^T on MFMA 32x32, per-lane online
//           (max, sum exp) for the lane's query column, merged over lanes and waves;
//   merge   per (head, row): combine chunk partials into LSE_r;
//   pass 2  per (head, page chunk): C[query][key] = Q K^T on MFMA 32x32, per-lane column
//           sum of exp(z - LSE) over the window rows; optionally, on the same K fragment,
//           C[ref][key] = Kref K^T for the cosine-redundancy metric.
//
// Operand mapping.  For the 32-row MFMA operands (32x32x16 bf16, 32x32x2 f32) lane l
// supplies row (l % 32) and one half of the contraction range.  The contraction index
// is permuted so that lane l always works on dims [ (l/32) * D/2, (l/32+1) * D/2 ) of its
// row: step kk uses the next 8 (bf16) or 1 (f32) of them.  Q and K use the same
// permutation, so the dot products are unchanged, every lane reads one contiguous half
// row of its key (D/2 elements, 16-byte loads), and one fragment serves as either the
// A or the B operand.
// Accumulator layout of the 32x32 MFMA: register r of lane l holds row
// 8*(r/4) + 4*(l/32) + (r%4), column l % 32.
#include "hk_internal.h"

namespace hk {

template <typename T, int D>
struct Frag;

// bf16: D/16 steps of 8 bf16 per lane
template <int D>
struct Frag<uint16_t, D> {
  static constexpr int KSTEPS = D / 16;
  static constexpr int BYTES_PER_STEP = 16;
  bf16x8 v[KSTEPS];
  __device__ __forceinline__ void load(const uint16_t* row_half) {
    const uint4* p = reinterpret_cast<const uint4*>(row_half);
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      uint4 u = p[kk];
      v[kk] = __builtin_bit_cast(bf16x8, u);
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) v[kk] = __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
  }
  __device__ __forceinline__ float sumsq() const {
    float s = 0.f;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      uint4 u = __builtin_bit_cast(uint4, v[kk]);
      uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float a = bf16_lo(w[i]), b = bf16_hi(w[i]);
        s = fmaf(a, a, s);
        s = fmaf(b, b, s);
      }
    }
    return s;
  }
  static __device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  // LDS fragment element for step kk
  static __device__ __forceinline__ bf16x8 lds(const char* base, int qb, int kk, int lane) {
    return *reinterpret_cast<const bf16x8*>(base + ((size_t)(qb * KSTEPS + kk) * 64 + lane) * 16);
  }
};

// f32: D/2 steps of 1 float per lane
template <int D>
struct Frag<float, D> {
  static constexpr int KSTEPS = D / 2;
  static constexpr int BYTES_PER_STEP = 4;
  float v[KSTEPS];
  __device__ __forceinline__ void load(const float* row_half) {
    const float4* p = reinterpret_cast<const float4*>(row_half);
#pragma unroll
    for (int i = 0; i < KSTEPS / 4; ++i) {
      float4 u = p[i];
      v[4 * i + 0] = u.x;
      v[4 * i + 1] = u.y;
      v[4 * i + 2] = u.z;
      v[4 * i + 3] = u.w;
    }
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) v[kk] = 0.f;
  }
  __device__ __forceinline__ float sumsq() const {
    float s = 0.f;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) s = fmaf(v[kk], v[kk], s);
    return s;
  }
  static __device__ __forceinline__ f32x16 mma(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ float lds(const char* base, int qb, int kk, int lane) {
    return *reinterpret_cast<const float*>(base + ((size_t)(qb * KSTEPS + kk) * 64 + lane) * 4);
  }
};

__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// Stage R rows of D elements into LDS in fragment-major order [blk][kk][lane].
// `row_ptr(r)` gives the global address of row r (< R) or nullptr (zero row).
template <typename T, int D, typename RowFn>
__device__ __forceinline__ void stage_rows(char* lds, int R, int R_pad, RowFn row_ptr) {
  using F = Frag<T, D>;
  constexpr int VEC = 16 / sizeof(T);          // elements per 16-byte chunk
  constexpr int CPR = D / VEC;                 // chunks per row
  constexpr int HALF = D / 2;
  for (int c = threadIdx.x; c < R_pad * CPR; c += blockDim.x) {
    const int r = c / CPR, ch = c % CPR;
    const T* src = (r < R) ? row_ptr(r) : nullptr;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (src) u = *reinterpret_cast<const uint4*>(src + ch * VEC);
    const int e0 = ch * VEC;
    const int half = e0 / HALF, off = e0 % HALF;
    const int lane = half * 32 + (r & 31), blk = r >> 5;
    if constexpr (sizeof(T) == 2) {
      const int kk = off / 8;
      *reinterpret_cast<uint4*>(lds + ((size_t)(blk * F::KSTEPS + kk) * 64 + lane) * 16) = u;
    } else {
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<uint32_t*>(lds + ((size_t)(blk * F::KSTEPS + off + i) * 64 + lane) * 4) = w[i];
    }
  }
}

constexpr int QB_MAX = 8;   // R_pad <= 256
constexpr int SCORE_NT = 256;

// ------------------------------------------------------------------ pass 1
template <typename T, int D>
__global__ __launch_bounds__(SCORE_NT) void score_pass1_kernel(
    const T* __restrict__ q_obs, const T* __restrict__ k_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const int32_t* __restrict__ n_pages_arr, int NS, int Hq,
    int Hkv, int W, int max_pages, int ppw, float c2, float2* __restrict__ part, int n_chunks) {
  using F = Frag<T, D>;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W, R_pad = (R + 31) & ~31, QB = R_pad >> 5;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  stage_rows<T, D>(smem, R, R_pad, [&](int r) -> const T* {
    const int w = r / G, g = r % G;
    return q_obs + ((size_t)(w * NS + s) * Hq + kv * G + g) * D;
  });
  float2* red = reinterpret_cast<float2*>(smem + (size_t)R_pad * D * sizeof(T));
  __syncthreads();

  const int n = n_pages_arr[h];
  const int p_begin = chunk * ppw, p_end = min(p_begin + ppw, n);
  float M[QB_MAX], L[QB_MAX];
#pragma unroll
  for (int q = 0; q < QB_MAX; ++q) { M[q] = -INFINITY; L[q] = 0.f; }

  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  for (int p0 = p_begin + 2 * wave; p0 < p_end; p0 += 2 * (SCORE_NT / 64)) {
    const int p1 = p0 + 1;
    const uint32_t m0 = mrow[p0], m1 = (p1 < p_end) ? mrow[p1] : 0u;
    const uint32_t tmask = m0 | (m1 << 16);
    if (tmask == 0) continue;
    const int kl = lane & 31, pg = p0 + (kl >> 4);
    F kf;
    if (pg < p_end) {
      const int phys = trow[pg];
      kf.load(k_pool + ((size_t)phys * HK_PAGE + (kl & 15)) * D + (lane >> 5) * (D / 2));
    } else {
      kf.zero();
    }
    const bool full = (tmask == 0xffffffffu);
#pragma unroll
    for (int qb = 0; qb < QB_MAX; ++qb) {
      if (qb < QB) {
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < F::KSTEPS; ++kk) acc = F::mma(kf.v[kk], F::lds(smem, qb, kk, lane), acc);
        float m = -INFINITY;
        if (full) {
#pragma unroll
          for (int r = 0; r < 16; ++r) m = fmaxf(m, acc[r]);
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if ((tmask >> acc_row(r, lane)) & 1u) m = fmaxf(m, acc[r]);
        }
        const float mn = fmaxf(M[qb], m);
        if (mn == -INFINITY) continue;   // nothing valid seen yet in this column
        const float mc = mn * c2;
        float sum = 0.f;
        if (full) {
#pragma unroll
          for (int r = 0; r < 16; ++r) sum += exp2f(fmaf(acc[r], c2, -mc));
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if ((tmask >> acc_row(r, lane)) & 1u) sum += exp2f(fmaf(acc[r], c2, -mc));
        }
        L[qb] = L[qb] * exp2f((M[qb] - mn) * c2) + sum;
        M[qb] = mn;
      }
    }
  }
  // merge lane halves (same query column), then waves
#pragma unroll
  for (int qb = 0; qb < QB_MAX; ++qb) {
    if (qb < QB) {
      const float Mo = __shfl_xor(M[qb], 32, 64), Lo = __shfl_xor(L[qb], 32, 64);
      const float mn = fmaxf(M[qb], Mo);
      float Ln = 0.f;
      if (mn != -INFINITY) Ln = L[qb] * exp2f((M[qb] - mn) * c2) + Lo * exp2f((Mo - mn) * c2);
      if (lane < 32) red[wave * R_pad + qb * 32 + lane] = make_float2(mn, Ln);
    }
  }
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += SCORE_NT) {
    float mn = -INFINITY;
    for (int w = 0; w < SCORE_NT / 64; ++w) mn = fmaxf(mn, red[w * R_pad + r].x);
    float Ln = 0.f;
    if (mn != -INFINITY)
      for (int w = 0; w < SCORE_NT / 64; ++w) {
        const float2 v = red[w * R_pad + r];
        Ln += v.y * exp2f((v.x - mn) * c2);
      }
    part[((size_t)h * n_chunks + chunk) * R_pad + r] = make_float2(mn, Ln);
  }
}

// merge chunk partials into natural-log row LSE, layout [W][NS][Hq]
__global__ __launch_bounds__(256) void score_lse_merge_kernel(const float2* __restrict__ part,
                                                               int n_chunks, int NS, int Hq,
                                                               int Hkv, int W, float c2,
                                                               float sm_scale, float* lse_out) {
  const int h = blockIdx.x, s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W, R_pad = (R + 31) & ~31;
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    const float2* p = part + (size_t)h * n_chunks * R_pad + r;
    float mn = -INFINITY;
    for (int c = 0; c < n_chunks; ++c) mn = fmaxf(mn, p[(size_t)c * R_pad].x);
    float L = 0.f;
    if (mn != -INFINITY)
      for (int c = 0; c < n_chunks; ++c) {
        const float2 v = p[(size_t)c * R_pad];
        L += v.y * exp2f((v.x - mn) * c2);
      }
    const float lse = (mn == -INFINITY) ? -INFINITY : fmaf(mn, sm_scale, logf(L));
    const int w = r / G, g = r % G;
    lse_out[((size_t)w * NS + s) * Hq + kv * G + g] = lse;
  }
}

constexpr int NREF_MAX = 256;

// ------------------------------------------------------------------ pass 2
template <typename T, int D, bool RED>
__global__ __launch_bounds__(SCORE_NT) void score_pass2_kernel(
    const T* __restrict__ q_obs, const T* __restrict__ k_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const int32_t* __restrict__ n_pages_arr, int NS, int Hq,
    int Hkv, int W, int max_pages, int ppw, int L_dense, float c2, float lnR,
    const float* __restrict__ row_lse, float* __restrict__ s_out, int32_t* __restrict__ cand_len_out,
    const int32_t* __restrict__ ref_slots, int n_ref, float* __restrict__ x_red) {
  using F = Frag<T, D>;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W, R_pad = (R + 31) & ~31, QB = R_pad >> 5;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t S_max = (size_t)max_pages * HK_PAGE;
  const int n = n_pages_arr[h];
  const int cand_len = HK_PAGE * max(0, n - dense_pages(L_dense));
  if (chunk == 0 && threadIdx.x == 0) cand_len_out[h] = cand_len;

  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  const int p_begin = chunk * ppw, p_end_all = min(p_begin + ppw, max_pages);
  const int p_cand_end = min(p_end_all, cand_len / HK_PAGE);

  // slots of this chunk that hold no candidate: -inf
  {
    const int j0 = max(p_cand_end, p_begin) * HK_PAGE, j1 = p_end_all * HK_PAGE;
    for (int j = j0 + threadIdx.x; j < j1; j += SCORE_NT) {
      s_out[(size_t)h * S_max + j] = -INFINITY;
      if (RED) x_red[(size_t)h * S_max + j] = -INFINITY;
    }
  }
  if (p_begin >= p_cand_end) return;

  stage_rows<T, D>(smem, R, R_pad, [&](int r) -> const T* {
    const int w = r / G, g = r % G;
    return q_obs + ((size_t)(w * NS + s) * Hq + kv * G + g) * D;
  });
  char* after_q = smem + (size_t)R_pad * D * sizeof(T);
  float* lse2 = reinterpret_cast<float*>(after_q);                 // [R_pad], log2 units
  for (int r = threadIdx.x; r < R_pad; r += SCORE_NT) {
    float v = INFINITY;                                            // padding rows weigh 0
    if (r < R) {
      const int w = r / G, g = r % G;
      v = row_lse[((size_t)w * NS + s) * Hq + kv * G + g] * kLog2e;
    }
    lse2[r] = v;
  }
  char* ref_lds = after_q + (size_t)R_pad * sizeof(float);
  float* rn_ref = nullptr;
  int32_t* ref_slot = nullptr;
  int RB = 0;
  if constexpr (RED) {
    const int nr_pad = (n_ref + 31) & ~31;
    RB = nr_pad >> 5;
    rn_ref = reinterpret_cast<float*>(ref_lds + (size_t)NREF_MAX * D * sizeof(T));
    ref_slot = reinterpret_cast<int32_t*>(rn_ref + NREF_MAX);
    const int32_t* rs = ref_slots + (size_t)h * n_ref;
    auto ref_row = [&](int i) -> const T* {
      const int j = rs[i];
      const int pp = j >> 4;
      if (j < 0 || pp >= n) return nullptr;
      return k_pool + ((size_t)trow[pp] * HK_PAGE + (j & 15)) * D;
    };
    stage_rows<T, D>(ref_lds, n_ref, nr_pad, ref_row);
    __syncthreads();
    for (int i = threadIdx.x; i < nr_pad; i += SCORE_NT) {
      // squared norm of reference row i, read back from its fragment-major LDS image
      float ss = 0.f;
      for (int half = 0; half < 2; ++half) {
        const int ln = half * 32 + (i & 31);
#pragma unroll
        for (int kk = 0; kk < F::KSTEPS; ++kk) {
          if constexpr (sizeof(T) == 2) {
            const uint4 u = *reinterpret_cast<const uint4*>(
                ref_lds + ((size_t)((i >> 5) * F::KSTEPS + kk) * 64 + ln) * 16);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float a0 = bf16_lo(w4[e]), a1 = bf16_hi(w4[e]);
              ss = fmaf(a0, a0, ss);
              ss = fmaf(a1, a1, ss);
            }
          } else {
            const float x = *reinterpret_cast<const float*>(
                ref_lds + ((size_t)((i >> 5) * F::KSTEPS + kk) * 64 + ln) * 4);
            ss = fmaf(x, x, ss);
          }
        }
      }
      rn_ref[i] = ss > 0.f ? 1.0f / sqrtf(ss) : 0.f;
      ref_slot[i] = (i < n_ref) ? rs[i] : -1;
    }
  }
  __syncthreads();

  for (int p0 = p_begin + 2 * wave; p0 < p_cand_end; p0 += 2 * (SCORE_NT / 64)) {
    const int p1 = p0 + 1;
    const uint32_t m0 = mrow[p0], m1 = (p1 < p_cand_end) ? mrow[p1] : 0u;
    const int kl = lane & 31, pg = p0 + (kl >> 4);
    const int slot = pg * HK_PAGE + (kl & 15);
    const bool cand = (pg < p_cand_end) && (((kl < 16 ? m0 : m1) >> (kl & 15)) & 1u);
    if ((m0 | m1) == 0) {
      if (lane < 32 && pg < p_cand_end) {
        s_out[(size_t)h * S_max + slot] = -INFINITY;
        if (RED) x_red[(size_t)h * S_max + slot] = -INFINITY;
      }
      continue;
    }
    F kf;
    if (pg < p_cand_end) {
      const int phys = trow[pg];
      kf.load(k_pool + ((size_t)phys * HK_PAGE + (kl & 15)) * D + (lane >> 5) * (D / 2));
    } else {
      kf.zero();
    }
    float col = 0.f;
#pragma unroll
    for (int qb = 0; qb < QB_MAX; ++qb) {
      if (qb < QB) {
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < F::KSTEPS; ++kk) acc = F::mma(F::lds(smem, qb, kk, lane), kf.v[kk], acc);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2 + qb * 32 + 8 * r4 + 4 * (lane >> 5));
#pragma unroll
          for (int i = 0; i < 4; ++i) col += exp2f(fmaf(acc[4 * r4 + i], c2, -l4[i]));
        }
      }
    }
    col += __shfl_xor(col, 32, 64);
    if constexpr (RED) {
      const float ss = kf.sumsq();
      const float nrm2 = ss + __shfl_xor(ss, 32, 64);
      const float rn = nrm2 > 0.f ? 1.0f / sqrtf(nrm2) : 0.f;
      float cmax = -INFINITY;
      int self = 0;
      for (int rb = 0; rb < RB; ++rb) {
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < F::KSTEPS; ++kk) acc = F::mma(F::lds(ref_lds, rb, kk, lane), kf.v[kk], acc);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = rb * 32 + acc_row(r, lane);
          if (i < n_ref) {
            if (ref_slot[i] == slot) self = 1;
            else cmax = fmaxf(cmax, acc[r] * rn_ref[i]);
          }
        }
      }
      cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
      self |= __shfl_xor(self, 32, 64);
      if (lane < 32 && pg < p_cand_end) {
        float x = -INFINITY;
        if (cand) x = (n_ref - self > 0) ? -(cmax * rn) : 1.0f;
        x_red[(size_t)h * S_max + slot] = x;
      }
    }
    if (lane < 32 && pg < p_cand_end)
      s_out[(size_t)h * S_max + slot] = cand ? fmaf(__log2f(col), kLn2, -lnR) : -INFINITY;
  }
}

template <typename K>
static void allow_lds(K kernel, size_t bytes) {
  if (bytes > 65536) hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

template <typename T, int D>
hipError_t launch_score_t(const hk_score_args& a, hipStream_t st) {
  const hk_paged_kv* kv = a.kv;
  const int G = a.Hq / a.Hkv, R = G * a.W, R_pad = (R + 31) & ~31;
  const int n_heads = a.NS * a.Hkv;
  const int ppw = 64;
  const int n_chunks = (kv->max_pages + ppw - 1) / ppw;
  const float c2 = a.sm_scale * kLog2e;
  char* ws = static_cast<char*>(a.ws);
  float2* part = reinterpret_cast<float2*>(ws);
  float* lse_buf = a.row_lse_out;
  size_t off = ((size_t)n_heads * n_chunks * R_pad * sizeof(float2) + 255) & ~(size_t)255;
  if (!lse_buf) lse_buf = reinterpret_cast<float*>(ws + off);
  const float* lse_use = a.row_lse_in;
  dim3 grid(n_chunks, n_heads);
  if (!lse_use) {
    const size_t lds1 = (size_t)R_pad * D * sizeof(T) + (size_t)(SCORE_NT / 64) * R_pad * sizeof(float2);
    allow_lds(score_pass1_kernel<T, D>, lds1);
    hipLaunchKernelGGL((score_pass1_kernel<T, D>), grid, dim3(SCORE_NT), lds1, st,
                       static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                       kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                       kv->max_pages, ppw, c2, part, n_chunks);
    hipLaunchKernelGGL(score_lse_merge_kernel, dim3(n_heads), dim3(256), 0, st, part, n_chunks,
                       a.NS, a.Hq, a.Hkv, a.W, c2, a.sm_scale, lse_buf);
    lse_use = lse_buf;
  } else if (a.row_lse_out && a.row_lse_out != a.row_lse_in) {
    hipMemcpyAsync(a.row_lse_out, a.row_lse_in, sizeof(float) * (size_t)a.W * a.NS * a.Hq,
                   hipMemcpyDeviceToDevice, st);
  }
  const float lnR = logf((float)R);
  size_t lds2 = (size_t)R_pad * D * sizeof(T) + (size_t)R_pad * sizeof(float);
  if (a.x_red) {
    lds2 += (size_t)NREF_MAX * D * sizeof(T) + (size_t)NREF_MAX * (sizeof(float) + sizeof(int32_t));
    allow_lds(score_pass2_kernel<T, D, true>, lds2);
    hipLaunchKernelGGL((score_pass2_kernel<T, D, true>), grid, dim3(SCORE_NT), lds2, st,
                       static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                       kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                       kv->max_pages, ppw, a.L_dense, c2, lnR, lse_use, a.s_attn, a.cand_len,
                       a.ref_slots, a.n_ref, a.x_red);
  } else {
    allow_lds(score_pass2_kernel<T, D, false>, lds2);
    hipLaunchKernelGGL((score_pass2_kernel<T, D, false>), grid, dim3(SCORE_NT), lds2, st,
                       static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                       kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                       kv->max_pages, ppw, a.L_dense, c2, lnR, lse_use, a.s_attn, a.cand_len,
                       nullptr, 0, nullptr);
  }
  return hipGetLastError();
}

}  // namespace hk

size_t hk_score_ws(int NS, int Hq, int Hkv, int D, int W, int max_pages) {
  (void)D;
  const int G = Hq / Hkv, R_pad = (G * W + 31) & ~31;
  const int n_chunks = (max_pages + 63) / 64;
  const size_t part = ((size_t)NS * Hkv * n_chunks * R_pad * sizeof(float2) + 255) & ~(size_t)255;
  const size_t lse = ((size_t)W * NS * Hq * sizeof(float) + 255) & ~(size_t)255;
  return part + lse;
}

size_t hk_score_lds_bytes(int R, int D, int esize, bool redundancy) {
  const size_t R_pad = (size_t)((R + 31) & ~31);
  const size_t p1 = R_pad * D * esize + (size_t)(hk::SCORE_NT / 64) * R_pad * 8;
  size_t p2 = R_pad * D * esize + R_pad * 4;
  if (redundancy) p2 += (size_t)hk::NREF_MAX * D * esize + (size_t)hk::NREF_MAX * 8;
  return p1 > p2 ? p1 : p2;
}

hipError_t hk_launch_score(const hk_score_args& a, hipStream_t st) {
  const bool bf = a.kv->dtype == HK_BF16;
  if (bf && a.D == 128) return hk::launch_score_t<uint16_t, 128>(a, st);
  if (bf && a.D == 64) return hk::launch_score_t<uint16_t, 64>(a, st);
  if (!bf && a.D == 128) return hk::launch_score_t<float, 128>(a, st);
  return hk::launch_score_t<float, 64>(a, st);
}

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
// supplies row (l % 32) and one half of each contraction step.  bf16 keeps the natural
// k-order: step kk covers dims [16 kk, 16 kk + 16), lanes l < 32 the first 8 and lanes
// l >= 32 the next 8, so the two lanes of a row read adjacent 16-byte pieces.  f32
// permutes the contraction index so that lane l works on dims [ (l/32) * D/2,
// (l/32+1) * D/2 ) of its row, one per step, and reads one contiguous half row.  Q and
// K use the same order, so the dot products are unchanged and one fragment serves as
// either the A or the B operand.
// Accumulator layout of the 32x32 MFMA: register r of lane l holds row
// 8*(r/4) + 4*(l/32) + (r%4), column l % 32.
#include <type_traits>

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
  // natural MFMA k-order: step kk covers dims [16 kk, 16 kk + 16), lanes l < 32 the first
  // 8 and lanes l >= 32 the next 8, so the two lanes of a key read 32 contiguous bytes
  __device__ __forceinline__ void load(const uint16_t* row, int half) {
    const uint4* p = reinterpret_cast<const uint4*>(row + half * 8);
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      uint4 u = p[2 * kk];
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
  // permuted k-order: lane l covers dims [(l/32) D/2, (l/32 + 1) D/2), one element per
  // step, so each lane loads its half row with 16-byte loads
  __device__ __forceinline__ void load(const float* row, int half) {
    const float4* p = reinterpret_cast<const float4*>(row + half * (D / 2));
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
    const int blk = r >> 5;
    if constexpr (sizeof(T) == 2) {
      const int kk = e0 / 16, lane = ((e0 / 8) & 1) * 32 + (r & 31);     // natural k-order
      *reinterpret_cast<uint4*>(lds + ((size_t)(blk * F::KSTEPS + kk) * 64 + lane) * 16) = u;
    } else {
      const int half = e0 / HALF, off = e0 % HALF;                       // permuted k-order
      const int lane = half * 32 + (r & 31);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<uint32_t*>(lds + ((size_t)(blk * F::KSTEPS + off + i) * 64 + lane) * 4) = w[i];
    }
  }
}

constexpr int SCORE_NT = 512;              // threads per workgroup
constexpr int SCORE_QD = 2;                // Q fragments read from LDS this many MFMA steps ahead
constexpr int SCORE_NW = SCORE_NT / 64;
constexpr int SCORE_PPW = 128;             // pages per workgroup
constexpr int SCORE_KT = 1;                // 32-key tiles a wave holds at once
constexpr int SCORE_WPP = 2 * SCORE_KT;    // pages per wave iteration
constexpr int NREF_MAX = 256;

// Query blocks of 32 rows are a compile-time count; other counts round up to the next
// instantiated one (the extra rows are zero and carry no weight).
__host__ __device__ constexpr int qb_eff(int qb) {
  return qb <= 1 ? 1 : qb <= 2 ? 2 : qb <= 4 ? 4 : qb <= 7 ? 7 : 8;
}
__host__ __device__ constexpr int score_rpad(int R) { return 32 * qb_eff((R + 31) / 32); }

// MFMA chain of one 32x32 output block over the whole head dimension.  LDS_IS_A: the
// LDS block is the A operand (rows of C), the register fragment the B operand.
template <typename F, bool LDS_IS_A>
__device__ __forceinline__ f32x16 mma_chain(const F& kf, const char* lds, int blk, int lane) {
  f32x16 acc = {};
#pragma unroll
  for (int kk = 0; kk < F::KSTEPS; ++kk) {
    if constexpr (LDS_IS_A) acc = F::mma(F::lds(lds, blk, kk, lane), kf.v[kk], acc);
    else acc = F::mma(kf.v[kk], F::lds(lds, blk, kk, lane), acc);
  }
  return acc;
}

// KT interleaved chains sharing each LDS operand read (KT register fragments).
template <typename F, bool LDS_IS_A, int KT>
__device__ __forceinline__ void mma_chains(const F* kf, const char* lds, int blk, int lane,
                                           f32x16* acc) {
#pragma unroll
  for (int t = 0; t < KT; ++t) acc[t] = f32x16{};
#pragma unroll
  for (int kk = 0; kk < F::KSTEPS; ++kk) {
    const auto op = F::lds(lds, blk, kk, lane);
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      if constexpr (LDS_IS_A) acc[t] = F::mma(op, kf[t].v[kk], acc[t]);
      else acc[t] = F::mma(kf[t].v[kk], op, acc[t]);
    }
  }
}

// ---------------------------------------------------------------------------------
// Software-pipelined full tiles (KT = 1).  Within one wave the MFMAs of query block qb
// are interleaved with the VALU work on block qb-1 (independent data), and each LDS
// fragment is read two MFMA steps before its use.  MFMA and VALU work of one wave overlap
// on the SIMD; split across different waves they do not, which is why the interleave is
// made explicit here and pinned with scheduling-group barriers.
template <typename F>
using lds_frag_t = decltype(F::lds(nullptr, 0, 0, 0));

// Maximum of MFMA results.  fmaxf must quiet signalling NaNs first, which costs one
// canonicalising v_max per operand that the compiler cannot prove canonical (every MFMA
// result); the NaN-propagating maximum (v_maximum3_f32 on gfx950) needs none.  A NaN
// score propagates either way, through the exponential sum.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

template <int N_MFMA, int N_VALU>
__device__ __forceinline__ void sched_step() {
  __builtin_amdgcn_sched_group_barrier(0x008, N_MFMA, 0);   // MFMA
  __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);        // one LDS read
  __builtin_amdgcn_sched_group_barrier(0x002, N_VALU, 0);   // VALU work
}

// pass 2: adds to col[t] this lane's partial column sum  sum_r exp2(c2*z[r][key] - lse2[r])
// for each of the KT key tiles; every Q fragment read from LDS feeds KT MFMAs.
template <typename F, int QB, int KT>
__device__ __forceinline__ void p2_tile_pipelined(const F* kf, const char* qlds, const float* lse2,
                                                  float c2, int lane, float* col) {
  constexpr int KS = F::KSTEPS;
  constexpr int NF = QB * KS;
  lds_frag_t<F> qf[SCORE_QD + 1];
#pragma unroll
  for (int g = 0; g < SCORE_QD && g < NF; ++g) qf[g] = F::lds(qlds, g / KS, g % KS, lane);
  f32x16 acc[2][KT];
#pragma unroll
  for (int qb = 0; qb <= QB; ++qb) {
    f32x4 l4[4];
    if (qb >= 1) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        l4[r4] = *reinterpret_cast<const f32x4*>(lse2 + (qb - 1) * 32 + 8 * r4 + 4 * (lane >> 5));
    }
    if (qb < QB) {
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[qb & 1][t] = f32x16{};
    }
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int g = qb * KS + kk;
      if (qb < QB) {
#pragma unroll
        for (int t = 0; t < KT; ++t) acc[qb & 1][t] = F::mma(qf[g % (SCORE_QD + 1)], kf[t].v[kk], acc[qb & 1][t]);
        if (g + SCORE_QD < NF)
          qf[(g + SCORE_QD) % (SCORE_QD + 1)] = F::lds(qlds, (g + SCORE_QD) / KS, (g + SCORE_QD) % KS, lane);
      }
      if (qb >= 1) {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (e * KS / 16 == kk) {
#pragma unroll
            for (int t = 0; t < KT; ++t)
              col[t] += fast_exp2(fmaf(acc[(qb - 1) & 1][t][e], c2, -l4[e >> 2][e & 3]));
          }
      }
    }
    if constexpr (sizeof(lds_frag_t<F>) == 16) {
      if (qb >= 1 && qb < QB) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sched_step<KT, 3 * 16 * KT / KS>();
      }
    }
  }
}

// per-row probabilities of one full tile (every row valid): stores the clamped
// exp2(c2*z[r][key] - lse2[r]) of each row r (0 at a non-candidate slot), the MFMAs of
// block qb interleaved with the exponentials and stores of block qb-1.  A row's place
// in the output is uniform across the wave for a given accumulator register, so the
// stores are buffer stores with the lane's column in the vector offset and the row's
// offset in a scalar one: no per-store address arithmetic.
template <typename F, int QB>
__device__ __forceinline__ void rows_tile_pipelined(const F& kf, const char* qlds, const float* lse2,
                                                    float c2, int lane, bool cand,
                                                    __amdgpu_buffer_rsrc_t out, uint32_t voff,
                                                    uint32_t row_bytes) {
  constexpr int KS = F::KSTEPS;
  constexpr int NF = QB * KS;
  lds_frag_t<F> qf[SCORE_QD + 1];
#pragma unroll
  for (int g = 0; g < SCORE_QD && g < NF; ++g) qf[g] = F::lds(qlds, g / KS, g % KS, lane);
  f32x16 acc[2];
#pragma unroll
  for (int qb = 0; qb <= QB; ++qb) {
    f32x4 l4[4];
    if (qb >= 1) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        l4[r4] = *reinterpret_cast<const f32x4*>(lse2 + (qb - 1) * 32 + 8 * r4 + 4 * (lane >> 5));
    }
    if (qb < QB) acc[qb & 1] = f32x16{};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int g = qb * KS + kk;
      if (qb < QB) {
        acc[qb & 1] = F::mma(qf[g % (SCORE_QD + 1)], kf.v[kk], acc[qb & 1]);
        if (g + SCORE_QD < NF)
          qf[(g + SCORE_QD) % (SCORE_QD + 1)] = F::lds(qlds, (g + SCORE_QD) / KS, (g + SCORE_QD) % KS, lane);
      }
      if (qb >= 1) {
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (e * KS / 16 == kk) {
            // a probability: rounding in exp and in LSE can put the largest a hair above 1
            const float a = fminf(fast_exp2(fmaf(acc[(qb - 1) & 1][e], c2, -l4[e >> 2][e & 3])), 1.0f);
            const int row = (qb - 1) * 32 + 8 * (e >> 2) + (e & 3);   // + 4 (lane / 32) in voff
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(cand ? a : 0.f), out, (int)voff,
                                                  (int)(row * row_bytes), 2 /* nontemporal */);
          }
      }
    }
    if constexpr (sizeof(lds_frag_t<F>) == 16) {
      if (qb >= 1 && qb < QB) {
        // per MFMA step: one MFMA, one LDS read, two rows' exponentials and their stores
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                 // LDS read
          __builtin_amdgcn_sched_group_barrier(0x002, 4 * 16 / KS, 0);       // VALU
          __builtin_amdgcn_sched_group_barrier(0x040, 16 / KS, 0);           // VMEM write
        }
      }
    }
  }
}

// pass 1: online (max, sum exp2) update of the lane's query column for every block, over
// KT key tiles; every Q fragment read from LDS feeds KT MFMAs.
template <typename F, int QB, int KT>
__device__ __forceinline__ void p1_tile_pipelined(const F* kf, const char* qlds, float c2, int lane,
                                                  float* M, float* L) {
  constexpr int KS = F::KSTEPS;
  constexpr int NF = QB * KS;
  lds_frag_t<F> qf[SCORE_QD + 1];
#pragma unroll
  for (int g = 0; g < SCORE_QD && g < NF; ++g) qf[g] = F::lds(qlds, g / KS, g % KS, lane);
  f32x16 acc[2][KT];
#pragma unroll
  for (int qb = 0; qb <= QB; ++qb) {
    if (qb < QB) {
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[qb & 1][t] = f32x16{};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int g = qb * KS + kk;
#pragma unroll
        for (int t = 0; t < KT; ++t) acc[qb & 1][t] = F::mma(kf[t].v[kk], qf[g % (SCORE_QD + 1)], acc[qb & 1][t]);
        if (g + SCORE_QD < NF)
          qf[(g + SCORE_QD) % (SCORE_QD + 1)] = F::lds(qlds, (g + SCORE_QD) / KS, (g + SCORE_QD) % KS, lane);
      }
    }
    if (qb >= 1) {
      const f32x16* a = acc[(qb - 1) & 1];
      // maximum over the KT * 16 values, three at a time
      float mt[KT];
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        float m0 = vmax(vmax(a[t][0], a[t][1]), a[t][2]), m1 = vmax(vmax(a[t][3], a[t][4]), a[t][5]);
        float m2 = vmax(vmax(a[t][6], a[t][7]), a[t][8]), m3 = vmax(vmax(a[t][9], a[t][10]), a[t][11]);
        float m4 = vmax(vmax(a[t][12], a[t][13]), a[t][14]);
        m0 = vmax(vmax(m0, m1), m2);
        m3 = vmax(vmax(m3, m4), a[t][15]);
        mt[t] = vmax(m0, m3);
      }
      float mn = M[qb - 1];
#pragma unroll
      for (int t = 0; t < KT; ++t) mn = vmax(mn, mt[t]);
      const float mc = mn * c2;
      float s0 = fast_exp2(fmaf(a[0][0], c2, -mc)), s1 = fast_exp2(fmaf(a[0][1], c2, -mc));
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int r = (t == 0 ? 2 : 0); r < 16; r += 2) {
          s0 += fast_exp2(fmaf(a[t][r], c2, -mc));
          s1 += fast_exp2(fmaf(a[t][r + 1], c2, -mc));
        }
      L[qb - 1] = fmaf(L[qb - 1], fast_exp2((M[qb - 1] - mn) * c2), s0 + s1);
      M[qb - 1] = mn;
    }
    if constexpr (sizeof(lds_frag_t<F>) == 16) {
      if (qb >= 1 && qb < QB) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sched_step<KT, (16 * 3 * KT + 22) / KS>();
      }
    }
  }
}

// Redundancy of one 32-key tile: the lane's running maximum over the reference blocks of
// cos-numerator * 1/|ref| (C[ref][key], refs as rows).  The MFMA chain of block rb+1 is
// interleaved with the maximum over block rb.  check_self: some reference of this tile's
// pages is one of its keys; that reference is then skipped for that key and `self` set.
template <typename F>
__device__ __forceinline__ void red_tile_max(const F& kf, const char* ref_lds, const float* rn_ref,
                                             const int32_t* ref_slot, int RB, int lane, int slot,
                                             bool check_self, float& cmax, int& self) {
  constexpr int KS = F::KSTEPS;
  if (RB <= 0) return;
  f32x16 cur = mma_chain<F, true>(kf, ref_lds, 0, lane);
  for (int rb = 0; rb < RB; ++rb) {
    const bool more = rb + 1 < RB;
    f32x16 nxt = {};
    f32x4 rn4[4];
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4)
      rn4[r4] = *reinterpret_cast<const f32x4*>(rn_ref + rb * 32 + 8 * r4 + 4 * (lane >> 5));
    if (!check_self) {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        if (more) nxt = F::mma(F::lds(ref_lds, rb + 1, kk, lane), kf.v[kk], nxt);
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (e * KS / 16 == kk) cmax = vmax(cmax, cur[e] * rn4[e >> 2][e & 3]);
      }
      if constexpr (sizeof(lds_frag_t<F>) == 16) {
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) sched_step<1, 2 * 16 / KS>();
      }
    } else {
      if (more) nxt = mma_chain<F, true>(kf, ref_lds, rb + 1, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = rb * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (ref_slot[i] == slot) self = 1;
        else cmax = vmax(cmax, cur[e] * rn4[e >> 2][e & 3]);
      }
    }
    cur = nxt;
  }
}

// K fragment of the tile at page p0 (2 pages = 32 keys); lanes past p_end get zeros.
template <typename T, int D>
__device__ __forceinline__ void load_tile(Frag<T, D>& kf, const T* __restrict__ k_pool,
                                          const int32_t* __restrict__ trow, int p0, int p_end,
                                          int lane) {
  const int kl = lane & 31, pg = p0 + (kl >> 4);
  if (pg < p_end) {
    const int phys = trow[pg];
    kf.load(k_pool + ((size_t)phys * HK_PAGE + (kl & 15)) * D, lane >> 5);
  } else {
    kf.zero();
  }
}

// validity of the 16 accumulator rows a lane holds, from the tile's 32-slot mask
__device__ __forceinline__ uint32_t lane_rows(uint32_t tmask, int lane) {
  const uint32_t t = tmask >> (4 * (lane >> 5));
  return (t & 0xfu) | ((t >> 4) & 0xf0u) | ((t >> 8) & 0xf00u) | ((t >> 12) & 0xf000u);
}


// Walk a wave's tiles p0, p0 + step, ...: load the tile's K fragments, then process them
// (the other waves of the CU cover the load latency).
template <typename F, typename LoadFn, typename ProcFn>
__device__ __forceinline__ void tile_loop(LoadFn load_group, ProcFn process, int p0, int p_end,
                                          int step) {
  for (; p0 < p_end; p0 += step) {
    F kf[SCORE_KT];
    load_group(kf, p0);
    process(kf, p0);
  }
}

// ------------------------------------------------------------------ pass 1
template <typename T, int D, int QB>
__global__ __launch_bounds__(SCORE_NT) void score_pass1_kernel(
    const T* __restrict__ q_obs, const T* __restrict__ k_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const int32_t* __restrict__ n_pages_arr, int NS, int Hq,
    int Hkv, int W, int max_pages, float c2, float2* __restrict__ part, int n_chunks) {
  using F = Frag<T, D>;
  constexpr int R_pad = 32 * QB;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  stage_rows<T, D>(smem, R, R_pad, [&](int r) -> const T* {
    const int w = r / G, g = r % G;
    return q_obs + ((size_t)(w * NS + s) * Hq + kv * G + g) * D;
  });
  float2* red = reinterpret_cast<float2*>(smem + (size_t)R_pad * D * sizeof(T));
  __syncthreads();

  const int n = n_pages_arr[h];
  const int p_begin = chunk * SCORE_PPW, p_end = min(p_begin + SCORE_PPW, n);
  float M[QB], L[QB];
#pragma unroll
  for (int q = 0; q < QB; ++q) { M[q] = -INFINITY; L[q] = 0.f; }

  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  auto load_group = [&](F* kf, int p0) {
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) load_tile<T, D>(kf[t], k_pool, trow, p0 + 2 * t, p_end, lane);
  };
  auto process = [&](F* kf, int p0) {
    uint32_t tm[SCORE_KT];
    bool all_full = true, any = false;
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) {
      const int pa = p0 + 2 * t, pb = pa + 1;
      tm[t] = (pa < p_end ? (uint32_t)mrow[pa] : 0u) | ((pb < p_end) ? (uint32_t)mrow[pb] << 16 : 0u);
      all_full = all_full && (tm[t] == 0xffffffffu);
      any = any || (tm[t] != 0u);
    }
    if (all_full) {
      p1_tile_pipelined<F, QB, SCORE_KT>(kf, smem, c2, lane, M, L);
    } else if (any) {
      uint32_t rows[SCORE_KT];
#pragma unroll
      for (int t = 0; t < SCORE_KT; ++t) rows[t] = lane_rows(tm[t], lane);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        f32x16 acc[SCORE_KT];
        mma_chains<F, false, SCORE_KT>(kf, smem, qb, lane, acc);
        float m = -INFINITY;
#pragma unroll
        for (int t = 0; t < SCORE_KT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if ((rows[t] >> r) & 1u) m = vmax(m, acc[t][r]);
        const float mn = vmax(M[qb], m);
        if (mn != -INFINITY) {           // this column has seen a valid key
          const float mc = mn * c2;
          float sum = 0.f;
#pragma unroll
          for (int t = 0; t < SCORE_KT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if ((rows[t] >> r) & 1u) sum += fast_exp2(fmaf(acc[t][r], c2, -mc));
          L[qb] = fmaf(L[qb], fast_exp2((M[qb] - mn) * c2), sum);
          M[qb] = mn;
        }
      }
    }
  };
  tile_loop<F>(load_group, process, p_begin + SCORE_WPP * wave, p_end, SCORE_WPP * SCORE_NW);
  // merge lane halves (same query column), then waves
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float Mo = __shfl_xor(M[qb], 32, 64), Lo = __shfl_xor(L[qb], 32, 64);
    const float mn = fmaxf(M[qb], Mo);
    float Ln = 0.f;
    if (mn != -INFINITY) Ln = L[qb] * fast_exp2((M[qb] - mn) * c2) + Lo * fast_exp2((Mo - mn) * c2);
    if (lane < 32) red[wave * R_pad + qb * 32 + lane] = make_float2(mn, Ln);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < R; r += SCORE_NT) {
    float mn = -INFINITY;
    for (int w = 0; w < SCORE_NW; ++w) mn = fmaxf(mn, red[w * R_pad + r].x);
    float Ln = 0.f;
    if (mn != -INFINITY)
      for (int w = 0; w < SCORE_NW; ++w) {
        const float2 v = red[w * R_pad + r];
        Ln += v.y * fast_exp2((v.x - mn) * c2);
      }
    part[((size_t)h * n_chunks + chunk) * R_pad + r] = make_float2(mn, Ln);
  }
}

// merge chunk partials into natural-log row LSE, layout [W][NS][Hq]
__global__ __launch_bounds__(256) void score_lse_merge_kernel(const float2* __restrict__ part,
                                                               int n_chunks, int R_pad, int NS,
                                                               int Hq, int Hkv, int W, float c2,
                                                               float sm_scale, float* lse_out,
                                                               const int32_t* __restrict__ n_pages_arr,
                                                               int L_dense, int32_t* cand_len_out) {
  const int h = blockIdx.x, s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W;
  // the candidate count, also written by pass 2, so that a call without it has one too
  if (threadIdx.x == 0) cand_len_out[h] = HK_PAGE * max(0, n_pages_arr[h] - dense_pages(L_dense));
  // the partials are read MB at a time, every load issued before any is used (a loop of
  // load-then-use waits on each in turn); up to MB chunks this is one batch and the sums
  // run in chunk order, as a plain two-sweep merge would
  constexpr int MB = 16;
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    const float2* p = part + (size_t)h * n_chunks * R_pad + r;
    float mn = -INFINITY, L = 0.f;
    for (int c0 = 0; c0 < n_chunks; c0 += MB) {
      float2 v[MB];
#pragma unroll
      for (int i = 0; i < MB; ++i) v[i] = p[(size_t)min(c0 + i, n_chunks - 1) * R_pad];
#pragma unroll
      for (int i = 0; i < MB; ++i)
        if (c0 + i >= n_chunks) v[i] = make_float2(-INFINITY, 0.f);   // no such chunk
      float nm = mn;
#pragma unroll
      for (int i = 0; i < MB; ++i) nm = fmaxf(nm, v[i].x);
      if (nm == -INFINITY) continue;
      float add = 0.f;
#pragma unroll
      for (int i = 0; i < MB; ++i) add += v[i].y * exp2f((v[i].x - nm) * c2);
      L = (mn == -INFINITY) ? add : fmaf(L, exp2f((mn - nm) * c2), add);
      mn = nm;
    }
    const float lse = (mn == -INFINITY) ? -INFINITY : fmaf(mn, sm_scale, logf(L));
    const int w = r / G, g = r % G;
    lse_out[((size_t)w * NS + s) * Hq + kv * G + g] = lse;
  }
}

// ------------------------------------------------------------------ pass 2
// Waves per SIMD the register allocator must leave room for: 4 lets two 512-thread
// workgroups share a CU; asked only where it fits without spilling.
// (The 1024-thread redundancy shape already caps registers at 128.)
template <typename T, int D, int QB, bool RED>
constexpr int pass2_min_waves() {
  if (SCORE_KT > 1 || RED) return 1;
  return (sizeof(T) == 2 && D == 128 && (QB == 7 || QB == 4)) ? 4 : 1;
}

// Pass-2 launch shape.  The redundancy variant stages up to 256 reference rows (64 KB at
// D = 128 bf16) beside the window block, so one workgroup fills a CU's LDS: it runs 1024
// threads over 512 pages to amortise the staging.  The plain variant keeps two
// 512-thread workgroups of 128 pages per CU.
template <bool RED>
struct P2Shape {
  static constexpr int NT = RED ? 1024 : SCORE_NT;
  static constexpr int PPW = RED ? 512 : SCORE_PPW;
};

template <typename T, int D, int QB, bool RED>
__global__ __launch_bounds__(P2Shape<RED>::NT) __attribute__((amdgpu_waves_per_eu(
    pass2_min_waves<T, D, QB, RED>(), pass2_min_waves<T, D, QB, RED>() > 1 ? pass2_min_waves<T, D, QB, RED>() : 8)))
void score_pass2_kernel(
    const T* __restrict__ q_obs, const T* __restrict__ k_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const int32_t* __restrict__ n_pages_arr, int NS, int Hq,
    int Hkv, int W, int max_pages, int L_dense, float c2, float lnR,
    const float* __restrict__ row_lse, float* __restrict__ s_out, int32_t* __restrict__ cand_len_out,
    const int32_t* __restrict__ ref_slots, int n_ref, float* __restrict__ x_red) {
  using F = Frag<T, D>;
  constexpr int R_pad = 32 * QB;
  extern __shared__ __align__(16) char smem[];
  constexpr int NT = P2Shape<RED>::NT, NW = NT / 64, PPW = P2Shape<RED>::PPW;
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t S_max = (size_t)max_pages * HK_PAGE;
  const int n = n_pages_arr[h];
  const int cand_len = HK_PAGE * max(0, n - dense_pages(L_dense));
  if (chunk == 0 && threadIdx.x == 0) cand_len_out[h] = cand_len;

  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  const int p_begin = chunk * PPW, p_end_all = min(p_begin + PPW, max_pages);
  const int p_cand_end = min(p_end_all, cand_len / HK_PAGE);

  // slots of this chunk that hold no candidate: -inf
  {
    const int j0 = max(p_cand_end, p_begin) * HK_PAGE, j1 = p_end_all * HK_PAGE;
    for (int j = j0 + threadIdx.x; j < j1; j += NT) {
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
  for (int r = threadIdx.x; r < R_pad; r += NT) {
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
  uint32_t* ref_bits = nullptr;
  int RB = 0;
  if constexpr (RED) {
    const int nr_pad = (n_ref + 31) & ~31;
    RB = nr_pad >> 5;
    rn_ref = reinterpret_cast<float*>(ref_lds + (size_t)NREF_MAX * D * sizeof(T));
    ref_slot = reinterpret_cast<int32_t*>(rn_ref + NREF_MAX);
    ref_bits = reinterpret_cast<uint32_t*>(ref_slot + NREF_MAX);   // [PPW / 2] words
    const int32_t* rs = ref_slots + (size_t)h * n_ref;
    auto ref_row = [&](int i) -> const T* {
      const int j = rs[i];
      const int pp = j >> 4;
      if (j < 0 || pp >= n) return nullptr;
      return k_pool + ((size_t)trow[pp] * HK_PAGE + (j & 15)) * D;
    };
    // padding rows (n_ref <= i < nr_pad) repeat reference 0: a repeated member changes
    // neither the maximum nor the self test (its slot is reference 0's)
    stage_rows<T, D>(ref_lds, nr_pad, nr_pad, [&](int i) { return ref_row(i < n_ref ? i : 0); });
    for (int i = threadIdx.x; i < PPW / 2; i += NT) ref_bits[i] = 0u;
    __syncthreads();
    for (int i = threadIdx.x; i < nr_pad; i += NT) {
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
      // a zero-norm reference has cosine 0 with every key
      rn_ref[i] = ss > 0.f ? 1.0f / sqrtf(ss) : 0.f;
      const int slot = rs[i < n_ref ? i : 0];
      ref_slot[i] = slot;
      const int rel = slot - p_begin * HK_PAGE;    // reference slots inside this chunk
      if (i < n_ref && rel >= 0 && rel < PPW * HK_PAGE)
        atomicOr(&ref_bits[rel >> 5], 1u << (rel & 31));
    }
  }
  __syncthreads();

  auto load_group = [&](F* kf, int p0) {
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) load_tile<T, D>(kf[t], k_pool, trow, p0 + 2 * t, p_cand_end, lane);
  };
  auto process = [&](F* kf, int p0) {
    uint32_t m0[SCORE_KT], m1[SCORE_KT];
    bool any = false;
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) {
      const int pa = p0 + 2 * t, pb = pa + 1;
      m0[t] = (pa < p_cand_end) ? (uint32_t)mrow[pa] : 0u;
      m1[t] = (pb < p_cand_end) ? (uint32_t)mrow[pb] : 0u;
      any = any || ((m0[t] | m1[t]) != 0u);
    }
    const int kl = lane & 31;
    float col[SCORE_KT];
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) col[t] = 0.f;
    if (any) p2_tile_pipelined<F, QB, SCORE_KT>(kf, smem, lse2, c2, lane, col);
#pragma unroll
    for (int t = 0; t < SCORE_KT; ++t) {
      const int pg = p0 + 2 * t + (kl >> 4);
      const int slot = pg * HK_PAGE + (kl & 15);
      const bool cand = (pg < p_cand_end) && (((kl < 16 ? m0[t] : m1[t]) >> (kl & 15)) & 1u);
      const bool write = (lane < 32) && (pg < p_cand_end);
      const float c_all = col[t] + __shfl_xor(col[t], 32, 64);
      if constexpr (RED) {
        float x = -INFINITY;
        if ((m0[t] | m1[t]) != 0u) {
          const float ss = kf[t].sumsq();
          const float nrm2 = ss + __shfl_xor(ss, 32, 64);
          const float rn = nrm2 > 0.f ? 1.0f / sqrtf(nrm2) : 0.f;
          const uint32_t self_word = ref_bits[(p0 + 2 * t - p_begin) >> 1];
          float cmax = -INFINITY;
          int self = 0;
          red_tile_max<F>(kf[t], ref_lds, rn_ref, ref_slot, RB, lane, slot, self_word != 0u, cmax, self);
          cmax = vmax(cmax, __shfl_xor(cmax, 32, 64));
          self |= __shfl_xor(self, 32, 64);
          if (cand) x = (n_ref - self > 0) ? -(cmax * rn) : 1.0f;
        }
        if (write) x_red[(size_t)h * S_max + slot] = x;
      }
      if (write) s_out[(size_t)h * S_max + slot] = cand ? fmaf(fast_log2(c_all), kLn2, -lnR) : -INFINITY;
    }
  };
  tile_loop<F>(load_group, process, p_begin + SCORE_WPP * wave, p_cand_end, SCORE_WPP * NW);
}

// ------------------------------------------------------------------ cooperative passes (bf16)
// The passes for bf16 caches without the redundancy metric.  Every wave of the workgroup owns
// one 32-row block of the window queries, held in registers as an MFMA fragment for the whole
// chunk; 32-key K tiles are shared by all waves.  The workgroup loads each tile cooperatively
// (one 16-byte piece per thread, the pieces of tile t + STAGES in flight while tile t is
// computed, so the prefetch costs a few registers per stage instead of a whole tile per wave),
// writes it to a double-buffered LDS tile in MFMA fragment order -- piece kk * 64 + lane holds
// key lane % 32, dims [16 kk + 8 (lane / 32), +8) -- and every wave reads the fragments with
// conflict-free 16-byte LDS reads.  One barrier per iteration orders the buffers.
//   pass 1  C[key][query] = K Q^T: lane-local online (max, sum exp) of the lane's query column;
//   pass 2  C[query][key] = Q K^T: lane-local sum over the wave's rows of exp(z - LSE) per key;
//           the per-wave column sums of a tile meet in LDS and are summed (and the log taken)
//           by the last wave one iteration later.
template <int D, int QB>
struct Coop {
  static constexpr int NT = 512, NW = 8;
  static constexpr int TPI = QB <= 4 ? 2 : 1;           // 32-key tiles per iteration
  static constexpr int KS = D / 16;                     // MFMA k-steps per tile
  static constexpr int TILE_CH = KS * 64;               // 16-byte pieces per tile
  static constexpr int ITER_CH = TPI * TILE_CH;         // pieces per iteration
  static constexpr int LPT = (ITER_CH + NT - 1) / NT;   // pieces each thread loads per iteration
  static constexpr int STAGES = 4;                      // iterations loaded ahead (4: unrolled)
  static constexpr int PPI = 2 * TPI;                   // pages per iteration
  static constexpr int PPW = 128;                       // pages per workgroup
  static constexpr int BUF = ITER_CH * 16;              // bytes of one LDS tile buffer
  static constexpr int ACTIVE = TPI * QB < NW ? TPI * QB : NW;   // waves with a query block
  static_assert(STAGES == 4, "the main loop is written out for four stages");
  static_assert(TPI * QB <= NW, "one query block per wave");
};

// LDS of a cooperative pass: 2 tile buffers, the chunk's page ids and masks, the per-wave
// reduction scratch (two iterations of column sums for pass 2; (max, sum) for pass 1) and the
// chunk's scores, written to memory once at the end.  No global store and no conditional load
// sits in the main loop: the compiler then counts the loads in flight exactly and waits for
// the oldest iteration's pieces only, instead of for every load.
template <int D, int QB>
struct CoopLds {
  using C = Coop<D, QB>;
  static constexpr size_t BUFS = 0;
  static constexpr size_t TABLE = BUFS + 2 * (size_t)C::BUF;
  static constexpr size_t MASK = TABLE + C::PPW * 4;
  static constexpr size_t RED = MASK + C::PPW * 4;
  static constexpr size_t RES = RED + 2 * C::NW * 32 * sizeof(float2);
  static constexpr size_t LSE = RES + C::PPW * HK_PAGE * sizeof(float);     // pass 2's scores
  static constexpr size_t TOTAL = LSE + 32 * QB * sizeof(float);           // pass 2's row LSEs
};

// Issues (into registers) the K pieces this thread loads for iteration `it`: pages past the
// chunk's last page are clamped to it (their keys are masked or never stored; the repeated
// page is a cache hit), so every iteration issues the same loads unconditionally.
// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled before any optimisation sees a loop
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (N > 0) {
    static_for<N - 1>(f);
    f(std::integral_constant<int, N - 1>{});
  }
}

// The issue is split in two so the page-id reads (LDS) of an iteration's loads can be made
// an iteration ahead of the loads themselves: coop_phys reads the physical page of each of
// the thread's pieces, coop_load issues the loads from them.
template <int D, int QB, int N>
__device__ __forceinline__ void coop_phys(int (&ph)[N], const int32_t* s_table, int p_begin, int p_last,
                                          int it) {
  using C = Coop<D, QB>;
  const int p0 = p_begin + it * C::PPI;
  static_for<C::LPT>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    const int c = i * C::NT + (int)threadIdx.x;
    if (C::ITER_CH % C::NT == 0 || c < C::ITER_CH) {
      const int ts = c / C::TILE_CH, key = (c % C::TILE_CH) & 31;
      ph[i] = s_table[min(p0 + 2 * ts + (key >> 4), p_last) - p_begin];
    }
  });
}
template <int D, int QB, int N>
__device__ __forceinline__ void coop_load(u32x4 (&r)[N], const uint16_t* __restrict__ k_pool, const int (&ph)[N]) {
  using C = Coop<D, QB>;
  static_for<C::LPT>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    const int c = i * C::NT + (int)threadIdx.x;
    if (C::ITER_CH % C::NT == 0 || c < C::ITER_CH) {
      const int f = c % C::TILE_CH;
      const int kk = f >> 6, ln = f & 63, key = ln & 31;
      r[i] = *reinterpret_cast<const u32x4*>(k_pool + ((size_t)ph[i] * HK_PAGE + (key & 15)) * D + kk * 16 +
                                             (ln >> 5) * 8);
    }
  });
}
template <int D, int QB, int N>
__device__ __forceinline__ void coop_issue(u32x4 (&r)[N], const uint16_t* __restrict__ k_pool,
                                           const int32_t* s_table, int p_begin, int p_last, int it) {
  int ph[N];
  coop_phys<D, QB>(ph, s_table, p_begin, p_last, it);
  coop_load<D, QB>(r, k_pool, ph);
}
template <int D, int QB, int N>
__device__ __forceinline__ void coop_store(const u32x4 (&r)[N], char* buf) {
  using C = Coop<D, QB>;
  static_for<C::LPT>([&](auto ic) {
    constexpr int i = decltype(ic)::value;
    const int c = i * C::NT + (int)threadIdx.x;
    if (C::ITER_CH % C::NT == 0 || c < C::ITER_CH) *reinterpret_cast<u32x4*>(buf + (size_t)c * 16) = r[i];
  });
}

// The chunk's page ids and masks into LDS; the wave's query block as an MFMA fragment.
template <int D, int QB, int KS>
__device__ __forceinline__ void coop_setup(char* smem, const int32_t* trow, const uint16_t* mrow,
                                           int p_begin, int p_stage_end, const uint16_t* __restrict__ q_obs,
                                           int NS, int Hq, int Hkv, int W, int s, int kv, int qb, bool active,
                                           bf16x8 (&qf)[KS]) {
  using C = Coop<D, QB>;
  using L = CoopLds<D, QB>;
  int32_t* s_table = reinterpret_cast<int32_t*>(smem + L::TABLE);
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(smem + L::MASK);
  for (int i = threadIdx.x; i < C::PPW; i += C::NT) {
    const int pg = p_begin + i;
    s_table[i] = pg < p_stage_end ? trow[pg] : 0;
    s_mask[i] = pg < p_stage_end ? (uint32_t)mrow[pg] : 0u;
  }
  const int lane = threadIdx.x & 63;
  const int G = Hq / Hkv, R = G * W;
  const int r = qb * 32 + (lane & 31);
  const int rc = min(r, R - 1);                  // padding rows read a real row, then are zeroed
  const uint16_t* row = q_obs + ((size_t)((rc / G) * NS + s) * Hq + kv * G + rc % G) * D + (lane >> 5) * 8;
  const bool keep = active && r < R;
#pragma unroll
  for (int kk = 0; kk < C::KS; ++kk) {
    u32x4 u = *reinterpret_cast<const u32x4*>(row + kk * 16);
    if (!keep) u = u32x4{0u, 0u, 0u, 0u};
    qf[kk] = __builtin_bit_cast(bf16x8, u);
  }
}

template <int D, int QB>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4, 4)))
void score_pass1_coop_kernel(const uint16_t* __restrict__ q_obs, const uint16_t* __restrict__ k_pool,
                             const int32_t* __restrict__ table, const uint16_t* __restrict__ masks,
                             const int32_t* __restrict__ n_pages_arr, int NS, int Hq, int Hkv, int W,
                             int max_pages, float c2, float2* __restrict__ part, int n_chunks) {
  using C = Coop<D, QB>;
  using L = CoopLds<D, QB>;
  constexpr int R_pad = 32 * QB;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool active = wave < C::ACTIVE;
  const int ts = wave / QB, qb = wave % QB;
  const int n = n_pages_arr[h];
  const int p_begin = chunk * C::PPW, p_end = min(p_begin + C::PPW, n);
  bf16x8 qf[C::KS];
  coop_setup<D, QB>(smem, table + (size_t)h * max_pages, masks + (size_t)h * max_pages, p_begin, p_end,
                    q_obs, NS, Hq, Hkv, W, s, kv, qb, active, qf);
  const int32_t* s_table = reinterpret_cast<const int32_t*>(smem + L::TABLE);
  const uint32_t* s_mask = reinterpret_cast<const uint32_t*>(smem + L::MASK);
  float2* red = reinterpret_cast<float2*>(smem + L::RED);            // [NW][32]
  __syncthreads();

  float M = -INFINITY, Lsum = 0.f;
  const int n_iter = p_end > p_begin ? (p_end - p_begin + C::PPI - 1) / C::PPI : 0;
  const int p_last = p_end - 1;
  u32x4 pre0[C::LPT], pre1[C::LPT], pre2[C::LPT], pre3[C::LPT];
  auto slot = [&](auto uc) -> u32x4(&)[C::LPT] {
    constexpr int u = decltype(uc)::value % 4;
    if constexpr (u == 0) return pre0;
    else if constexpr (u == 1) return pre1;
    else if constexpr (u == 2) return pre2;
    else return pre3;
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  if (n_iter > 0) {
    coop_issue<D, QB>(pre0, k_pool, s_table, p_begin, p_last, 0);
    coop_issue<D, QB>(pre1, k_pool, s_table, p_begin, p_last, 1);
    coop_issue<D, QB>(pre2, k_pool, s_table, p_begin, p_last, 2);
    coop_issue<D, QB>(pre3, k_pool, s_table, p_begin, p_last, 3);
    coop_store<D, QB>(pre0, smem + L::BUFS);
    coop_issue<D, QB>(pre0, k_pool, s_table, p_begin, p_last, C::STAGES);
  }

  // Online (max, sum exp) update of the lane's query column with one tile's accumulator:
  // every key of the tile valid (fast path) or under the tile's 32-slot mask.
  auto update_masked = [&](const f32x16& a, uint32_t tm) {
    const uint32_t rows = lane_rows(tm, lane);
    float m = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if ((rows >> e) & 1u) m = vmax(m, a[e]);
    const float mn = vmax(M, m);
    if (mn != -INFINITY) {                       // this column has seen a valid key
      const float mc = mn * c2;
      float sum = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if ((rows >> e) & 1u) sum += fast_exp2(fmaf(a[e], c2, -mc));
      Lsum = fmaf(Lsum, fast_exp2((M - mn) * c2), sum);
      M = mn;
    }
  };
  // the 16-bit masks of a tile's two pages (chunk-relative page pl, pl + 1; past the end: 0),
  // read as one 64-bit LDS load at a clamped, always valid page
  auto tile_mask_raw = [&](int it_) {
    const int pl = min(it_ * C::PPI + 2 * ts, C::PPW - 2);
    return *reinterpret_cast<const uint2*>(s_mask + pl);
  };

  // Software pipeline inside each wave: the MFMAs of tile it run beside the sum of
  // exponentials of tile it - 1's accumulator, one step per scheduling region.  Tiles with
  // masked keys take the plain update after the chain.  Iterations run in groups of four up to
  // n_iter + 1 (the last drains the pipeline); those past n_iter only move data.
  f32x16 accs[2] = {f32x16{}, f32x16{}};     // tile it's MFMAs: accs[it & 1]
  // the masks of the tile whose exponentials an iteration takes, loaded one iteration ahead
  // and only combined when used, so no iteration waits for its own mask read
  uint2 mask_next = make_uint2(0u, 0u);
  auto iteration = [&](auto uc, int it) {
    constexpr int u = decltype(uc)::value;
    __syncthreads();
    int ph[C::LPT];
    coop_phys<D, QB>(ph, s_table, p_begin, p_last, it + 1 + C::STAGES);
    const uint2 mraw = mask_next;
    mask_next = tile_mask_raw(it);
    if (active) {
      const bool prev = it >= 1 && it - 1 < n_iter;
      const uint32_t tmp = prev ? mraw.x | (mraw.y << 16) : 0u;
      const bool fuse = tmp == 0xffffffffu;
      if (it < n_iter) {
        const char* tb = smem + L::BUFS + (size_t)(u & 1) * C::BUF + (size_t)ts * C::TILE_CH * 16 +
                         (size_t)lane * 16;
        constexpr int KD = 2;                    // fragments read this many steps ahead
        bf16x8 kf[KD + 1];
#pragma unroll
        for (int g = 0; g < KD; ++g) kf[g] = *reinterpret_cast<const bf16x8*>(tb + (size_t)g * 1024);
        f32x16& acc = accs[u & 1];
        acc = f32x16{};
        if (fuse) {
          // exponentials against the lane's current reference maximum M, no maximum per
          // tile: the sum is exact unless a key exceeds M by more than 64 powers of two (or
          // M is still -inf, or the tile holds a NaN), in which case the sum is not <= 2^64
          // and the lane redoes the tile with the exact update
          const float mc = M * c2;
          float s0 = 0.f, s1 = 0.f;
#pragma unroll
          for (int kk = 0; kk < C::KS; ++kk) {
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk % (KD + 1)], qf[kk], acc, 0, 0, 0);
            if (kk + KD < C::KS)
              kf[(kk + KD) % (KD + 1)] = *reinterpret_cast<const bf16x8*>(tb + (size_t)(kk + KD) * 1024);
#pragma unroll
            for (int e = 0; e < 16; ++e)
              if (e * C::KS / 16 == kk) {
                if (e & 1) s1 += fast_exp2(fmaf(accs[(u + 1) & 1][e], c2, -mc));
                else s0 += fast_exp2(fmaf(accs[(u + 1) & 1][e], c2, -mc));
              }
            __builtin_amdgcn_sched_barrier(0);
          }
          const float st = s0 + s1;
          if (st <= 0x1p64f) Lsum += st;
          else update_masked(accs[(u + 1) & 1], 0xffffffffu);
        } else {
#pragma unroll
          for (int kk = 0; kk < C::KS; ++kk) {
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk % (KD + 1)], qf[kk], acc, 0, 0, 0);
            if (kk + KD < C::KS)
              kf[(kk + KD) % (KD + 1)] = *reinterpret_cast<const bf16x8*>(tb + (size_t)(kk + KD) * 1024);
          }
          if (tmp != 0u) update_masked(accs[(u + 1) & 1], tmp);
        }
      } else if (prev && tmp != 0u) {
        update_masked(accs[(u + 1) & 1], tmp);
      }
    }
    coop_store<D, QB>(slot(std::integral_constant<int, u + 1>{}), smem + L::BUFS + (size_t)((u + 1) & 1) * C::BUF);
    coop_load<D, QB>(slot(std::integral_constant<int, u + 1>{}), k_pool, ph);
  };
  // A chunk with no page (n_iter = 0) runs no iteration: each ends by issuing clamped loads
  // for a later one, and with no page the clamp (to p_last = p_end - 1 < p_begin) would read
  // the page table below its first entry.
  for (int it0 = 0; n_iter > 0 && it0 < n_iter + 1; it0 += 4) {
    iteration(I0{}, it0);
    iteration(I1{}, it0 + 1);
    iteration(I2{}, it0 + 2);
    iteration(I3{}, it0 + 3);
  }
  // merge the lane halves (same query column), then the tile slots of one query block
  {
    const float Mo = __shfl_xor(M, 32, 64), Lo = __shfl_xor(Lsum, 32, 64);
    const float mn = fmaxf(M, Mo);
    float Ln = 0.f;
    if (mn != -INFINITY) Ln = Lsum * fast_exp2((M - mn) * c2) + Lo * fast_exp2((Mo - mn) * c2);
    if (active && lane < 32) red[wave * 32 + lane] = make_float2(mn, Ln);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < R_pad; r += C::NT) {
    const int b = r >> 5, j = r & 31;
    float mn = -INFINITY;
#pragma unroll
    for (int t = 0; t < C::TPI; ++t) mn = fmaxf(mn, red[(t * QB + b) * 32 + j].x);
    float Ln = 0.f;
    if (mn != -INFINITY)
#pragma unroll
      for (int t = 0; t < C::TPI; ++t) {
        const float2 v = red[(t * QB + b) * 32 + j];
        Ln += v.y * fast_exp2((v.x - mn) * c2);
      }
    part[((size_t)h * n_chunks + chunk) * R_pad + r] = make_float2(mn, Ln);
  }
}

template <int D, int QB>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4, 4)))
void score_pass2_coop_kernel(const uint16_t* __restrict__ q_obs, const uint16_t* __restrict__ k_pool,
                             const int32_t* __restrict__ table, const uint16_t* __restrict__ masks,
                             const int32_t* __restrict__ n_pages_arr, int NS, int Hq, int Hkv, int W,
                             int max_pages, int L_dense, float c2, float lnR,
                             const float* __restrict__ row_lse, float* __restrict__ s_out,
                             int32_t* __restrict__ cand_len_out) {
  using C = Coop<D, QB>;
  using L = CoopLds<D, QB>;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool active = wave < C::ACTIVE;
  const int ts = wave / QB, qb = wave % QB;
  const size_t S_max = (size_t)max_pages * HK_PAGE;
  const int n = n_pages_arr[h];
  const int cand_len = HK_PAGE * max(0, n - dense_pages(L_dense));
  if (chunk == 0 && threadIdx.x == 0) cand_len_out[h] = cand_len;
  const int p_begin = chunk * C::PPW, p_end_all = min(p_begin + C::PPW, max_pages);
  const int p_cand_end = min(p_end_all, cand_len / HK_PAGE);
  float* srow = s_out + (size_t)h * S_max;
  {
    // slots of this chunk that hold no candidate: -inf
    const int j0 = max(p_cand_end, p_begin) * HK_PAGE, j1 = p_end_all * HK_PAGE;
    for (int j = j0 + threadIdx.x; j < j1; j += C::NT) srow[j] = -INFINITY;
  }
  if (p_begin >= p_cand_end) return;

  bf16x8 qf[C::KS];
  coop_setup<D, QB>(smem, table + (size_t)h * max_pages, masks + (size_t)h * max_pages, p_begin, p_cand_end,
                    q_obs, NS, Hq, Hkv, W, s, kv, qb, active, qf);
  const int32_t* s_table = reinterpret_cast<const int32_t*>(smem + L::TABLE);
  const uint32_t* s_mask = reinterpret_cast<const uint32_t*>(smem + L::MASK);
  float* red = reinterpret_cast<float*>(smem + L::RED);              // [2][NW][32]
  float* res = reinterpret_cast<float*>(smem + L::RES);              // the chunk's scores
  float* lse2 = reinterpret_cast<float*>(smem + L::LSE);             // [32 QB], log2 units
  for (int r = threadIdx.x; r < 32 * QB; r += C::NT) {
    const int rc = min(r, R - 1);                 // every load issued; padding rows weigh 0
    const float v = row_lse[((size_t)(rc / G) * NS + s) * Hq + kv * G + rc % G];
    lse2[r] = r < R ? v * kLog2e : INFINITY;
  }
  __syncthreads();

  // the last wave's lanes sum the column partials of one tile iteration (key k of tile slot
  // k / 32), take the log and keep the score in LDS
  constexpr int NRED = C::TPI * 32;
  const int rk = (int)threadIdx.x - (C::NT - NRED);
  auto reduce = [&](int it_done, int par) {
    if (rk < 0) return;
    const int t = rk >> 5, j = rk & 31;
    const int pl = it_done * C::PPI + 2 * t + (j >> 4);              // chunk-relative page
    if (p_begin + pl >= p_cand_end) return;
    float sum = 0.f;
#pragma unroll
    for (int b = 0; b < QB; ++b) sum += red[(par * C::NW + t * QB + b) * 32 + j];
    const bool cand = (s_mask[pl] >> (j & 15)) & 1u;
    res[pl * HK_PAGE + (j & 15)] = cand ? fmaf(fast_log2(sum), kLn2, -lnR) : -INFINITY;
  };

  const int n_iter = (p_cand_end - p_begin + C::PPI - 1) / C::PPI;
  const int p_last = p_cand_end - 1;
  u32x4 pre0[C::LPT], pre1[C::LPT], pre2[C::LPT], pre3[C::LPT];
  auto slot = [&](auto uc) -> u32x4(&)[C::LPT] {
    constexpr int u = decltype(uc)::value % 4;
    if constexpr (u == 0) return pre0;
    else if constexpr (u == 1) return pre1;
    else if constexpr (u == 2) return pre2;
    else return pre3;
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  coop_issue<D, QB>(pre0, k_pool, s_table, p_begin, p_last, 0);
  coop_issue<D, QB>(pre1, k_pool, s_table, p_begin, p_last, 1);
  coop_issue<D, QB>(pre2, k_pool, s_table, p_begin, p_last, 2);
  coop_issue<D, QB>(pre3, k_pool, s_table, p_begin, p_last, 3);
  coop_store<D, QB>(pre0, smem + L::BUFS);
  coop_issue<D, QB>(pre0, k_pool, s_table, p_begin, p_last, C::STAGES);

  // Software pipeline inside each wave: the MFMAs of tile it run beside the exponentials of
  // tile it - 1 (its accumulator kept from the previous iteration; independent work, which
  // the SIMD overlaps within a wave), pinned step by step with scheduling-group barriers;
  // the last wave reduces tile it - 2.  Iterations run in groups of four up to n_iter + 2
  // (the two after the last tile drain the pipeline); those past n_iter only move data.
  const float* lrow = lse2 + qb * 32 + 4 * (lane >> 5);
  const int swap_addr = (lane ^ 32) << 2;        // ds_bpermute address of the other half's lane
  f32x16 accp = {};
  auto iteration = [&](auto uc, int it) {
    constexpr int u = decltype(uc)::value;
    __syncthreads();
    int ph[C::LPT];
    coop_phys<D, QB>(ph, s_table, p_begin, p_last, it + 1 + C::STAGES);
    if (it >= 2 && it - 2 < n_iter) reduce(it - 2, u & 1);
    if (active) {
      const bool prev = it >= 1 && it - 1 < n_iter;
      f32x4 l4[4];
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) l4[r4] = *reinterpret_cast<const f32x4*>(lrow + 8 * r4);
      float c0 = 0.f, c1 = 0.f;
      if (it < n_iter) {
        const char* tb = smem + L::BUFS + (size_t)(u & 1) * C::BUF + (size_t)ts * C::TILE_CH * 16 +
                         (size_t)lane * 16;
        // K fragments are read KD MFMA steps ahead of their use
        constexpr int KD = 2;
        bf16x8 kf[KD + 1];
#pragma unroll
        for (int g = 0; g < KD; ++g) kf[g] = *reinterpret_cast<const bf16x8*>(tb + (size_t)g * 1024);
        f32x16 acc = {};
#pragma unroll
        for (int kk = 0; kk < C::KS; ++kk) {
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[kk], kf[kk % (KD + 1)], acc, 0, 0, 0);
          if (kk + KD < C::KS)
            kf[(kk + KD) % (KD + 1)] = *reinterpret_cast<const bf16x8*>(tb + (size_t)(kk + KD) * 1024);
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (e * C::KS / 16 == kk) {
              if (e & 1) c1 += fast_exp2(fmaf(accp[e], c2, -l4[e >> 2][e & 3]));
              else c0 += fast_exp2(fmaf(accp[e], c2, -l4[e >> 2][e & 3]));
            }
          // one step per scheduling region: the MFMA, the fragment read KD steps ahead and
          // 16 / KS exponentials of the previous tile stay together, in this order
          __builtin_amdgcn_sched_barrier(0);
        }
        accp = acc;
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          if (e & 1) c1 += fast_exp2(fmaf(accp[e], c2, -l4[e >> 2][e & 3]));
          else c0 += fast_exp2(fmaf(accp[e], c2, -l4[e >> 2][e & 3]));
        }
      }
      if (prev) {
        float col = c0 + c1;
        col += __int_as_float(__builtin_amdgcn_ds_bpermute(swap_addr, __float_as_int(col)));
        if (lane < 32) red[(((u + 1) & 1) * C::NW + wave) * 32 + lane] = col;
      }
    }
    coop_store<D, QB>(slot(std::integral_constant<int, u + 1>{}), smem + L::BUFS + (size_t)((u + 1) & 1) * C::BUF);
    coop_load<D, QB>(slot(std::integral_constant<int, u + 1>{}), k_pool, ph);
  };
  for (int it0 = 0; it0 < n_iter + 2; it0 += 4) {
    iteration(I0{}, it0);
    iteration(I1{}, it0 + 1);
    iteration(I2{}, it0 + 2);
    iteration(I3{}, it0 + 3);
  }
  __syncthreads();
  for (int j = threadIdx.x; j < (p_cand_end - p_begin) * HK_PAGE; j += C::NT)
    srow[(size_t)p_begin * HK_PAGE + j] = res[j];
}

static size_t pass1_lds(int R_pad, int D, int es) {
  return (size_t)R_pad * D * es + (size_t)SCORE_NW * R_pad * sizeof(float2);
}
static size_t pass2_lds(int R_pad, int D, int es, bool red) {
  size_t b = (size_t)R_pad * D * es + (size_t)R_pad * sizeof(float);
  if (red) b += (size_t)NREF_MAX * D * es + (size_t)NREF_MAX * 8 + (P2Shape<true>::PPW / 2) * 4;
  return b;
}

// ------------------------------------------------------------------ per-row probabilities
// a[h][r][j] = exp(z[r][j] - LSE_r) for candidate slots j, 0 for every other slot: each window
// row's own attention distribution, which the Cautious Update strategy (Sec. 3.1) lets vote
// one by one.  Same tiles as pass 2 (C[query][key] on MFMA 32x32); each accumulator value is
// stored instead of summed over rows.  Register e of lane l is row 8*(e/4) + 4*(l/32) + e%4 of
// the block and key l % 32, so each half wave stores 32 consecutive floats of one row.
// (Four waves per SIMD cap the registers at 128, as for pass 2: uncapped, the compiler
// holds every query block's operands at once and spills.)
template <typename T, int D, int QB>
constexpr int rows_min_waves() {
  return (sizeof(T) == 2 && D == 128 && (QB == 7 || QB == 4)) ? 4 : 1;
}

template <typename T, int D, int QB>
__global__ __launch_bounds__(SCORE_NT) __attribute__((amdgpu_waves_per_eu(
    rows_min_waves<T, D, QB>(), rows_min_waves<T, D, QB>() > 1 ? rows_min_waves<T, D, QB>() : 8)))
void score_rows_kernel(
    const T* __restrict__ q_obs, const T* __restrict__ k_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const int32_t* __restrict__ n_pages_arr, int NS, int Hq,
    int Hkv, int W, int max_pages, int L_dense, float c2, const float* __restrict__ row_lse,
    float* __restrict__ a_rows) {
  using F = Frag<T, D>;
  constexpr int R_pad = 32 * QB;
  extern __shared__ __align__(16) char smem[];
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv, G = Hq / Hkv;
  const int R = G * W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t S_max = (size_t)max_pages * HK_PAGE;
  const int n = n_pages_arr[h];
  const int cand_len = HK_PAGE * max(0, n - dense_pages(L_dense));
  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  const int p_begin = chunk * SCORE_PPW, p_end_all = min(p_begin + SCORE_PPW, max_pages);
  const int p_cand_end = min(p_end_all, cand_len / HK_PAGE);
  float* arow = a_rows + (size_t)h * R * S_max;

  // slots of this chunk that hold no candidate: 0 in every row
  {
    const int j0 = max(p_cand_end, p_begin) * HK_PAGE, width = p_end_all * HK_PAGE - j0;
    if (width > 0)
      for (int i = threadIdx.x; i < R * width; i += SCORE_NT)
        arow[(size_t)(i / width) * S_max + j0 + i % width] = 0.f;
  }
  if (p_begin >= p_cand_end) return;

  stage_rows<T, D>(smem, R, R_pad, [&](int r) -> const T* {
    const int w = r / G, g = r % G;
    return q_obs + ((size_t)(w * NS + s) * Hq + kv * G + g) * D;
  });
  float* lse2 = reinterpret_cast<float*>(smem + (size_t)R_pad * D * sizeof(T));
  for (int r = threadIdx.x; r < R_pad; r += SCORE_NT) {
    float v = INFINITY;
    if (r < R) {
      const int w = r / G, g = r % G;
      v = row_lse[((size_t)w * NS + s) * Hq + kv * G + g] * kLog2e;
    }
    lse2[r] = v;
  }
  __syncthreads();

  const int kl = lane & 31;
  // the head's R rows as one buffer (R * S_max * 4 <= 32 MiB)
  const __amdgpu_buffer_rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(
      (void*)arow, (short)0, (int)((size_t)R * S_max * sizeof(float)), 0x00020000);
  auto load_group = [&](F* kf, int p0) { load_tile<T, D>(kf[0], k_pool, trow, p0, p_cand_end, lane); };
  auto process = [&](F* kfs, int p0) {
    const F& kf = kfs[0];
    const int pg = p0 + (kl >> 4);
    const int slot = pg * HK_PAGE + (kl & 15);
    const bool in = pg < p_cand_end;
    const bool cand = in && (((uint32_t)mrow[pg] >> (kl & 15)) & 1u);
    const uint32_t voff = (uint32_t)((4 * (lane >> 5)) * S_max + slot) * 4u;
    const uint32_t row_bytes = (uint32_t)S_max * 4u;
    if (p0 + 1 < p_cand_end && R == R_pad) {
      rows_tile_pipelined<F, QB>(kf, smem, lse2, c2, lane, cand, out, voff, row_bytes);
      return;
    }
    // a tile at the end of the candidates or a row count that is not a multiple of 32
#pragma unroll 1
    for (int qb = 0; qb < QB; ++qb) {
      const f32x16 acc = mma_chain<F, true>(kf, smem, qb, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = qb * 32 + acc_row(e, lane);
        if (in && row < R) {
          // a probability: rounding in exp and in LSE can put the largest a hair above 1
          const float a = cand ? fminf(fast_exp2(fmaf(acc[e], c2, -lse2[row])), 1.0f) : 0.f;
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(a), out, (int)voff,
                                                (int)((qb * 32 + 8 * (e >> 2) + (e & 3)) * row_bytes),
                                                2 /* nontemporal */);
        }
      }
    }
  };
  tile_loop<F>(load_group, process, p_begin + 2 * wave, p_cand_end, 2 * SCORE_NW);
}

template <typename T, int D, int QB>
hipError_t launch_score_rows_q(int NS, int Hq, int Hkv, int W, const void* q_obs,
                               const hk_paged_kv* kv, int L_dense, float sm_scale,
                               const float* row_lse, float* a_rows, hipStream_t st) {
  constexpr int R_pad = 32 * QB;
  const int n_heads = NS * Hkv;
  const int n_chunks = (kv->max_pages + SCORE_PPW - 1) / SCORE_PPW;
  const size_t lds = (size_t)R_pad * D * sizeof(T) + (size_t)R_pad * sizeof(float);
  allow_dynamic_lds<score_rows_kernel<T, D, QB>>(lds);
  TimedLaunch t(HK_TK_SCORE_ROWS, st);
  hipLaunchKernelGGL((score_rows_kernel<T, D, QB>), dim3(n_chunks, n_heads), dim3(SCORE_NT), lds, st,
                     static_cast<const T*>(q_obs), static_cast<const T*>(kv->k_pool), kv->page_table,
                     kv->page_mask, kv->n_pages, NS, Hq, Hkv, W, kv->max_pages, L_dense,
                     sm_scale * kLog2e, row_lse, a_rows);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_score_rows_t(int NS, int Hq, int Hkv, int W, const void* q_obs,
                               const hk_paged_kv* kv, int L_dense, float sm_scale,
                               const float* row_lse, float* a_rows, hipStream_t st) {
  switch (qb_eff((Hq / Hkv * W + 31) / 32)) {
    case 1: return launch_score_rows_q<T, D, 1>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
    case 2: return launch_score_rows_q<T, D, 2>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
    case 4: return launch_score_rows_q<T, D, 4>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
    case 7: return launch_score_rows_q<T, D, 7>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
    default: return launch_score_rows_q<T, D, 8>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
  }
}

template <typename T, int D, int QB>
hipError_t launch_score_q(const hk_score_args& a, hipStream_t st) {
  const hk_paged_kv* kv = a.kv;
  constexpr int R_pad = 32 * QB;
  const int n_heads = a.NS * a.Hkv;
  const int n_chunks = (kv->max_pages + SCORE_PPW - 1) / SCORE_PPW;
  const float c2 = a.sm_scale * kLog2e;
  char* ws = static_cast<char*>(a.ws);
  float2* part = reinterpret_cast<float2*>(ws);
  float* lse_buf = a.row_lse_out;
  const size_t off = ((size_t)n_heads * n_chunks * R_pad * sizeof(float2) + 255) & ~(size_t)255;
  if (!lse_buf) lse_buf = reinterpret_cast<float*>(ws + off);
  const float* lse_use = a.row_lse_in;
  dim3 grid(n_chunks, n_heads);
  // bf16 caches: the cooperative passes; fp32 caches (and the redundancy variant of pass 2):
  // the per-wave tile passes
  constexpr bool coop = sizeof(T) == 2;
  if (!lse_use) {
    if constexpr (coop) {
      using Cp = Coop<D, QB>;
      const int nc = (kv->max_pages + Cp::PPW - 1) / Cp::PPW;      // <= n_chunks (workspace size)
      const size_t lds = CoopLds<D, QB>::TOTAL;
      allow_dynamic_lds<score_pass1_coop_kernel<D, QB>>(lds);
      {
        TimedLaunch t(HK_TK_SCORE_PASS1, st);
        hipLaunchKernelGGL((score_pass1_coop_kernel<D, QB>), dim3(nc, n_heads), dim3(Cp::NT), lds, st,
                           static_cast<const uint16_t*>(a.q_obs), static_cast<const uint16_t*>(kv->k_pool),
                           kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                           kv->max_pages, c2, part, nc);
      }
      {
        TimedLaunch t(HK_TK_SCORE_MERGE, st);
        hipLaunchKernelGGL(score_lse_merge_kernel, dim3(n_heads), dim3(256), 0, st, part, nc,
                           R_pad, a.NS, a.Hq, a.Hkv, a.W, c2, a.sm_scale, lse_buf, kv->n_pages,
                           a.L_dense, a.cand_len);
      }
      lse_use = lse_buf;
      if (!a.s_attn) return hipGetLastError();      // row LSEs (and candidate counts) only
    } else {
      const size_t lds1 = pass1_lds(R_pad, D, sizeof(T));
      allow_dynamic_lds<score_pass1_kernel<T, D, QB>>(lds1);
      {
        TimedLaunch t(HK_TK_SCORE_PASS1, st);
        hipLaunchKernelGGL((score_pass1_kernel<T, D, QB>), grid, dim3(SCORE_NT), lds1, st,
                           static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                           kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                           kv->max_pages, c2, part, n_chunks);
      }
      {
        TimedLaunch t(HK_TK_SCORE_MERGE, st);
        hipLaunchKernelGGL(score_lse_merge_kernel, dim3(n_heads), dim3(256), 0, st, part, n_chunks,
                           R_pad, a.NS, a.Hq, a.Hkv, a.W, c2, a.sm_scale, lse_buf, kv->n_pages,
                           a.L_dense, a.cand_len);
      }
      lse_use = lse_buf;
      if (!a.s_attn) return hipGetLastError();      // row LSEs (and candidate counts) only
    }
  } else if (a.row_lse_out && a.row_lse_out != a.row_lse_in) {
    (void)hipMemcpyAsync(a.row_lse_out, a.row_lse_in, sizeof(float) * (size_t)a.W * a.NS * a.Hq,
                         hipMemcpyDeviceToDevice, st);
  }
  const float lnR = logf((float)(a.Hq / a.Hkv * a.W));
  const size_t lds2 = pass2_lds(R_pad, D, sizeof(T), a.x_red != nullptr);
  TimedLaunch t(HK_TK_SCORE_PASS2, st);
  if (a.x_red) {
    constexpr int PPW2 = P2Shape<true>::PPW;
    const dim3 grid2((kv->max_pages + PPW2 - 1) / PPW2, n_heads);
    allow_dynamic_lds<score_pass2_kernel<T, D, QB, true>>(lds2);
    hipLaunchKernelGGL((score_pass2_kernel<T, D, QB, true>), grid2, dim3(P2Shape<true>::NT), lds2, st,
                       static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                       kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                       kv->max_pages, a.L_dense, c2, lnR, lse_use, a.s_attn, a.cand_len,
                       a.ref_slots, a.n_ref, a.x_red);
  } else if constexpr (coop) {
    using Cp = Coop<D, QB>;
    const size_t lds = CoopLds<D, QB>::TOTAL;
    allow_dynamic_lds<score_pass2_coop_kernel<D, QB>>(lds);
    hipLaunchKernelGGL((score_pass2_coop_kernel<D, QB>), dim3((kv->max_pages + Cp::PPW - 1) / Cp::PPW, n_heads),
                       dim3(Cp::NT), lds, st, static_cast<const uint16_t*>(a.q_obs),
                       static_cast<const uint16_t*>(kv->k_pool), kv->page_table, kv->page_mask,
                       kv->n_pages, a.NS, a.Hq, a.Hkv, a.W, kv->max_pages, a.L_dense, c2, lnR, lse_use,
                       a.s_attn, a.cand_len);
  } else {
    allow_dynamic_lds<score_pass2_kernel<T, D, QB, false>>(lds2);
    hipLaunchKernelGGL((score_pass2_kernel<T, D, QB, false>), grid, dim3(P2Shape<false>::NT), lds2, st,
                       static_cast<const T*>(a.q_obs), static_cast<const T*>(kv->k_pool),
                       kv->page_table, kv->page_mask, kv->n_pages, a.NS, a.Hq, a.Hkv, a.W,
                       kv->max_pages, a.L_dense, c2, lnR, lse_use, a.s_attn, a.cand_len,
                       nullptr, 0, nullptr);
  }
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_score_t(const hk_score_args& a, hipStream_t st) {
  switch (qb_eff((a.Hq / a.Hkv * a.W + 31) / 32)) {
    case 1: return launch_score_q<T, D, 1>(a, st);
    case 2: return launch_score_q<T, D, 2>(a, st);
    case 4: return launch_score_q<T, D, 4>(a, st);
    case 7: return launch_score_q<T, D, 7>(a, st);
    default: return launch_score_q<T, D, 8>(a, st);
  }
}

}  // namespace hk

size_t hk_score_ws(int NS, int Hq, int Hkv, int D, int W, int max_pages) {
  (void)D;
  const int R_pad = hk::score_rpad(Hq / Hkv * W);
  const int n_chunks = (max_pages + hk::SCORE_PPW - 1) / hk::SCORE_PPW;
  const size_t part = ((size_t)NS * Hkv * n_chunks * R_pad * sizeof(float2) + 255) & ~(size_t)255;
  const size_t lse = ((size_t)W * NS * Hq * sizeof(float) + 255) & ~(size_t)255;
  return part + lse;
}

size_t hk_score_lds_bytes(int R, int D, int esize, bool redundancy) {
  const int R_pad = hk::score_rpad(R);
  const size_t p1 = hk::pass1_lds(R_pad, D, esize);
  const size_t p2 = hk::pass2_lds(R_pad, D, esize, redundancy);
  return p1 > p2 ? p1 : p2;
}

hipError_t hk_launch_score_rows(int NS, int Hq, int Hkv, int D, int W, const void* q_obs,
                                const hk_paged_kv* kv, int L_dense, float sm_scale,
                                const float* row_lse, float* a_rows, hipStream_t st) {
  const bool bf = kv->dtype == HK_BF16;
  if (bf && D == 128) return hk::launch_score_rows_t<uint16_t, 128>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
  if (bf && D == 64) return hk::launch_score_rows_t<uint16_t, 64>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
  if (!bf && D == 128) return hk::launch_score_rows_t<float, 128>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
  return hk::launch_score_rows_t<float, 64>(NS, Hq, Hkv, W, q_obs, kv, L_dense, sm_scale, row_lse, a_rows, st);
}

hipError_t hk_launch_score(const hk_score_args& a, hipStream_t st) {
  const bool bf = a.kv->dtype == HK_BF16;
  if (bf && a.D == 128) return hk::launch_score_t<uint16_t, 128>(a, st);
  if (bf && a.D == 64) return hk::launch_score_t<uint16_t, 64>(a, st);
  if (!bf && a.D == 128) return hk::launch_score_t<float, 128>(a, st);
  return hk::launch_score_t<float, 64>(a, st);
}

// a5 / a6: paged decode attention over the variable-budget Cascade Cache, and the
// append-only dense-tier write of one decode step (gfx950).
//
// Decode (App. F): every (sequence, KV head) is split into ranges of pages; a workgroup
// computes the attention state (o, m, l) of the G query heads of that KV head over its
// range (each K/V page is read once for all G heads: head expansion), and a merge kernel
// combines the ranges with the merge operator
//   o(I u J) = (o(I) SE(I) + o(J) SE(J)) / (SE(I) + SE(J)),  SE(I u J) = SE(I) + SE(J).
// Only pages below n_pages are visited and page masks drop invalid slots, so the work
// follows each head's own budget: a row's pages are shared by the launch's splits, a split
// past the row's end exits at once, and the merge reads only the splits that held pages.
// Each split stages its page ids and masks in LDS, and every wave keeps the next page's
// loads in flight while it computes the current one.
//
// Lane mapping inside a wave, for one 16-slot page:
//   scores  lane = 4 * t + c: slot t, quarter c of the head dimension; partial dot
//           products are summed over the 4 lanes of a slot with two xor-shuffles;
//   values  lane = LPR * kg + dc: 16-byte chunk dc of the row, slots kg*KPL .. +KPL;
//           the probabilities reach those lanes by shuffles.
#include <mutex>

#include "hk_internal.h"

namespace hk {

constexpr int DEC_NT = 256;                 // threads per workgroup
constexpr int DEC_NW = DEC_NT / 64;
constexpr int DEC_PPS = 128;                // most pages per split (one workgroup)
constexpr int DEC_PPS_MIN = 16;             // fewest pages per split
constexpr int DEC_TARGET_WG = 2048;         // workgroups a launch should offer the chip

// Pages per split for a row of n pages: the row is shared evenly by the launch's n_split
// splits, at least DEC_PPS_MIN pages each and at most pps (never above DEC_PPS).  Split i
// covers pages [i * share, min((i + 1) * share, n)); the splits with i * share >= n hold
// nothing, write nothing, and the merge reads only the ceil(n / share) splits before them.
__device__ __forceinline__ int decode_share(int n, int n_split, int pps) {
  return min(min(pps, DEC_PPS), max((n + n_split - 1) / n_split, DEC_PPS_MIN));
}

template <typename T, int D, int G>
__global__ __launch_bounds__(DEC_NT) void decode_split_kernel(
    const T* __restrict__ q, const T* __restrict__ k_pool, const T* __restrict__ v_pool,
    const int32_t* __restrict__ table, const uint16_t* __restrict__ masks,
    const int32_t* __restrict__ n_pages_arr, int Hq, int Hkv, int max_pages, float c2,
    float* __restrict__ part, int n_split, int pps) {
  constexpr int ES = sizeof(T);
  constexpr int DQ = D / 4;                 // dims per quarter
  constexpr int VEC = 16 / ES;              // elements per 16-byte chunk
  constexpr int LPR = D / VEC;              // lanes per value row
  constexpr int KG = 64 / LPR;              // slot groups
  constexpr int KPL = HK_PAGE / KG;         // slots per lane (values)
  constexpr int QW = DQ * ES / 4;           // 32-bit words of the query quarter
  __shared__ float s_m[DEC_NW][G], s_l[DEC_NW][G];
  __shared__ float s_o[DEC_NW][G][D];

  const int h = blockIdx.y, split = blockIdx.x;
  const int s = h / Hkv, kv = h % Hkv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = min(n_pages_arr[h], max_pages);
  // this head's pages are shared evenly by the launch's splits, so short rows are not left
  // to few waves; a split past the row's end leaves at once (the merge skips it)
  const int per = decode_share(n, n_split, pps);
  const int p_begin = split * per, p_end = min(p_begin + per, n);
  if (p_begin >= n) return;
  const int t = lane >> 2, c = lane & 3;
  const int kg = lane / LPR, dc = lane % LPR;

  // the G query rows of this KV head (contiguous in q), 16 bytes per thread
  __shared__ uint4 s_q[G * D * ES / 16];
  {
    const uint4* src = reinterpret_cast<const uint4*>(q + ((size_t)s * Hq + kv * G) * D);
    for (int i = threadIdx.x; i < G * D * ES / 16; i += DEC_NT) s_q[i] = src[i];
  }
  // the split's page ids and masks, staged once: a page's loads then wait on no global
  // read of the table (the per-share bound above keeps the range within DEC_PPS)
  const int32_t* trow = table + (size_t)h * max_pages;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  __shared__ int32_t s_pid[DEC_PPS];
  __shared__ uint16_t s_pm[DEC_PPS];
  for (int i = threadIdx.x; i < p_end - p_begin; i += DEC_NT) {
    s_pid[i] = trow[p_begin + i];
    s_pm[i] = mrow[p_begin + i];
  }
  __syncthreads();
  const int q_lane = c * DQ * ES / 16;
  auto q_word = [&](int qb, int g, int i) -> uint32_t {
    const uint4 u = s_q[qb + g * D * ES / 16 + i / 4];
    return (i & 3) == 0 ? u.x : (i & 3) == 1 ? u.y : (i & 3) == 2 ? u.z : u.w;
  };
  float m_run[G], l_part[G], o[G][VEC];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = -INFINITY;
    l_part[g] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[g][e] = 0.f;
  }
  struct PageRegs {
    uint4 k[QW / 4];
    uint4 v[KPL];
    uint32_t m16;
  };
  // the wave's pages are p_begin + wave + DEC_NW * j, j < npg; load_page(r, j) reads
  // page min(j, npg - 1) and gives it an empty mask when j >= npg
  const int npg = p_begin + wave < p_end ? (p_end - 1 - p_begin - wave) / DEC_NW + 1 : 0;
  auto load_page = [&](PageRegs& r, int j) {
    const int li = wave + DEC_NW * min(j, npg - 1);
    r.m16 = j < npg ? s_pm[li] : 0u;
    const size_t page = (size_t)s_pid[li] * HK_PAGE;
    const uint4* ks = reinterpret_cast<const uint4*>(k_pool + (page + t) * D + c * DQ);
#pragma unroll
    for (int i = 0; i < QW / 4; ++i) r.k[i] = ks[i];
#pragma unroll
    for (int i = 0; i < KPL; ++i)
      r.v[i] = *reinterpret_cast<const uint4*>(v_pool + (page + kg * KPL + i) * D + dc * VEC);
  };
  auto process_page = [&](const PageRegs& r) {
    const uint32_t m16 = r.m16;
    uint32_t kw[QW];
#pragma unroll
    for (int i = 0; i < QW / 4; ++i) {
      kw[4 * i + 0] = r.k[i].x;
      kw[4 * i + 1] = r.k[i].y;
      kw[4 * i + 2] = r.k[i].z;
      kw[4 * i + 3] = r.k[i].w;
    }
    const bool valid = (m16 >> t) & 1u;
    // the query words are read from LDS for every page (an opaque offset keeps the
    // compiler from hoisting them into 64 more registers per lane)
    int qb = q_lane;
    asm volatile("" : "+v"(qb));
    float zl[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float z = 0.f;
      if constexpr (ES == 2) {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int i = 0; i < QW; ++i)
          z = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, q_word(qb, g, i)),
                                              __builtin_bit_cast(bf16x2, kw[i]), z, false);
      } else {
#pragma unroll
        for (int i = 0; i < QW; ++i) z = fmaf(__uint_as_float(q_word(qb, g, i)), __uint_as_float(kw[i]), z);
      }
      z += __shfl_xor(z, 1, 64);
      z += __shfl_xor(z, 2, 64);
      zl[g] = valid ? z * c2 : -INFINITY;      // log2 units
    }
    float pr[G], alpha[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      // the 4 lanes of a slot hold the same value, so within a 16-lane row the half-row
      // and row mirrors (lane l <-> 7 - l within 8, l <-> 15 - l) meet every slot of the row
      float pm = zl[g];
      pm = fmaxf(pm, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                         0, __builtin_bit_cast(int, pm), 0x141, 0xf, 0xf, false)));
      pm = fmaxf(pm, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                         0, __builtin_bit_cast(int, pm), 0x140, 0xf, 0xf, false)));
      pm = fmaxf(pm, __shfl_xor(pm, 16, 64));
      pm = fmaxf(pm, __shfl_xor(pm, 32, 64));
      // a page with no valid slot leaves the state as it is (alpha 1 or the state still
      // empty, pr 0); the guards keep -inf - -inf out of the exponentials
      const float mn = fmaxf(m_run[g], pm);
      alpha[g] = m_run[g] == -INFINITY ? 0.f : fast_exp2(m_run[g] - mn);
      pr[g] = valid ? fast_exp2(zl[g] - mn) : 0.f;
      m_run[g] = mn;
      l_part[g] = l_part[g] * alpha[g] + (c == 0 ? pr[g] : 0.f);
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[g][e] *= alpha[g];
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int src_lane = 4 * (kg * KPL + i);
      float vf[VEC];
      const uint32_t vv[4] = {r.v[i].x, r.v[i].y, r.v[i].z, r.v[i].w};
      if constexpr (ES == 2) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vf[2 * e] = bf16_lo(vv[e]);
          vf[2 * e + 1] = bf16_hi(vv[e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) vf[e] = __uint_as_float(vv[e]);
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pg = __shfl(pr[g], src_lane, 64);
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[g][e] = fmaf(pg, vf[e], o[g][e]);
      }
    }
  };

  // the wave's next page is loaded (into the other register set) before the current one
  // is processed; the loop is unrolled by two so both sets stay in registers.  Every
  // trip issues both loads and processes both sets (a page past the wave's run is its
  // last page again with an empty mask, which leaves the state as it is), so no load is
  // moved behind the processing it should overlap.
  if (npg > 0) {
    PageRegs ra, rb;
    load_page(ra, 0);
    for (int j = 0; j < npg; j += 2) {
      load_page(rb, j + 1);
      process_page(ra);
      load_page(ra, j + 2);
      process_page(rb);
    }
  }
  // reduce over slot groups (lanes with the same value chunk) and over all lanes for l
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int x = LPR; x < 64; x <<= 1)
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[g][e] += __shfl_xor(o[g][e], x, 64);
    l_part[g] = wave_sum(l_part[g]);
    if (lane == 0) {
      s_m[wave][g] = m_run[g];
      s_l[wave][g] = l_part[g];
    }
    if (lane < LPR)
#pragma unroll
      for (int e = 0; e < VEC; ++e) s_o[wave][g][dc * VEC + e] = o[g][e];
  }
  __syncthreads();
  // combine the waves -> one partial state per (head, split, g): [o(D) unnormalised, m, l]
  for (int idx = threadIdx.x; idx < G * D; idx += DEC_NT) {
    const int g = idx / D, d = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < DEC_NW; ++w) M = fmaxf(M, s_m[w][g]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY)
#pragma unroll
      for (int w = 0; w < DEC_NW; ++w) {
        const float a = fast_exp2(s_m[w][g] - M);
        L += s_l[w][g] * a;
        O += s_o[w][g][d] * a;
      }
    float* dst = part + (((size_t)h * n_split + split) * G + g) * (D + 2);
    dst[d] = O;
    if (d == 0) {
      dst[D] = M;
      dst[D + 1] = L;
    }
  }
}

// One workgroup per KV head merges the split states of its G query heads (App. F).  A
// 32-lane group per query head loads the (m, l) of up to DEC_MRG_CACHE splits once into
// registers, finds the running maximum M and the rescaled sum L from them, and leaves each
// split's factor exp2(m - M) in LDS; then each (query head, dim) thread sums its split
// outputs times those factors.  Only the splits that held pages of the row count (none for
// an empty row, which gives o = 0, lse = -inf).  When the launch has at most
// DEC_MRG_SPEC splits, every load -- the row's page count, the split states, the thread's
// split outputs -- is issued at once, before the count of splits that held pages is known,
// and the states of the others are dropped unread (their memory holds an earlier call's
// values); otherwise the outputs are loaded after the factors, and rows with more splits
// than the register cache read the rest from memory.
constexpr int DEC_MRG_CACHE = 128;            // splits per query head kept in registers / LDS
constexpr int DEC_MRG_SPEC = 8;               // splits loaded before the split count is known
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(const float* __restrict__ part,
                                                           const int32_t* __restrict__ n_pages_arr,
                                                           int max_pages, int n_split_all, int pps,
                                                           int G, int Hq, int Hkv, float* __restrict__ o,
                                                           float* __restrict__ lse) {
  constexpr int KPL = DEC_MRG_CACHE / 32;     // cached splits per lane
  constexpr int OPT = 8 * D / 256;            // outputs per thread at the largest group (8)
  __shared__ float s_M[8], s_L[8];
  __shared__ float s_a[8][DEC_MRG_CACHE];
  const int h = blockIdx.x, s = h / Hkv, kv = h % Hkv;
  const size_t stride = (size_t)G * (D + 2);
  const float* base = part + (size_t)h * n_split_all * stride;
  const bool spec = n_split_all <= DEC_MRG_SPEC;
  const int n = min(n_pages_arr[h], max_pages);
  const int g = threadIdx.x >> 5, l32 = threadIdx.x & 31;
  const float* pg = base + g * (D + 2);
  // split states (speculatively up to n_split_all when spec) and the thread's split outputs
  const int n_load = spec ? n_split_all : 0;
  float mv[KPL], lv[KPL];
#pragma unroll
  for (int k = 0; k < KPL; ++k) {
    const int i = l32 + 32 * k;
    mv[k] = -INFINITY;
    lv[k] = 0.f;
    if (g < G && i < n_load) {
      mv[k] = pg[i * stride + D];
      lv[k] = pg[i * stride + D + 1];
    }
  }
  float ov[OPT][DEC_MRG_SPEC];
  if (spec) {
#pragma unroll
    for (int q = 0; q < OPT; ++q) {
      const int idx = threadIdx.x + 256 * q;
      const int gq = idx / D, d = idx % D;
#pragma unroll
      for (int i = 0; i < DEC_MRG_SPEC; ++i)
        ov[q][i] = (idx < G * D && i < n_split_all) ? base[i * stride + gq * (D + 2) + d] : 0.f;
    }
  }
  const int share = decode_share(n, n_split_all, pps);
  const int n_split = n > 0 ? min(n_split_all, (n + share - 1) / share) : 0;
  {
    float M = -INFINITY, L = 0.f;
#pragma unroll
    for (int k = 0; k < KPL; ++k) {
      const int i = l32 + 32 * k;
      if (g < G && i < n_split && !spec) {
        mv[k] = pg[i * stride + D];
        lv[k] = pg[i * stride + D + 1];
      }
      if (i >= n_split) {                       // a split that held no pages of this row
        mv[k] = -INFINITY;
        lv[k] = 0.f;
      }
      M = fmaxf(M, mv[k]);
    }
    if (g < G)
      for (int i = l32 + DEC_MRG_CACHE; i < n_split; i += 32) M = fmaxf(M, pg[i * stride + D]);
#pragma unroll
    for (int x = 1; x < 32; x <<= 1) M = fmaxf(M, __shfl_xor(M, x, 32));
    if (g < G && M != -INFINITY) {
#pragma unroll
      for (int k = 0; k < KPL; ++k) {
        const float a = exp2f(mv[k] - M);         // 0 for a split past n_split
        L += lv[k] * a;
        s_a[g][l32 + 32 * k] = a;
      }
      for (int i = l32 + DEC_MRG_CACHE; i < n_split; i += 32) {
        const float* p = pg + i * stride;
        L += p[D + 1] * exp2f(p[D] - M);
      }
    }
#pragma unroll
    for (int x = 1; x < 32; x <<= 1) L += __shfl_xor(L, x, 32);
    if (g < G && l32 == 0) {
      s_M[g] = M;
      s_L[g] = L;
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < OPT; ++q) {
    const int idx = threadIdx.x + 256 * q;
    if (idx >= G * D) break;
    const int gq = idx / D, d = idx % D;
    const float M = s_M[gq], L = s_L[gq];
    const float* p = base + gq * (D + 2);
    const float* a = s_a[gq];
    float O0 = 0.f, O1 = 0.f, O2 = 0.f, O3 = 0.f;
    if (M != -INFINITY) {
      if (spec) {
        // the same grouping as below: fours into O0..O3, the rest into O0, slot order
#pragma unroll
        for (int i = 0; i + 4 <= DEC_MRG_SPEC; i += 4)
          if (i + 4 <= n_split) {
            O0 = fmaf(ov[q][i], a[i], O0);
            O1 = fmaf(ov[q][i + 1], a[i + 1], O1);
            O2 = fmaf(ov[q][i + 2], a[i + 2], O2);
            O3 = fmaf(ov[q][i + 3], a[i + 3], O3);
          }
#pragma unroll
        for (int i = 0; i < DEC_MRG_SPEC; ++i)
          if (i >= (n_split & ~3) && i < n_split) O0 = fmaf(ov[q][i], a[i], O0);
      } else {
        const int nc = min(n_split, DEC_MRG_CACHE);
        int i = 0;
        for (; i + 4 <= nc; i += 4) {
          const float* q0 = p + i * stride;
          const float v0 = q0[d], v1 = q0[stride + d], v2 = q0[2 * stride + d], v3 = q0[3 * stride + d];
          O0 = fmaf(v0, a[i], O0);
          O1 = fmaf(v1, a[i + 1], O1);
          O2 = fmaf(v2, a[i + 2], O2);
          O3 = fmaf(v3, a[i + 3], O3);
        }
        for (; i < nc; ++i) O0 = fmaf(p[i * stride + d], a[i], O0);
        for (; i < n_split; ++i) O0 = fmaf(p[i * stride + d], exp2f(p[i * stride + D] - M), O0);
      }
    }
    const float O = (O0 + O1) + (O2 + O3);
    const size_t row = (size_t)s * Hq + kv * G + gq;
    o[row * D + d] = (L > 0.f) ? O / L : 0.f;
    if (d == 0) lse[row] = (L > 0.f) ? (M + __log2f(L)) * kLn2 : -INFINITY;
  }
}

// ------------------------------------------------------------------ a6: append
// Two launches.  Count: one wave per 64 heads records how many of its heads need a fresh
// page (row empty, or newest page full) and whether any such row is already at max_pages,
// and block 0 snapshots the free-list top.  Write: every workgroup re-derives its heads'
// needs, takes the exclusive prefix over the preceding workgroups' counts (head order, so
// the pops are the same as a sequential scan), decides success from the global totals,
// and writes its heads.  Only block 0 updates free_top; every block reads the snapshot.
// Workspace (int32): [0] top snapshot, [1, 1+nblk) counts, [1+nblk, 1+2*nblk) full flags.
constexpr int AP_HPB = 64;     // heads per workgroup
constexpr int AP_NT = 256;

__device__ inline void append_need(int h, int n_heads, const int32_t* n_pages, const uint16_t* masks,
                                   int max_pages, int& n, uint32_t& m, int& need, int& full) {
  n = 0;
  m = 0;
  need = 0;
  full = 0;
  if (h >= n_heads) return;
  n = n_pages[h];
  m = n > 0 ? masks[(size_t)h * max_pages + n - 1] : 0xffffu;
  if ((m & 0x8000u) || n == 0) {
    need = 1;
    full = n >= max_pages;
  }
}

__global__ __launch_bounds__(64) void append_count_kernel(int n_heads, const int32_t* __restrict__ n_pages,
                                                          const uint16_t* __restrict__ masks, int max_pages,
                                                          const int32_t* __restrict__ free_top,
                                                          int32_t* __restrict__ ws) {
  const int nblk = gridDim.x;
  int n, need, full;
  uint32_t m;
  append_need(blockIdx.x * AP_HPB + threadIdx.x, n_heads, n_pages, masks, max_pages, n, m, need, full);
  need = wave_sum(need);
  full = __any(full) ? 1 : 0;
  if (threadIdx.x == 0) {
    ws[1 + blockIdx.x] = need;
    ws[1 + nblk + blockIdx.x] = full;
    if (blockIdx.x == 0) ws[0] = *free_top;
  }
}

template <int ROW_BYTES>
__global__ __launch_bounds__(AP_NT) void append_write_kernel(
    int n_heads, char* __restrict__ k_pool, char* __restrict__ v_pool, int32_t* __restrict__ table,
    uint16_t* __restrict__ masks, int32_t* __restrict__ n_pages, int max_pages,
    const char* __restrict__ k_new, const char* __restrict__ v_new, const int32_t* __restrict__ free_ids,
    int32_t* __restrict__ free_top, int32_t* __restrict__ status, const int32_t* __restrict__ ws) {
  constexpr int CH = ROW_BYTES / 16;
  __shared__ int s_red[3][AP_NT / 64];
  __shared__ int64_t s_dst[AP_HPB];
  const int nblk = gridDim.x, blk = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // global totals and this block's offset, from the counts of the first launch
  int before = 0, total = 0, anyfull = 0;
  for (int b = threadIdx.x; b < nblk; b += AP_NT) {
    const int c = ws[1 + b];
    total += c;
    if (b < blk) before += c;
    anyfull |= ws[1 + nblk + b];
  }
  before = wave_sum(before);
  total = wave_sum(total);
  anyfull = __any(anyfull) ? 1 : 0;
  if (lane == 0) {
    s_red[0][wave] = before;
    s_red[1][wave] = total;
    s_red[2][wave] = anyfull;
  }
  __syncthreads();
  before = total = anyfull = 0;
#pragma unroll
  for (int w = 0; w < AP_NT / 64; ++w) {
    before += s_red[0][w];
    total += s_red[1][w];
    anyfull |= s_red[2][w];
  }
  const int top = ws[0];
  const bool ok = !anyfull && total <= top;
  if (blk == 0 && threadIdx.x == 0) {
    if (ok) *free_top = top - total;
    else if (status) atomicOr(status, HK_FLAG_NOSPACE);
  }
  if (!ok) return;
  if (wave == 0) {
    const int h = blk * AP_HPB + lane;
    int n, need, full;
    uint32_t m;
    append_need(h, n_heads, n_pages, masks, max_pages, n, m, need, full);
    int x = need;   // inclusive scan over the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    int64_t dst = -1;
    if (h < n_heads) {
      int page, slot;
      if (need) {
        page = free_ids[top - total + before + x - 1];
        table[(size_t)h * max_pages + n] = page;
        masks[(size_t)h * max_pages + n] = 1;
        n_pages[h] = n + 1;
        slot = 0;
      } else {
        page = table[(size_t)h * max_pages + n - 1];
        slot = 32 - __clz(m);               // one past the highest valid slot
        masks[(size_t)h * max_pages + n - 1] = (uint16_t)(m | (1u << slot));
      }
      dst = ((int64_t)page * HK_PAGE + slot) * ROW_BYTES;
    }
    s_dst[lane] = dst;
  }
  __syncthreads();
  // rows of the workgroup's heads: K then V, 16-byte chunks, consecutive threads on one row
  const int h0 = blk * AP_HPB;
  for (int i = threadIdx.x; i < 2 * AP_HPB * CH; i += AP_NT) {
    const int kv = i / (AP_HPB * CH), r = i % (AP_HPB * CH);
    const int hl = r / CH, ch = r % CH;
    const int64_t dst = s_dst[hl];
    if (dst < 0) continue;
    const size_t src = (size_t)(h0 + hl) * ROW_BYTES + ch * 16;
    const uint4 u = *reinterpret_cast<const uint4*>((kv ? v_new : k_new) + src);
    *reinterpret_cast<uint4*>((kv ? v_pool : k_pool) + dst + ch * 16) = u;
  }
}

template <typename T, int D, int G>
static void launch_split(dim3 grid, hipStream_t st, const void* q, const hk_paged_kv* kv, int Hq,
                         int Hkv, float c2, float* part, int n_split, int pps) {
  hipLaunchKernelGGL((decode_split_kernel<T, D, G>), grid, dim3(DEC_NT), 0, st,
                     static_cast<const T*>(q), static_cast<const T*>(kv->k_pool),
                     static_cast<const T*>(kv->v_pool), kv->page_table, kv->page_mask, kv->n_pages,
                     Hq, Hkv, kv->max_pages, c2, part, n_split, pps);
}

template <typename T, int D>
static bool launch_split_g(int G, dim3 grid, hipStream_t st, const void* q, const hk_paged_kv* kv,
                           int Hq, int Hkv, float c2, float* part, int n_split, int pps) {
  switch (G) {
    case 1: launch_split<T, D, 1>(grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps); return true;
    case 2: launch_split<T, D, 2>(grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps); return true;
    case 4: launch_split<T, D, 4>(grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps); return true;
    case 7: launch_split<T, D, 7>(grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps); return true;
    case 8: launch_split<T, D, 8>(grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps); return true;
    default: return false;
  }
}

}  // namespace hk

using namespace hk;

bool hk_decode_supports_group(int G) { return G == 1 || G == 2 || G == 4 || G == 7 || G == 8; }

size_t hk_decode_ws(int NS, int Hq, int Hkv, int D, int max_pages) {
  const int G = Hq / Hkv, n_split = (max_pages + DEC_PPS_MIN - 1) / DEC_PPS_MIN;
  return (size_t)NS * Hkv * n_split * G * (D + 2) * sizeof(float);
}

void hk_decode_split_plan(int n_heads, int max_pages, int* pps_out, int* n_split_out) {
  // pages per split: the most (DEC_PPS) that still gives the launch DEC_TARGET_WG
  // workgroups, down to DEC_PPS_MIN -- few heads get short splits, so no wave walks a
  // long serial chain of pages
  int pps = DEC_PPS;
  while (pps > DEC_PPS_MIN && (long long)n_heads * ((max_pages + pps - 1) / pps) < DEC_TARGET_WG)
    pps >>= 1;
  *pps_out = pps;
  *n_split_out = (max_pages + pps - 1) / pps;
}

hipError_t hk_launch_decode(int NS, int Hq, int Hkv, int D, const void* q, const hk_paged_kv* kv,
                            float sm_scale, float* o, float* lse, void* ws, hipStream_t st,
                            bool timed) {
  const int G = Hq / Hkv, n_heads = NS * Hkv;
  int pps, n_split;
  hk_decode_split_plan(n_heads, kv->max_pages, &pps, &n_split);
  const float c2 = sm_scale * kLog2e;
  float* part = static_cast<float*>(ws);
  dim3 grid(n_split, n_heads);
  const bool bf = kv->dtype == HK_BF16;
  bool ok;
  {
  TimedLaunch t(timed ? HK_TK_DECODE_SPLIT : -1, st);
  if (bf && D == 128) ok = launch_split_g<uint16_t, 128>(G, grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps);
  else if (bf) ok = launch_split_g<uint16_t, 64>(G, grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps);
  else if (D == 128) ok = launch_split_g<float, 128>(G, grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps);
  else ok = launch_split_g<float, 64>(G, grid, st, q, kv, Hq, Hkv, c2, part, n_split, pps);
  }
  if (!ok) return hipErrorInvalidValue;
  TimedLaunch t(timed ? HK_TK_DECODE_MERGE : -1, st);
  if (D == 128)
    hipLaunchKernelGGL(decode_merge_kernel<128>, dim3(n_heads), dim3(256), 0, st, part, kv->n_pages,
                       kv->max_pages, n_split, pps, G, Hq, Hkv, o, lse);
  else
    hipLaunchKernelGGL(decode_merge_kernel<64>, dim3(n_heads), dim3(256), 0, st, part, kv->n_pages,
                       kv->max_pages, n_split, pps, G, Hq, Hkv, o, lse);
  return hipGetLastError();
}

// ------------------------------------------------------------------ decode without allocation
// The split partial states of hk_decode_attn_noalloc live in this file-scope device array
// instead of a caller workspace: one copy per GPU the library runs on, held until the
// process ends.  Host code never uses the array's name as an address: its device address is
// looked up once per device (with that device current) and kept here.
static __device__ __align__(256) char scratch[HK_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t hk_noalloc_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

size_t hk_decode_noalloc_bytes(int NS, int Hq, int Hkv, int D, int max_pages) {
  int pps, n_split;
  hk_decode_split_plan(NS * Hkv, max_pages, &pps, &n_split);
  return (size_t)NS * Hkv * n_split * (Hq / Hkv) * (D + 2) * sizeof(float);
}

size_t hk_append_ws(int NS, int Hkv) {
  const int nblk = (NS * Hkv + AP_HPB - 1) / AP_HPB;
  return (size_t)(1 + 2 * nblk) * sizeof(int32_t);
}

hipError_t hk_launch_append(int NS, int Hkv, int D, const hk_paged_kv* kv, const void* k_new,
                            const void* v_new, const hk_allocator* alloc, int32_t* status, void* ws,
                            hipStream_t st) {
  const int n_heads = NS * Hkv, nblk = (n_heads + AP_HPB - 1) / AP_HPB;
  const int row_bytes = D * (kv->dtype == HK_BF16 ? 2 : 4);
  char* kp = static_cast<char*>(kv->k_pool);
  char* vp = static_cast<char*>(kv->v_pool);
  const char* kn = static_cast<const char*>(k_new);
  const char* vn = static_cast<const char*>(v_new);
  int32_t* w = static_cast<int32_t*>(ws);
  TimedLaunch t(HK_TK_APPEND, st);
  hipLaunchKernelGGL(append_count_kernel, dim3(nblk), dim3(64), 0, st, n_heads, kv->n_pages,
                     kv->page_mask, kv->max_pages, alloc->free_top, w);
#define HK_APPEND_WRITE(RB)                                                                       \
  hipLaunchKernelGGL((append_write_kernel<RB>), dim3(nblk), dim3(AP_NT), 0, st, n_heads, kp, vp, \
                     kv->page_table, kv->page_mask, kv->n_pages, kv->max_pages, kn, vn,           \
                     alloc->free_ids, alloc->free_top, status, w)
  switch (row_bytes) {
    case 128: HK_APPEND_WRITE(128); break;
    case 256: HK_APPEND_WRITE(256); break;
    default: HK_APPEND_WRITE(512); break;
  }
#undef HK_APPEND_WRITE
  return hipGetLastError();
}

// Step 4 of the compression pipeline (Sec. 3.1): the hard budget, with Cautious Update
// voting and attention sinks (gfx950).
//
//   vote_topp    one workgroup per (head, group of window rows): each row's own Top-p
//                set of the candidates under its attention probabilities (the a3 rule),
//                written as a per-row bitmap, found by a radix search over the keys;
//   vote_count   votes[h][j] = number of rows whose set holds j (column bit counts);
//   budget_plan  one wave per head: the head's state from its page count and valid slots
//                against L_lower / L_upper, and its cap;
//   budget_select one workgroup per head: sinks, then the base set ranked by (votes, c,
//                slot) and cut at the cap by a radix search on the 64-bit rank key.
//
// Layout: 512 threads per workgroup; slot j of a row is thread j % 512's element j / 512,
// so a wave's 64 lanes cover 64 consecutive slots (coalesced loads; one ballot gives two
// words of a bitmap).  A row's keys stay in registers (S_max <= 32768 -> <= 64 each).
#include "hk_internal.h"

namespace hk {

constexpr int BG_NT = 512;
constexpr int BG_NW = BG_NT / 64;
constexpr int RADIX_BITS = 11;
constexpr int RADIX_BINS = 1 << RADIX_BITS;
constexpr int BINS_PER_THREAD = RADIX_BINS / BG_NT;
constexpr int BG_EPT_MAX = 64;
constexpr float kMassScale = 1099511627776.0f;   // 2^40, fixed-point unit of the Top-p mass

struct BgLds {
  unsigned long long hist[RADIX_BINS];
  unsigned long long red64[BG_NW];
  uint32_t redu[2][BG_NW];
  int redi[BG_NW];
  int tiecnt[BG_EPT_MAX * BG_NW];
  unsigned long long pick_above;
  uint32_t pick_digit;
};

// floor(v * 2^40) for a probability v in [0, 1]: the product is exact in fp32 (a power of
// two scale) with at most 24 significant bits, so truncation gives the integer exactly.
__device__ __forceinline__ unsigned long long mass_weight(uint32_t key) {
  return (unsigned long long)truncf(__uint_as_float(key) * kMassScale);
}

// A copy of x the compiler cannot see through.  Per-element predicates such as
// (flags >> i) & 1 are otherwise computed once and kept, as EPT lane masks in scalar
// registers, across every loop that tests them; that overflows the scalar file.  Testing
// a fresh copy in each loop keeps each mask short-lived.
template <typename X>
__device__ __forceinline__ X opaque(X x) {
  asm volatile("" : "+v"(x));
  return x;
}

template <typename K>
__device__ __forceinline__ K low_mask(int pos) {
  constexpr int KB = 8 * sizeof(K);
  return pos >= KB ? ~K(0) : (K(1) << pos) - K(1);
}
template <typename K>
__device__ __forceinline__ int highest_bit(K x) {   // x != 0
  if constexpr (sizeof(K) == 8) return 63 - __clzll((long long)x);
  else return 31 - __clz((int)x);
}

// wave-wide min / max of 64-bit keys on DPP moves of both halves
template <bool MAX>
__device__ __forceinline__ uint64_t wave_minmax_u64(uint64_t v) {
  const uint64_t id = MAX ? 0ull : ~0ull;
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#define HK_MM_STEP(CTRL, RM)                                                                      \
  {                                                                                               \
    const uint64_t o = ((uint64_t)dpp_u32<CTRL, RM>(hi, (uint32_t)(id >> 32)) << 32) |            \
                       dpp_u32<CTRL, RM>(lo, (uint32_t)id);                                       \
    const uint64_t c = ((uint64_t)hi << 32) | lo;                                                 \
    const uint64_t r = MAX ? (o > c ? o : c) : (o < c ? o : c);                                   \
    lo = (uint32_t)r;                                                                             \
    hi = (uint32_t)(r >> 32);                                                                     \
  }
  HK_MM_STEP(0xb1, 0xf)
  HK_MM_STEP(0x4e, 0xf)
  HK_MM_STEP(0x141, 0xf)
  HK_MM_STEP(0x140, 0xf)
  HK_MM_STEP(0x142, 0xa)
  HK_MM_STEP(0x143, 0xc)
#undef HK_MM_STEP
  lo = (uint32_t)__builtin_amdgcn_readlane((int)lo, 63);
  hi = (uint32_t)__builtin_amdgcn_readlane((int)hi, 63);
  return ((uint64_t)hi << 32) | lo;
}

// Block minimum and maximum of one key per thread (u32 or u64 keys).
template <typename K>
__device__ __forceinline__ void block_key_range(K kmin, K kmax, BgLds& sh, K* out_min, K* out_max) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if constexpr (sizeof(K) == 8) {
    kmin = wave_minmax_u64<false>(kmin);
    kmax = wave_minmax_u64<true>(kmax);
    __syncthreads();
    if (l == 0) {
      sh.red64[w] = kmin;
      sh.hist[w] = kmax;            // the histogram is not live during this reduction
    }
    __syncthreads();
    K a = sh.red64[0], b = sh.hist[0];
#pragma unroll
    for (int i = 1; i < BG_NW; ++i) {
      a = min(a, (K)sh.red64[i]);
      b = max(b, (K)sh.hist[i]);
    }
    *out_min = a;
    *out_max = b;
  } else {
    kmin = wave_reduce_u32(kmin, 0xffffffffu, [](uint32_t a, uint32_t b) { return a < b ? a : b; });
    kmax = wave_reduce_u32(kmax, 0u, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    __syncthreads();
    if (l == 0) {
      sh.redu[0][w] = kmin;
      sh.redu[1][w] = kmax;
    }
    __syncthreads();
    K a = sh.redu[0][0], b = sh.redu[1][0];
#pragma unroll
    for (int i = 1; i < BG_NW; ++i) {
      a = min(a, (K)sh.redu[0][i]);
      b = max(b, (K)sh.redu[1][i]);
    }
    *out_min = a;
    *out_max = b;
  }
}

// Largest key v of the flagged elements with W(key >= v) >= target, where W sums the
// elements' weights (weight(key) of each); requires 0 < target <= W(all flagged).  The
// bits above the highest one where the flagged keys differ are common to all of them,
// hence to v; below them v is found RADIX_BITS at a time from a histogram of weights per
// digit (LDS atomics) and a suffix scan over the digits.  Returns v and, in *above,
// W(key > v).
template <int EPT, typename K, typename WF>
__device__ __forceinline__ K radix_threshold(const K* key, uint64_t flags, unsigned long long target,
                                             WF weight, K kmin, K kmax, BgLds& sh,
                                             unsigned long long* above_out) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (kmin == kmax) {
    *above_out = 0;
    return kmin;
  }
  int pos = highest_bit<K>(kmin ^ kmax) + 1;
  K prefix = kmin & ~low_mask<K>(pos);
  unsigned long long above = 0;
  while (pos > 0) {
    const int nb = min(RADIX_BITS, pos), lo = pos - nb;
    const K hi_mask = ~low_mask<K>(pos);
    const uint32_t dmask = (1u << nb) - 1u;
    __syncthreads();                 // earlier readers of the LDS scratch are done
#pragma unroll
    for (int b = 0; b < BINS_PER_THREAD; ++b) sh.hist[tid * BINS_PER_THREAD + b] = 0ull;
    __syncthreads();
    const uint64_t fl = opaque(flags);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      // (an opaque key keeps the compiler from hoisting the EPT weights, which do not
      // change between rounds, into registers of their own: they would spill)
      const K k = opaque(key[i]);
      if (((fl >> i) & 1ull) && (k & hi_mask) == prefix) {
        const unsigned long long wt = weight(k);
        if (wt) atomicAdd(&sh.hist[(uint32_t)(k >> lo) & dmask], wt);
      }
    }
    __syncthreads();
    // thread t owns digits [t * BPT, (t + 1) * BPT); suffix sums over threads
    unsigned long long own = 0;
#pragma unroll
    for (int b = 0; b < BINS_PER_THREAD; ++b) own += sh.hist[tid * BINS_PER_THREAD + b];
    unsigned long long x = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned long long y = __shfl_down(x, o, 64);
      if (lane + o < 64) x += y;
    }
    if (lane == 0) sh.red64[wave] = x;
    __syncthreads();
    unsigned long long suf = x - own;
    for (int w = wave + 1; w < BG_NW; ++w) suf += sh.red64[w];
    const unsigned long long lo_m = above + suf;
    if (lo_m < target && lo_m + own >= target) {
      unsigned long long cum = lo_m;
      for (int b = BINS_PER_THREAD - 1; b >= 0; --b) {
        const unsigned long long nxt = cum + sh.hist[tid * BINS_PER_THREAD + b];
        if (nxt >= target) {
          sh.pick_digit = (uint32_t)(tid * BINS_PER_THREAD + b);
          sh.pick_above = cum;
          break;
        }
        cum = nxt;
      }
    }
    __syncthreads();
    prefix |= (K)sh.pick_digit << lo;
    above = sh.pick_above;
    pos = lo;
  }
  *above_out = above;
  return prefix;
}

// Among the elements flagged in `tie`, select the `take` with the largest slot index
// (slot = tid + BG_NT * i: later elements, then later waves, then higher lanes).
template <int EPT>
__device__ __forceinline__ uint64_t take_top_ties_bg(uint64_t tie, int take, int* cnt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const unsigned long long b = __ballot((tie >> i) & 1ull);
    if (lane == 0) cnt[i * BG_NW + wave] = __popcll(b);
  }
  __syncthreads();
  uint64_t out = 0;
  int above_rows = 0;
  tie = opaque(tie);                 // ballots taken again, not kept from the loop above
#pragma unroll
  for (int i = EPT - 1; i >= 0; --i) {
    int above = above_rows;
    for (int w = wave + 1; w < BG_NW; ++w) above += cnt[i * BG_NW + w];
    const unsigned long long b = __ballot((tie >> i) & 1ull);
    const unsigned long long hi = (lane == 63) ? 0ull : (b >> (lane + 1));
    above += __popcll(hi);
    if (((tie >> i) & 1ull) && above < take) out |= 1ull << i;
    int row = 0;
    for (int w = 0; w < BG_NW; ++w) row += cnt[i * BG_NW + w];
    above_rows += row;
  }
  return out;
}

template <int EPT>
__device__ __forceinline__ uint64_t cand_flags(int h, int S_max, const int32_t* __restrict__ cand_len,
                                               const uint16_t* __restrict__ mask) {
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  uint64_t f = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = threadIdx.x + BG_NT * i;
    if (j < S_max && is_cand(mrow, cl, j)) f |= 1ull << i;
  }
  return f;
}

// One bitmap row from per-element selection flags.
template <int EPT>
__device__ __forceinline__ void write_bitmap(uint64_t sel, uint32_t* __restrict__ brow, int S_max) {
  // addresses and bounds computed afresh on each call: hoisted out of a row loop they would
  // hold registers per element for the whole loop
  const int lane = threadIdx.x & 63, wave = opaque((int)(threadIdx.x >> 6));
  S_max = opaque(S_max);
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const unsigned long long b = __ballot((sel >> i) & 1ull);
    const int j0 = BG_NT * i + 64 * wave;
    if (lane == 0 && j0 < S_max) {
      brow[j0 / 32] = (uint32_t)b;
      if (j0 + 32 < S_max) brow[j0 / 32 + 1] = (uint32_t)(b >> 32);
    }
  }
}

// ------------------------------------------------------------------ Cautious Update votes
template <int EPT>
__global__ __launch_bounds__(BG_NT) void vote_topp_kernel(
    int R, int S_max, int rows_per_wg, const int32_t* __restrict__ cand_len,
    const uint16_t* __restrict__ mask, const float* __restrict__ a_rows, int p_q,
    uint32_t* __restrict__ row_sel, int32_t* __restrict__ row_k, int32_t* __restrict__ status) {
  __shared__ BgLds sh;
  const int h = blockIdx.y, tid = threadIdx.x;
  const uint64_t cf = cand_flags<EPT>(h, S_max, cand_len, mask);
  const int n_cand = block_sum_int<BG_NT>(__popcll(cf), sh.redi);
  const int r0 = blockIdx.x * rows_per_wg, r1 = min(R, r0 + rows_per_wg);
  int flags_all = 0;
  for (int r = r0; r < r1; ++r) {
    const float* arow = a_rows + ((size_t)h * R + r) * S_max;
    const int t = opaque(tid);       // per-row copy: element addresses are not hoisted
    uint32_t key[EPT];
    int flags = 0;
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    double m = 0.0;
    const uint64_t f1 = opaque(cf);  // per-row copy: per-element tests are not hoisted
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      float v = 0.f;
      if ((f1 >> i) & 1ull) {
        v = arow[t + BG_NT * i];
        if (v != v) { v = 0.f; flags |= HK_FLAG_NAN; }
        if (v > 1.f) { v = 1.f; flags |= HK_FLAG_RANGE; }
        if (v < 0.f) { v = 0.f; flags |= HK_FLAG_RANGE; }
        if (v == 0.f) v = 0.f;                    // canonical +0
      }
      key[i] = __float_as_uint(v);
      if ((f1 >> i) & 1ull) {
        kmin = min(kmin, key[i]);
        kmax = max(kmax, key[i]);
        m += (double)truncf(v * kMassScale);      // exact: see mass_weight
      }
    }
    flags_all |= flags;
    const unsigned long long tot = block_sum_u64<BG_NT>((unsigned long long)m, sh.red64);
    block_key_range<uint32_t>(kmin, kmax, sh, &kmin, &kmax);
    const unsigned long long pq = (unsigned long long)p_q;
    const unsigned long long target =
        pq * (tot / 1000000ull) + (pq * (tot % 1000000ull) + 999999ull) / 1000000ull;
    uint32_t v = 0xffffffffu;
    int take = 0, k = 0;
    if (target > 0) {
      unsigned long long mass_gt = 0;
      v = radix_threshold<EPT, uint32_t>(key, f1, target, [](uint32_t k) { return mass_weight(k); },
                                         kmin, kmax, sh, &mass_gt);
      const unsigned long long wv = mass_weight(v);         // > 0: the crossing element weighs
      take = (int)((target - mass_gt + wv - 1) / wv);
      int gt = 0;
      const uint64_t f2 = opaque(cf);
#pragma unroll
      for (int i = 0; i < EPT; ++i) gt += (((f2 >> i) & 1ull) && opaque(key[i]) > v) ? 1 : 0;
      k = block_sum_int<BG_NT>(gt, sh.redi) + take;
    } else if (n_cand > 0) {
      // no mass to reach: k_min = 1 keeps the largest value, the most recent on ties
      v = kmax;
      take = 1;
      k = 1;
    }
    uint64_t sel = 0, tie = 0;
    const uint64_t f3 = opaque(cf);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const uint32_t k = opaque(key[i]);
      if ((f3 >> i) & 1ull) {
        if (v != 0xffffffffu && k > v) sel |= 1ull << i;
        if (k == v) tie |= 1ull << i;
      }
    }
    const int n_tie = block_sum_int<BG_NT>(__popcll(tie), sh.redi);
    if (take >= n_tie) sel |= tie;
    else if (take > 0) sel |= take_top_ties_bg<EPT>(tie, take, sh.tiecnt);
    write_bitmap<EPT>(sel, row_sel + ((size_t)h * R + r) * (S_max / 32), S_max);
    if (row_k && tid == 0) row_k[(size_t)h * R + r] = k;
  }
  if (status) {
    const int any_nan = __syncthreads_or(flags_all & HK_FLAG_NAN);
    const int any_range = __syncthreads_or(flags_all & HK_FLAG_RANGE);
    if (tid == 0 && (any_nan || any_range))
      atomicOr(status, (any_nan ? HK_FLAG_NAN : 0) | (any_range ? HK_FLAG_RANGE : 0));
  }
}

// votes[h][j] = sum over the R rows of bit j of row_sel[h][r]; one thread per 32-slot word
constexpr int VC_NT = 256;
__global__ __launch_bounds__(VC_NT) void vote_count_kernel(int R, int S_max,
                                                           const uint32_t* __restrict__ row_sel,
                                                           uint16_t* __restrict__ votes) {
  const int h = blockIdx.y;
  const int nw = S_max / 32;
  const int w = blockIdx.x * VC_NT + threadIdx.x;
  if (w >= nw) return;
  uint32_t cnt[32];
#pragma unroll
  for (int b = 0; b < 32; ++b) cnt[b] = 0;
  const uint32_t* base = row_sel + (size_t)h * R * nw + w;
  for (int r = 0; r < R; ++r) {
    const uint32_t x = base[(size_t)r * nw];
#pragma unroll
    for (int b = 0; b < 32; ++b) cnt[b] += (x >> b) & 1u;
  }
  uint4* out = reinterpret_cast<uint4*>(votes + (size_t)h * S_max + (size_t)w * 32);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint4 u;
    u.x = cnt[8 * q + 0] | (cnt[8 * q + 1] << 16);
    u.y = cnt[8 * q + 2] | (cnt[8 * q + 3] << 16);
    u.z = cnt[8 * q + 4] | (cnt[8 * q + 5] << 16);
    u.w = cnt[8 * q + 6] | (cnt[8 * q + 7] << 16);
    out[q] = u;
  }
}

// ------------------------------------------------------------------ budget state
// One wave per head: used = 16 n_pages, valid = set mask bits.
__global__ __launch_bounds__(256) void budget_plan_kernel(int n_heads, int max_pages,
                                                          const int32_t* __restrict__ n_pages,
                                                          const uint16_t* __restrict__ mask,
                                                          int L_dense, int L_lower, int L_upper,
                                                          int32_t* __restrict__ mode_out,
                                                          int32_t* __restrict__ cap_out) {
  const int h = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (h >= n_heads) return;
  const int n = n_pages[h];
  const uint16_t* mrow = mask + (size_t)h * max_pages;
  int valid = 0;
  for (int pp = lane; pp < n; pp += 64) valid += __popc((uint32_t)mrow[pp]);
  valid = wave_sum_i(valid);
  if (lane == 0) {
    const int nd = min(n, dense_pages(L_dense));
    int mode = HK_BUDGET_KEEP, cap = -1;
    if (HK_PAGE * (long long)n > L_upper) {
      mode = HK_BUDGET_REWRITE;
      cap = max(0, HK_PAGE * (L_upper / HK_PAGE) - HK_PAGE * nd);
    } else if (valid > L_lower) {
      mode = HK_BUDGET_SPARSE;
    }
    mode_out[h] = mode;
    cap_out[h] = cap;
  }
}

// ------------------------------------------------------------------ budget selection
template <int EPT>
__global__ __launch_bounds__(BG_NT) void budget_select_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const uint16_t* __restrict__ votes, const float* __restrict__ c, const uint32_t* __restrict__ sel_in,
    const int32_t* __restrict__ head_mode, const int32_t* __restrict__ k_cap, int n_sink,
    uint32_t* __restrict__ sel_out, int32_t* __restrict__ k_out) {
  __shared__ BgLds sh;
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint64_t cf = cand_flags<EPT>(h, S_max, cand_len, mask);
  const int mode = head_mode ? head_mode[h] : HK_BUDGET_REWRITE;
  uint32_t* brow = sel_out + (size_t)h * (S_max / 32);
  if (mode == HK_BUDGET_KEEP) {
    write_bitmap<EPT>(cf, brow, S_max);
    const int n = block_sum_int<BG_NT>(__popcll(cf), sh.redi);
    if (tid == 0) k_out[h] = n;
    return;
  }
  const uint16_t* vrow = votes ? votes + (size_t)h * S_max : nullptr;
  const float* crow = c ? c + (size_t)h * S_max : nullptr;
  const uint32_t* srow = sel_in ? sel_in + (size_t)h * (S_max / 32) : nullptr;
  uint64_t sinks = 0, base = 0;
  uint64_t key[EPT];
  uint64_t kmin = ~0ull, kmax = 0ull;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = tid + BG_NT * i;
    key[i] = 0;
    if (!((cf >> i) & 1ull)) continue;
    if (j < n_sink) {
      sinks |= 1ull << i;
      continue;
    }
    const uint32_t vt = vrow ? (uint32_t)vrow[j] : 0u;
    if (vrow && vt == 0u) continue;
    if (srow && !((srow[j >> 5] >> (j & 31)) & 1u)) continue;
    float cv = crow ? crow[j] : 0.f;
    if (cv != cv) cv = 0.f;
    cv = fminf(fmaxf(cv, 0.f), 1.f);
    if (cv == 0.f) cv = 0.f;                      // canonical +0
    key[i] = ((uint64_t)vt << 32) | __float_as_uint(cv);
    base |= 1ull << i;
    kmin = min(kmin, key[i]);
    kmax = max(kmax, key[i]);
  }
  const int n_sinks = block_sum_int<BG_NT>(__popcll(sinks), sh.redi);
  const int n_base = block_sum_int<BG_NT>(__popcll(base), sh.redi);
  const int kc = k_cap ? k_cap[h] : -1;
  const int cap = kc < 0 ? n_base : min(n_base, max(0, kc - n_sinks));
  uint64_t sel = sinks;
  if (cap >= n_base) {
    sel |= base;
  } else if (cap > 0) {
    block_key_range<uint64_t>(kmin, kmax, sh, &kmin, &kmax);
    unsigned long long cnt_gt = 0;
    const uint64_t v = radix_threshold<EPT, uint64_t>(key, base, (unsigned long long)cap,
                                                      [](uint64_t) { return 1ull; }, kmin, kmax, sh, &cnt_gt);
    const int take = cap - (int)cnt_gt;
    uint64_t tie = 0;
    const uint64_t fb = opaque(base);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const uint64_t k = opaque(key[i]);
      if ((fb >> i) & 1ull) {
        if (k > v) sel |= 1ull << i;
        if (k == v) tie |= 1ull << i;
      }
    }
    const int n_tie = block_sum_int<BG_NT>(__popcll(tie), sh.redi);
    if (take >= n_tie) sel |= tie;
    else if (take > 0) sel |= take_top_ties_bg<EPT>(tie, take, sh.tiecnt);
  }
  write_bitmap<EPT>(sel, brow, S_max);
  if (tid == 0) k_out[h] = n_sinks + cap;
}

template <template <int> class Launch, typename... A>
hipError_t by_ept(int S_max, A... args) {
  const int e = (S_max + BG_NT - 1) / BG_NT;
  if (e <= 1) return Launch<1>::run(args...);
  if (e <= 2) return Launch<2>::run(args...);
  if (e <= 4) return Launch<4>::run(args...);
  if (e <= 8) return Launch<8>::run(args...);
  if (e <= 16) return Launch<16>::run(args...);
  if (e <= 32) return Launch<32>::run(args...);
  return Launch<64>::run(args...);
}

template <int EPT>
struct VoteLaunch {
  static hipError_t run(int n_heads, int R, int S_max, const int32_t* cand_len, const uint16_t* mask,
                        const float* a_rows, int p_q, uint32_t* row_sel, int32_t* row_k,
                        int32_t* status, uint16_t* votes, hipStream_t st) {
    // enough row groups to fill the chip several times over, a few rows per workgroup
    int rows_per_wg = 1;
    while (rows_per_wg < 8 && (long long)n_heads * ((R + 2 * rows_per_wg - 1) / (2 * rows_per_wg)) >= 4096)
      rows_per_wg *= 2;
    {
      TimedLaunch t(HK_TK_VOTE, st);
      hipLaunchKernelGGL((vote_topp_kernel<EPT>), dim3((R + rows_per_wg - 1) / rows_per_wg, n_heads),
                         dim3(BG_NT), 0, st, R, S_max, rows_per_wg, cand_len, mask, a_rows, p_q,
                         row_sel, row_k, status);
    }
    {
      TimedLaunch t(HK_TK_VOTE_COUNT, st);
      const int nw = S_max / 32;
      hipLaunchKernelGGL(vote_count_kernel, dim3((nw + VC_NT - 1) / VC_NT, n_heads), dim3(VC_NT), 0,
                         st, R, S_max, row_sel, votes);
    }
    return hipGetLastError();
  }
};

template <int EPT>
struct BudgetSelectLaunch {
  static hipError_t run(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                        const uint16_t* votes, const float* c, const uint32_t* sel_in,
                        const int32_t* head_mode, const int32_t* k_cap, int n_sink, uint32_t* sel_out,
                        int32_t* k_out, hipStream_t st) {
    TimedLaunch t(HK_TK_BUDGET_SELECT, st);
    hipLaunchKernelGGL((budget_select_kernel<EPT>), dim3(n_heads), dim3(BG_NT), 0, st, S_max, cand_len,
                       mask, votes, c, sel_in, head_mode, k_cap, n_sink, sel_out, k_out);
    return hipGetLastError();
  }
};

}  // namespace hk

using namespace hk;

hipError_t hk_launch_vote_topp(int n_heads, int R, int S_max, const int32_t* cand_len,
                               const uint16_t* mask, const float* a_rows, int p_q, uint16_t* votes,
                               int32_t* row_k, uint32_t* row_sel, int32_t* status, hipStream_t st) {
  return by_ept<VoteLaunch>(S_max, n_heads, R, S_max, cand_len, mask, a_rows, p_q, row_sel, row_k,
                            status, votes, st);
}

hipError_t hk_launch_budget_plan(int n_heads, int max_pages, const int32_t* n_pages,
                                 const uint16_t* mask, int L_dense, int L_lower, int L_upper,
                                 int32_t* head_mode, int32_t* k_cap, hipStream_t st) {
  TimedLaunch t(HK_TK_BUDGET_PLAN, st);
  hipLaunchKernelGGL(budget_plan_kernel, dim3((n_heads + 3) / 4), dim3(256), 0, st, n_heads, max_pages,
                     n_pages, mask, L_dense, L_lower, L_upper, head_mode, k_cap);
  return hipGetLastError();
}

hipError_t hk_launch_budget_select(int n_heads, int S_max, const int32_t* cand_len,
                                   const uint16_t* mask, const uint16_t* votes, const float* c,
                                   const uint32_t* sel_in, const int32_t* head_mode,
                                   const int32_t* k_cap, int n_sink, uint32_t* sel_out,
                                   int32_t* k_out, hipStream_t st) {
  return by_ept<BudgetSelectLaunch>(S_max, n_heads, S_max, cand_len, mask, votes, c, sel_in, head_mode,
                                    k_cap, n_sink, sel_out, k_out, st);
}

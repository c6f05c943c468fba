// Step 4 of the compression pipeline (Sec. 3.1): the hard budget, with Cautious Update
// voting and attention sinks (gfx950).
//
//   vote_topp    one workgroup per (head, window row): the row's own Top-p
//                set of the candidates under its attention probabilities (the a3 rule),
//                written as a per-row bitmap, found by a radix search over the keys;
//   vote_count   votes[h][j] = number of rows whose set holds j (column bit counts);
//   budget_plan  one wave per head: the head's state from its page count and valid slots
//                against L_lower / L_upper, and its cap;
//   budget_select one workgroup per head: sinks, then the base set ranked by (votes, c,
//                slot) and cut at the cap by a radix search on the 64-bit rank key.
//
// Layout: NT threads per workgroup (512 up to 32768 slots, 1024 up to 65536); slot j of a
// row is thread j % NT's element j / NT, so a wave's 64 lanes cover 64 consecutive slots
// (coalesced loads; one ballot gives two words of a bitmap).  A row's keys stay in
// registers (at most 64 each).
#include "hk_internal.h"

namespace hk {

constexpr int RADIX_BITS = 11;
constexpr int RADIX_BINS = 1 << RADIX_BITS;
constexpr int BG_EPT_MAX = 64;
constexpr int BG_SLOTS_512 = 512 * BG_EPT_MAX;    // rows up to this many slots take 512 threads

constexpr int BG_LIST_BYTES = 32768;   // keys of the boundary digit, staged for later rounds

template <int NT>
struct BgLds {
  static constexpr int NW = NT / 64;
  static constexpr int BPT = RADIX_BINS / NT;    // histogram digits per thread
  unsigned long long hist[RADIX_BINS];
  uint32_t list[BG_LIST_BYTES / 4];
  uint16_t mrow[BG_EPT_MAX * NT / HK_PAGE];      // the head's page masks
  unsigned long long red64[NW];
  uint32_t redu[2][NW];
  int redi[NW];
  int tiecnt[BG_EPT_MAX * NW];
  unsigned long long pick_above;
  uint32_t pick_digit;
};

// floor(v * 2^40) for a probability v in [0, 1], as its two 32-bit halves: with t = v * 2^8
// (exact, t <= 256) the high half is floor(t) and the low half floor(fract(t) * 2^32); the
// fraction and its scaling are exact in fp32, so each truncation gives its integer exactly.
__device__ __forceinline__ unsigned long long mass_weight(uint32_t key) {
  const float t = __uint_as_float(key) * 256.0f;
  const uint32_t hi = (uint32_t)t;
  const uint32_t lo = (uint32_t)(__builtin_amdgcn_fractf(t) * 4294967296.0f);
  return ((unsigned long long)hi << 32) | lo;
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
template <typename K, int NT>
__device__ __forceinline__ void block_key_range(K kmin, K kmax, BgLds<NT>& sh, K* out_min, K* out_max) {
  constexpr int BG_NW = NT / 64;
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

template <int NT>
__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* red) {
  constexpr int BG_NW = NT / 64;
  v = wave_reduce_u32(v, 0u, [](uint32_t a, uint32_t b) { return a + b; });
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < BG_NW; ++i) r += red[i];
  return r;
}

// Exclusive prefix (thread order) of one int per thread (.x) and the block sum (.y).
template <int NT>
__device__ __forceinline__ int2 block_exscan_bg(int v, int* red) {
  constexpr int BG_NW = NT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) red[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < BG_NW; ++w) {
    if (w < wave) before += red[w];
    all += red[w];
  }
  return make_int2(before + x - v, all);
}

// After a histogram round: the largest digit d with above + W(digits >= d) >= target, and
// above + W(digits > d).  Thread t owns digits [t * BPT, (t + 1) * BPT); a suffix scan over
// the threads' sums finds the one thread whose digits hold the crossing.
// On the first round the target is not known yet: it is target_of(the histogram's total),
// which is every member's weight; it comes back in *target (0: nothing to reach, no digit).
template <int NT, typename TF>
__device__ __forceinline__ void pick_digit(BgLds<NT>& sh, bool first, TF target_of,
                                           unsigned long long* target_io,
                                           unsigned long long above, uint32_t* d_out,
                                           unsigned long long* above_out) {
  constexpr int BG_NW = NT / 64, BINS_PER_THREAD = RADIX_BINS / NT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
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
  if (first) {
    unsigned long long total = 0;
#pragma unroll
    for (int w = 0; w < BG_NW; ++w) total += sh.red64[w];
    *target_io = target_of(total);
  }
  const unsigned long long target = *target_io;
  if (target == 0) return;
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
  *d_out = sh.pick_digit;
  *above_out = sh.pick_above;
}

// Zero the histogram between two barriers.
template <int NT>
__device__ __forceinline__ void clear_hist(BgLds<NT>& sh) {
  constexpr int BINS_PER_THREAD = RADIX_BINS / NT;
  const int tid = threadIdx.x;
  __syncthreads();                   // earlier readers of the LDS scratch are done
#pragma unroll
  for (int b = 0; b < BINS_PER_THREAD; ++b) sh.hist[tid * BINS_PER_THREAD + b] = 0ull;
  __syncthreads();
}

// Stage into the LDS list the keys whose bits from `pos` up equal `prefix`, if they fit;
// returns their number, or -1 when they do not fit (later rounds then read the registers).
// Each thread counts its own, an exclusive scan gives its offset, and it writes them there.
template <int EPT, typename K, int NT>
__device__ __forceinline__ int stage_list(const K* key, int pos, K prefix, BgLds<NT>& sh) {
  constexpr int CAP = BG_LIST_BYTES / (int)sizeof(K);
  K* list = reinterpret_cast<K*>(sh.list);
  const K m2 = ~low_mask<K>(pos);
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) cnt += ((key[i] & m2) == prefix) ? 1 : 0;
  const int2 sc = block_exscan_bg<NT>(cnt, sh.redi);
  if (sc.y > CAP) return -1;
  int off = sc.x;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const K k = key[i];
    if ((k & m2) == prefix) list[off++] = k;
  }
  return sc.y;
}

// Largest key v of the member elements with W(key >= v) >= target, where W sums the
// elements' weights (weight(key) of each) and target = target_of(W(all members)), which
// must not exceed W(all members); the target comes back in *target_out, and for a target
// of 0 nothing else is computed (v is then meaningless).  Member
// keys have their top bit clear; every other element holds the all-ones key, which the
// tests below exclude, so no per-element flags are needed.  The
// bits above the highest one where the flagged keys differ are common to all of them,
// hence to v; below them v is found RADIX_BITS at a time from a histogram of weights per
// digit (LDS atomics) and a suffix scan over the digits.  The first round reads the keys
// in registers; the keys that share the digits found so far are then packed into an LDS
// list (when they fit) and the remaining rounds read only that list.  Returns v and, in
// *above, W(key > v).
template <int EPT, typename K, typename WF, typename TF, int NT>
__device__ __forceinline__ K radix_threshold(const K* key, TF target_of, WF weight, K kmin, K kmax,
                                             BgLds<NT>& sh, unsigned long long* target_out,
                                             unsigned long long* above_out) {
  constexpr int CAP = BG_LIST_BYTES / (int)sizeof(K);
  const int tid = threadIdx.x;
  K* list = reinterpret_cast<K*>(sh.list);
  *above_out = 0;
  if (kmin == kmax) {
    // one key value: the total is the members' count times its weight
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < EPT; ++i) cnt += (key[i] == kmin) ? 1 : 0;
    cnt = block_sum_int<NT>(cnt, sh.redi);
    *target_out = target_of((unsigned long long)cnt * weight(kmin));
    return kmin;
  }
  unsigned long long target = 0;
  int pos = highest_bit<K>(kmin ^ kmax) + 1;
  K prefix = kmin & ~low_mask<K>(pos);
  unsigned long long above = 0;
  int n_list = -1;                   // < 0: keys still read from registers
  {
    // First round, outside the loop (inside it the compiler would keep the EPT weights,
    // which no later round changes, in registers of their own).  Every member shares the
    // prefix, so the only test is against the all-ones key of non-members, and a
    // member's digit is its key minus the prefix, shifted.  (Sending non-members to a
    // spare bin instead would serialise their atomics on one address.)
    const int nb = min(RADIX_BITS, pos), lo = pos - nb;
    clear_hist(sh);
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const K k = key[i];
      if (k != ~K(0)) atomicAdd(&sh.hist[(uint32_t)((k - prefix) >> lo)], weight(k));
    }
    __syncthreads();
    uint32_t d;
    pick_digit(sh, true, target_of, &target, above, &d, &above);
    if (target == 0) {
      *target_out = 0;
      *above_out = 0;
      return prefix;
    }
    prefix |= (K)d << lo;
    pos = lo;
    if (pos > 0) n_list = stage_list<EPT>(key, pos, prefix, sh);
  }
  while (pos > 0) {
    const int nb = min(RADIX_BITS, pos), lo = pos - nb;
    const K hi_mask = ~low_mask<K>(pos);
    const uint32_t dmask = (1u << nb) - 1u;
    clear_hist(sh);
    if (n_list < 0) {
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        // (an opaque key keeps the compiler from hoisting the EPT weights, which do not
        // change between rounds, into registers of their own: they would spill)
        const K k = opaque(key[i]);
        if ((k & hi_mask) == prefix)
          atomicAdd(&sh.hist[(uint32_t)(k >> lo) & dmask], weight(k));
      }
    } else {
      for (int j = tid; j < n_list; j += NT) {
        const K k = list[j];
        if ((k & hi_mask) == prefix) atomicAdd(&sh.hist[(uint32_t)(k >> lo) & dmask], weight(k));
      }
    }
    __syncthreads();
    uint32_t d;
    pick_digit(sh, false, target_of, &target, above, &d, &above);
    prefix |= (K)d << lo;
    pos = lo;
    if (pos > 0 && n_list < 0) n_list = stage_list<EPT>(key, pos, prefix, sh);
  }
  *target_out = target;
  *above_out = above;
  return prefix;
}

// Among the elements flagged in `tie`, select the `take` with the largest slot index
// (slot = tid + NT * i: later elements, then later waves, then higher lanes).
template <int NT, int EPT>
__device__ __forceinline__ uint64_t take_top_ties_bg(uint64_t tie, int take, int* cnt) {
  constexpr int BG_NW = NT / 64;
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

// Candidate flags of the thread's elements.  The head's page masks are staged in LDS by
// coalesced loads first: per-element global loads would each hold an address pair and a
// value in registers while in flight, and inside per-element branches they would be
// waited on one by one.
template <int EPT, int NT>
__device__ __forceinline__ uint64_t cand_flags(int h, int S_max, const int32_t* __restrict__ cand_len,
                                               const uint16_t* __restrict__ mask, BgLds<NT>& sh) {
  const int cl = min(cand_len[h], S_max);
  const int np = S_max / HK_PAGE;
  if (mask) {
    const uint16_t* mrow = mask + (size_t)h * np;
    for (int q = threadIdx.x; q < np; q += NT) sh.mrow[q] = mrow[q];
  }
  __syncthreads();
  uint64_t f = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = threadIdx.x + NT * i;
    const bool ok = j < cl && (!mask || (((uint32_t)sh.mrow[j >> 4] >> (j & 15)) & 1u));
    f |= ok ? 1ull << i : 0ull;
  }
  return f;
}

// One bitmap row from per-element selection flags.
template <int NT, int EPT>
__device__ __forceinline__ void write_bitmap(uint64_t sel, uint32_t* __restrict__ brow, int S_max) {
  // addresses and bounds computed afresh on each call: hoisted out of a row loop they would
  // hold registers per element for the whole loop
  const int lane = threadIdx.x & 63, wave = opaque((int)(threadIdx.x >> 6));
  S_max = opaque(S_max);
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const unsigned long long b = __ballot((sel >> i) & 1ull);
    const int j0 = NT * i + 64 * wave;
    if (lane == 0 && j0 < S_max) {
      brow[j0 / 32] = (uint32_t)b;
      if (j0 + 32 < S_max) brow[j0 / 32 + 1] = (uint32_t)(b >> 32);
    }
  }
}

// ------------------------------------------------------------------ Cautious Update votes
// The head's page masks staged in LDS with every slot at or past cand_len cleared, for
// all NT * EPT slots a workgroup covers (pages past S_max hold no candidates).
template <int EPT, int NT>
__device__ __forceinline__ void stage_cand_masks(int h, int S_max, const int32_t* __restrict__ cand_len,
                                                 const uint16_t* __restrict__ mask, BgLds<NT>& sh) {
  const int cl = min(cand_len[h], S_max);
  const int np = S_max / HK_PAGE;
  const uint16_t* mrow = mask ? mask + (size_t)h * np : nullptr;
  for (int q = threadIdx.x; q < EPT * NT / HK_PAGE; q += NT) {
    const int keep = min(max(cl - q * HK_PAGE, 0), HK_PAGE);
    uint32_t m = (q < np && mrow) ? (uint32_t)mrow[q] : 0xffffu;
    sh.mrow[q] = (uint16_t)(m & ((1u << keep) - 1u));
  }
  __syncthreads();
}

// All ones when slot tid + NT * i is a candidate, else zero (masks staged as above).
template <int NT>
__device__ __forceinline__ uint32_t cand_lanes(const BgLds<NT>& sh, int i) {
  const int tid = threadIdx.x;
  const uint32_t m = sh.mrow[(tid >> 4) + (NT / HK_PAGE) * i];
  return (uint32_t)((int32_t)(m << (31 - (tid & 15))) >> 31);
}

// v_writelane through its compiler intrinsic (which also keeps the wait states a
// writelane needs after a VALU write of the scalar it reads, e.g. a ballot in vcc)
extern "C" __device__ int hk_intrinsic_writelane(int value, int lane, int old)
    __asm("llvm.amdgcn.writelane.i32");

// Lane LANE of x takes the wave-uniform value s; the other lanes keep theirs.
template <int LANE>
__device__ __forceinline__ void write_lane(uint32_t& x, uint32_t s) {
  x = (uint32_t)hk_intrinsic_writelane((int)s, LANE, (int)x);
}

template <int I>
struct IntC {
  static constexpr int value = I;
};
// f(IntC<I>) for I = B .. E-1, unrolled at compile time
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(IntC<B>{});
    static_for<B + 1, E>(f);
  }
}

// Four waves per SIMD (two workgroups per CU) cap the registers at 128: the allocator
// then keeps fewer loads in flight rather than lowering the occupancy.
template <int NT, int EPT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4, 8))) void vote_topp_kernel(
    int R, int S_max, const int32_t* __restrict__ cand_len,
    const uint16_t* __restrict__ mask, const float* __restrict__ a_rows, int p_q,
    uint32_t* __restrict__ row_sel, int32_t* __restrict__ row_k, int32_t* __restrict__ status) {
  constexpr int BG_NW = NT / 64;
  __shared__ BgLds<NT> sh;
  constexpr uint32_t NONE = 0xffffffffu;  // key of a non-candidate
  constexpr uint32_t ONE = 0x3f800000u;   // bits of 1.0f: in-range probabilities are <= ONE
  const int h = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  // one row per workgroup: a loop over rows would let the compiler keep per-element
  // addresses, masks and constants in registers across rows
  const int r = blockIdx.x;
  stage_cand_masks<EPT>(h, S_max, cand_len, mask, sh);
  // buffer loads: slots past the row's end read as 0 (they are no candidates), so no
  // clamped addresses are needed
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a_rows + ((size_t)h * R + r) * S_max), (short)0, S_max * 4, 0x00020000);
  uint32_t key[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    key[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, (tid + NT * i) * 4, 0, 0);
  // a candidate keeps its bits, anything else takes the all-ones key; for non-negative
  // floats the bit order is the value order
  uint32_t kmin = NONE, kmax = 0u;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const uint32_t m = cand_lanes(sh, i);
    const uint32_t b = key[i] & m;
    key[i] = b | ~m;
    kmin = min(kmin, key[i]);
    kmax = max(kmax, b);
  }
  block_key_range<uint32_t>(kmin, kmax, sh, &kmin, &kmax);
  if (kmax > ONE) {
    // some candidate is NaN, negative (-0 included) or above 1: clean every candidate
    // (NaN -> 0, clamp to [0, 1], +0) and report what was found
    int flags = 0;
    kmin = NONE;
    kmax = 0u;
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      uint32_t k = NONE;
      if (cand_lanes(sh, i)) {
        float v = __uint_as_float(key[i]);    // a candidate's key holds its bits
        if (v != v) { v = 0.f; flags |= HK_FLAG_NAN; }
        if (v > 1.f) { v = 1.f; flags |= HK_FLAG_RANGE; }
        if (v < 0.f) { v = 0.f; flags |= HK_FLAG_RANGE; }
        if (v == 0.f) v = 0.f;                  // canonical +0
        k = __float_as_uint(v);
        kmin = min(kmin, k);
        kmax = max(kmax, k);
      }
      key[i] = k;
    }
    block_key_range<uint32_t>(kmin, kmax, sh, &kmin, &kmax);
    const int any_nan = __syncthreads_or(flags & HK_FLAG_NAN);
    const int any_range = __syncthreads_or(flags & HK_FLAG_RANGE);
    if (status && tid == 0 && (any_nan || any_range))
      atomicOr(status, (any_nan ? HK_FLAG_NAN : 0) | (any_range ? HK_FLAG_RANGE : 0));
  }
  const unsigned long long pq = (unsigned long long)p_q;
  // target = ceil(p_q * Total / 10^6) without overflow
  const auto target_of = [pq](unsigned long long tot) {
    return pq * (tot / 1000000ull) + (pq * (tot % 1000000ull) + 999999ull) / 1000000ull;
  };
  uint32_t v = NONE;
  int take = 0;
  if (kmin != NONE) {
    unsigned long long target = 0, mass_gt = 0;
    v = radix_threshold<EPT, uint32_t>(key, target_of, [](uint32_t k) { return mass_weight(k); },
                                       kmin, kmax, sh, &target, &mass_gt);
    if (target > 0) {
      const unsigned long long wv = mass_weight(v);       // > 0: the crossing element weighs
      take = (int)((target - mass_gt + wv - 1) / wv);
    } else {
      // no mass to reach: k_min = 1 keeps the largest value, the most recent on ties
      v = kmax;
      take = 1;
    }
  }
  v = (uint32_t)__builtin_amdgcn_readfirstlane((int)v);     // uniform: from LDS
  take = __builtin_amdgcn_readfirstlane(take);
  // The row's bitmap straight from ballots: lane i of a wave keeps the wave's ballot of
  // its element i (64 consecutive slots from NT * i + 64 * wave, two bitmap words) for
  // the keys at or above the threshold; the wave's counts stay scalar.
  uint32_t ge_lo = 0, ge_hi = 0;
  int n_ge = 0, n_eq = 0;
  if (v != NONE) {
    static_for<0, EPT>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      const uint32_t kk = opaque(key[i]);
      const uint64_t bge = __ballot(kk - v < NONE - v);   // v <= kk < NONE
      const uint64_t beq = __ballot(kk == v);
      n_ge += __popcll(bge);
      n_eq += __popcll(beq);
      write_lane<i>(ge_lo, (uint32_t)bge);
      write_lane<i>(ge_hi, (uint32_t)(bge >> 32));
    });
  }
  __syncthreads();
  if (lane == 0) {
    sh.redi[wave] = n_ge;
    sh.tiecnt[wave] = n_eq;
  }
  __syncthreads();
  int n_tie = 0, n_above = 0;
#pragma unroll
  for (int w = 0; w < BG_NW; ++w) {
    n_above += sh.redi[w];
    n_tie += sh.tiecnt[w];
  }
  n_above -= n_tie;
  const int k = n_above + min(take, n_tie);
  if (take < n_tie) {
    // only `take` (possibly 0) of the keys equal to v are kept: those at the largest slots.  The ballots
    // are taken again: lane i of each wave keeps those of its element i, counts them in
    // LDS, and a suffix sum in slot order (element, then wave) says how many lie above.
    uint32_t eq_lo = 0, eq_hi = 0;
    static_for<0, EPT>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      const uint64_t beq = __ballot(opaque(key[i]) == v);
      write_lane<i>(eq_lo, (uint32_t)beq);
      write_lane<i>(eq_hi, (uint32_t)(beq >> 32));
    });
    __syncthreads();
    sh.tiecnt[lane * BG_NW + wave] = __popc(eq_lo) + __popc(eq_hi);
    __syncthreads();
    const int e = NT - 1 - tid;        // entries in descending slot order
    const int2 sc = block_exscan_bg<NT>(sh.tiecnt[e], sh.redi);
    int* above = reinterpret_cast<int*>(sh.list);
    above[e] = sc.x;
    __syncthreads();
    uint64_t eq = ((uint64_t)eq_hi << 32) | eq_lo;
    const int cnt = __popcll(eq);
    const int need = max(0, min(take - above[lane * BG_NW + wave], cnt));
    for (int d = cnt - need; d > 0; --d) eq &= eq - 1;   // drop the lowest slots
    const uint64_t ge = ((uint64_t)ge_hi << 32) | ge_lo;
    const uint64_t eqall = ((uint64_t)eq_hi << 32) | eq_lo;
    const uint64_t sel = (ge & ~eqall) | eq;
    ge_lo = (uint32_t)sel;
    ge_hi = (uint32_t)(sel >> 32);
  }
  uint32_t* brow = row_sel + ((size_t)h * R + r) * (S_max / 32);
  const int j0 = NT * lane + 64 * wave;
  if (lane < EPT && j0 < S_max) {
    brow[j0 / 32] = ge_lo;
    if (j0 + 32 < S_max) brow[j0 / 32 + 1] = ge_hi;
  }
  if (row_k && tid == 0) row_k[(size_t)h * R + r] = k;
}

// votes[h][j] = sum over the R rows of bit j of row_sel[h][r]; one thread per 32-slot word.
// The 32 column counts are kept bit-sliced (plane p holds bit p of every count) and the
// rows are added 16 at a time by a carry-save adder tree (Harley-Seal): two bitwise
// operations per row word instead of 32 shifts and adds.  ones, twos, fours and eights
// carry the low count bits across chunks; each chunk's carry out (sixteens) enters a
// ripple counter of multiples of 16 (R <= 256: at most 16 of them, 5 planes).
constexpr int VC_NT = 256;
constexpr int VC_HI = 5;

// full adder on 32 bit positions at once: l = a ^ b ^ c, h = majority(a, b, c)
__device__ __forceinline__ void vc_csa(uint32_t& h, uint32_t& l, uint32_t a, uint32_t b, uint32_t c) {
  const uint32_t u = a ^ b;
  h = (a & b) | (u & c);
  l = u ^ c;
}

__global__ __launch_bounds__(VC_NT) void vote_count_kernel(int R, int S_max,
                                                           const uint32_t* __restrict__ row_sel,
                                                           uint16_t* __restrict__ votes) {
  const int h = blockIdx.y;
  const int nw = S_max / 32;
  const int w = blockIdx.x * VC_NT + threadIdx.x;
  if (w >= nw) return;
  const uint32_t* base = row_sel + (size_t)h * R * nw + w;
  uint32_t ones = 0, twos = 0, fours = 0, eights = 0;
  uint32_t hi[VC_HI];
#pragma unroll
  for (int p = 0; p < VC_HI; ++p) hi[p] = 0;
  for (int r0 = 0; r0 < R; r0 += 16) {
    // all 16 loads first (rows past R read row R-1 and count as zero words)
    uint32_t x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = base[(size_t)min(r0 + i, R - 1) * nw];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = (r0 + i < R) ? x[i] : 0u;
    uint32_t twosA, twosB, foursA, foursB, eightsA, eightsB, sixteens;
    vc_csa(twosA, ones, ones, x[0], x[1]);
    vc_csa(twosB, ones, ones, x[2], x[3]);
    vc_csa(foursA, twos, twos, twosA, twosB);
    vc_csa(twosA, ones, ones, x[4], x[5]);
    vc_csa(twosB, ones, ones, x[6], x[7]);
    vc_csa(foursB, twos, twos, twosA, twosB);
    vc_csa(eightsA, fours, fours, foursA, foursB);
    vc_csa(twosA, ones, ones, x[8], x[9]);
    vc_csa(twosB, ones, ones, x[10], x[11]);
    vc_csa(foursA, twos, twos, twosA, twosB);
    vc_csa(twosA, ones, ones, x[12], x[13]);
    vc_csa(twosB, ones, ones, x[14], x[15]);
    vc_csa(foursB, twos, twos, twosA, twosB);
    vc_csa(eightsB, fours, fours, foursA, foursB);
    vc_csa(sixteens, eights, eights, eightsA, eightsB);
    uint32_t c = sixteens;
#pragma unroll
    for (int p = 0; p < VC_HI; ++p) {
      const uint32_t t = hi[p] & c;
      hi[p] ^= c;
      c = t;
    }
  }
  // count of bit b = ones_b + 2 twos_b + 4 fours_b + 8 eights_b + 16 (hi counter)_b
  uint32_t cnt[32];
#pragma unroll
  for (int b = 0; b < 32; ++b) {
    uint32_t n = ((ones >> b) & 1u) | (((twos >> b) & 1u) << 1) | (((fours >> b) & 1u) << 2) |
                 (((eights >> b) & 1u) << 3);
#pragma unroll
    for (int p = 0; p < VC_HI; ++p) n |= ((hi[p] >> b) & 1u) << (4 + p);
    cnt[b] = n;
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
template <int NT, int EPT>
__global__ __launch_bounds__(NT) void budget_select_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const uint16_t* __restrict__ votes, const float* __restrict__ c, const uint32_t* __restrict__ sel_in,
    const int32_t* __restrict__ head_mode, const int32_t* __restrict__ k_cap, int n_sink,
    uint32_t* __restrict__ sel_out, int32_t* __restrict__ k_out) {
  __shared__ BgLds<NT> sh;
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint64_t cf = cand_flags<EPT>(h, S_max, cand_len, mask, sh);
  const int mode = head_mode ? head_mode[h] : HK_BUDGET_REWRITE;
  uint32_t* brow = sel_out + (size_t)h * (S_max / 32);
  if (mode == HK_BUDGET_KEEP) {
    write_bitmap<NT, EPT>(cf, brow, S_max);
    const int n = block_sum_int<NT>(__popcll(cf), sh.redi);
    if (tid == 0) k_out[h] = n;
    return;
  }
  const uint16_t* vrow = votes ? votes + (size_t)h * S_max : nullptr;
  const float* crow = c ? c + (size_t)h * S_max : nullptr;
  const uint32_t* srow = sel_in ? sel_in + (size_t)h * (S_max / 32) : nullptr;
  uint64_t sinks = 0, base = 0;
  uint64_t key[EPT];                 // rank keys of the base set, all ones elsewhere
  uint64_t kmin = ~0ull, kmax = 0ull;
  // (per-element loads: a head's selection is one launch of n_heads workgroups, and
  // loading all elements up front would not fit beside the 64-bit keys)
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = tid + NT * i;
    key[i] = ~0ull;
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
  const int n_sinks = block_sum_int<NT>(__popcll(sinks), sh.redi);
  const int n_base = block_sum_int<NT>(__popcll(base), sh.redi);
  const int kc = k_cap ? k_cap[h] : -1;
  const int cap = kc < 0 ? n_base : min(n_base, max(0, kc - n_sinks));
  uint64_t sel = sinks;
  if (cap >= n_base) {
    sel |= base;
  } else if (cap > 0) {
    block_key_range<uint64_t>(kmin, kmax, sh, &kmin, &kmax);
    unsigned long long cnt_gt = 0, tgt = 0;
    const unsigned long long capu = (unsigned long long)cap;
    const uint64_t v = radix_threshold<EPT, uint64_t>(
        key, [capu](unsigned long long) { return capu; }, [](uint64_t) { return 1ull; }, kmin, kmax, sh,
        &tgt, &cnt_gt);
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
    const int n_tie = block_sum_int<NT>(__popcll(tie), sh.redi);
    if (take >= n_tie) sel |= tie;
    else if (take > 0) sel |= take_top_ties_bg<NT, EPT>(tie, take, sh.tiecnt);
  }
  write_bitmap<NT, EPT>(sel, brow, S_max);
  if (tid == 0) k_out[h] = n_sinks + cap;
}

// 512 threads and the fewest elements per thread that cover the row, or, past 512 * 64
// slots, 1024 threads with 64 elements each
template <template <int, int> class Launch, typename... A>
hipError_t by_ept(int S_max, A... args) {
  if (S_max > BG_SLOTS_512) return Launch<1024, 64>::run(args...);
  const int e = (S_max + 511) / 512;
  if (e <= 1) return Launch<512, 1>::run(args...);
  if (e <= 2) return Launch<512, 2>::run(args...);
  if (e <= 4) return Launch<512, 4>::run(args...);
  if (e <= 8) return Launch<512, 8>::run(args...);
  if (e <= 16) return Launch<512, 16>::run(args...);
  if (e <= 32) return Launch<512, 32>::run(args...);
  return Launch<512, 64>::run(args...);
}

template <int NT, int EPT>
struct VoteLaunch {
  static hipError_t run(int n_heads, int R, int S_max, const int32_t* cand_len, const uint16_t* mask,
                        const float* a_rows, int p_q, uint32_t* row_sel, int32_t* row_k,
                        int32_t* status, uint16_t* votes, hipStream_t st) {
    {
      TimedLaunch t(HK_TK_VOTE, st);
      hipLaunchKernelGGL((vote_topp_kernel<NT, EPT>), dim3(R, n_heads), dim3(NT), 0, st, R, S_max,
                         cand_len, mask, a_rows, p_q, row_sel, row_k, status);
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

template <int NT, int EPT>
struct BudgetSelectLaunch {
  static hipError_t run(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                        const uint16_t* votes, const float* c, const uint32_t* sel_in,
                        const int32_t* head_mode, const int32_t* k_cap, int n_sink, uint32_t* sel_out,
                        int32_t* k_out, hipStream_t st) {
    TimedLaunch t(HK_TK_BUDGET_SELECT, st);
    hipLaunchKernelGGL((budget_select_kernel<NT, EPT>), dim3(n_heads), dim3(NT), 0, st, S_max, cand_len,
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

// a2 / a2' / a3: Logits Calibration, temperature solve and head-adaptive Top-p (gfx950).
//
// One workgroup of 1024 threads per head.  Slot j of the head is owned by thread
// j % 1024 as its element j / 1024, so a wave's 64 lanes always cover 64 consecutive
// slots (coalesced loads, and one ballot gives two words of the selection bitmap).
// Every head's candidates stay in registers (S_max <= 32768 -> <= 32 per thread).
#include "hk_internal.h"

namespace hk {

constexpr int SEL_NT = 1024;
constexpr int SEL_NW = SEL_NT / 64;
constexpr unsigned long long kMassOne = 1ull << 40;   // fixed-point unit of the Top-p mass

// ------------------------------------------------------------------ a2: calibrate
// c = sum_m w_m Softmax(x_m / T_m) over the candidates (Solution 2, Sec. 3.2), for the
// thread's EPT slots; the fused select kernel runs the same code, so both paths produce
// identical values.  Each metric's row, divided by its temperature, is first staged in LDS
// (`xs`, EPT * SEL_NT floats) by unconditional coalesced loads: the three sweeps (max,
// sum, values) then read LDS, where reads inside the per-candidate branches cost little,
// instead of global memory, where each one would be waited on in turn.
template <int EPT>
__device__ __forceinline__ void calib_values(int h, int S_max, uint32_t cbits, int n_metrics,
                                             const float* __restrict__ x0, const float* __restrict__ x1,
                                             const float* __restrict__ T0, const float* __restrict__ T1,
                                             float w0, float w1, float* __restrict__ lse_out, float* red,
                                             float* xs, float* c) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < EPT; ++i) c[i] = 0.f;
  for (int m = 0; m < n_metrics; ++m) {
    const float* x = (m == 0 ? x0 : x1) + (size_t)h * S_max;
    const float* Tp = (m == 0 ? T0 : T1);
    const float T = Tp ? Tp[h] : 1.0f;
    const float wm = (m == 0 ? w0 : w1);
    {
      // xs holds EPT * SEL_NT floats, so the stores need no bound; the loads clamp theirs.
      // (The opaque index keeps the compiler from computing the EPT addresses once for
      // all metrics and holding them.)
      int j0 = tid;
      asm volatile("" : "+v"(j0));
      float t[EPT];
#pragma unroll
      for (int i = 0; i < EPT; ++i) t[i] = x[min(j0 + SEL_NT * i, S_max - 1)];
      __syncthreads();                   // the previous metric's readers are done
#pragma unroll
      for (int i = 0; i < EPT; ++i) xs[j0 + SEL_NT * i] = t[i] / T;   // x / T, once
      __syncthreads();
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if ((cbits >> i) & 1u) mx = fmaxf(mx, xs[tid + SEL_NT * i]);
    mx = block_max<SEL_NT>(mx, red);
    float lse = -INFINITY;
    if (mx != -INFINITY) {
      float sm = 0.f;
#pragma unroll
      for (int i = 0; i < EPT; ++i)
        if ((cbits >> i) & 1u) sm += expf(xs[tid + SEL_NT * i] - mx);
      sm = block_sum<SEL_NT>(sm, red);
      lse = mx + logf(sm);
#pragma unroll
      for (int i = 0; i < EPT; ++i)
        if ((cbits >> i) & 1u) c[i] = fmaf(wm, expf(xs[tid + SEL_NT * i] - lse), c[i]);
    }
    if (lse_out && tid == 0) lse_out[(size_t)h * n_metrics + m] = lse;
  }
}

// Candidate bits of the thread's slots.  The head's page masks are first staged in LDS by
// coalesced loads: per-slot loads inside the candidate test would be waited on one by one.
template <int EPT>
__device__ __forceinline__ uint32_t cand_bits(int h, int S_max, const int32_t* __restrict__ cand_len,
                                              const uint16_t* __restrict__ mask) {
  __shared__ uint16_t mrow_lds[32768 / HK_PAGE];
  const int cl = min(cand_len[h], S_max);
  const int np = S_max / HK_PAGE;
  if (mask) {
    const uint16_t* mrow = mask + (size_t)h * np;
    for (int q = threadIdx.x; q < np; q += SEL_NT) mrow_lds[q] = mrow[q];
    __syncthreads();
  }
  uint32_t cbits = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = threadIdx.x + SEL_NT * i;
    const bool ok = j < cl && (!mask || (((uint32_t)mrow_lds[j >> 4] >> (j & 15)) & 1u));
    cbits |= ok ? 1u << i : 0u;
  }
  return cbits;
}

template <int EPT>
__global__ __launch_bounds__(SEL_NT) void calibrate_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask, int n_metrics,
    const float* __restrict__ x0, const float* __restrict__ x1, const float* __restrict__ T0,
    const float* __restrict__ T1, float w0, float w1, float* __restrict__ c_out,
    float* __restrict__ lse_out) {
  extern __shared__ float xs_dyn[];     // EPT * SEL_NT floats: a metric's row
  __shared__ float red[SEL_NW];
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint32_t cbits = cand_bits<EPT>(h, S_max, cand_len, mask);
  float c[EPT];
  calib_values<EPT>(h, S_max, cbits, n_metrics, x0, x1, T0, T1, w0, w1, lse_out, red, xs_dyn, c);
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = tid + SEL_NT * i;
    if (j < S_max) c_out[(size_t)h * S_max + j] = c[i];
  }
}

// Fixed-point weight of a Top-p value v in [0, 1] given by its bits: floor(v * 2^40).
// The product is exact in fp32 (a power-of-two scale) and keeps at most 24 significant
// bits, so the truncated float is that integer exactly; a thread's sum of up to 32 of
// them stays below 2^46 and is exact in fp64.
__device__ __forceinline__ float fixed_weight(uint32_t key) {
  return truncf(__uint_as_float(key) * (float)kMassOne);
}

// Count of the thread's candidates with key >= t.
template <int EPT, typename K>
__device__ __forceinline__ int count_ge(const K& key, uint32_t cbits, uint32_t t) {
  int n = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) n += (((cbits >> i) & 1u) && key[i] >= t) ? 1 : 0;
  return n;
}

// Select, among elements with key == v (flags in `tie`), the `take` with the largest slot
// index.  Returns the per-element selection bits for the ties.
template <int EPT>
__device__ __forceinline__ uint32_t take_top_ties(uint32_t tie, int take, int* cnt /* LDS [EPT][SEL_NW] */) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const unsigned long long b = __ballot((tie >> i) & 1u);
    if (lane == 0) cnt[i * SEL_NW + wave] = __popcll(b);
  }
  __syncthreads();
  uint32_t out = 0;
  // ties with a larger slot index: later rows, later waves of this row, higher lanes (the
  // ballots are taken again rather than kept: EPT 64-bit registers would spill)
  int above_rows = 0;
#pragma unroll
  for (int i = EPT - 1; i >= 0; --i) {
    int above = above_rows;
    for (int w = wave + 1; w < SEL_NW; ++w) above += cnt[i * SEL_NW + w];
    const unsigned long long b = __ballot((tie >> i) & 1u);
    const unsigned long long hi = (lane == 63) ? 0ull : (b >> (lane + 1));
    above += __popcll(hi);
    if (((tie >> i) & 1u) && above < take) out |= 1u << i;
    int row = 0;
    for (int w = 0; w < SEL_NW; ++w) row += cnt[i * SEL_NW + w];
    above_rows += row;
  }
  return out;
}

// ------------------------------------------------------------------ a3: Top-p
// Exclusive prefix (thread order) of one int per thread (.x) and the block sum (.y).
__device__ __forceinline__ int2 block_exscan_int(int v, int* red) {
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
  for (int w = 0; w < SEL_NW; ++w) {
    if (w < wave) before += red[w];
    all += red[w];
  }
  return make_int2(before + x - v, all);
}

template <bool MAX>
__device__ __forceinline__ uint32_t block_minmax_u32(uint32_t v, int* red) {
  v = wave_reduce_u32(v, MAX ? 0u : 0xffffffffu,
                      [](uint32_t a, uint32_t b) { return MAX ? (a > b ? a : b) : (a < b ? a : b); });
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = (int)v;
  __syncthreads();
  uint32_t r = (uint32_t)red[0];
#pragma unroll
  for (int i = 1; i < SEL_NW; ++i) r = MAX ? max(r, (uint32_t)red[i]) : min(r, (uint32_t)red[i]);
  return r;
}
__device__ __forceinline__ uint32_t block_min_u32(uint32_t v, int* red) { return block_minmax_u32<false>(v, red); }
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, int* red) { return block_minmax_u32<true>(v, red); }

// Block-uniform values (results of block reductions) moved to scalar registers, so the
// 64-bit divisions of the mass rule run on the scalar unit.
__device__ __forceinline__ unsigned long long uniform_u64(unsigned long long x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((unsigned long long)hi << 32) | lo;
}

constexpr int SEL_RADIX_BITS = 11;
constexpr int SEL_BINS = 1 << SEL_RADIX_BITS;
constexpr int SEL_BPT = SEL_BINS / SEL_NT;        // digits per thread in the suffix scan

struct SelLds {
  unsigned long long red64[SEL_NW];
  int redi[SEL_NW];
  unsigned long long hist[SEL_BINS];
  unsigned long long pick_above;
  uint32_t pick_digit;
};



// Head-adaptive Top-p (Sec. 3.3) on the thread's EPT values: the smallest set whose
// fixed-point mass reaches ceil(p_q * Total / 10^6), ties at the threshold broken toward
// the larger slot index; the count is clamped to [k_min, k_max].
// Read-only view of a thread's values as ordering keys (their bit patterns).
template <int EPT>
struct KeyView {
  const float* v;
  __device__ __forceinline__ uint32_t operator[](int i) const { return __float_as_uint(v[i]); }
};

// A copy of x the compiler cannot see through: per-element tests of a fresh copy are not
// hoisted out of the search rounds and kept (as EPT lane masks) across them.
template <typename X>
__device__ __forceinline__ X sel_opaque(X x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Fixed-point weight floor(v * 2^40) of a value v in [0, 1] from its bits, as its two
// exact 32-bit halves: with t = v * 2^8 (exact, t <= 256) the high half is floor(t) and
// the low half floor(fract(t) * 2^32).
__device__ __forceinline__ unsigned long long weight_u64(uint32_t key) {
  const float t = __uint_as_float(key) * 256.0f;
  const uint32_t hi = (uint32_t)t;
  const uint32_t lo = (uint32_t)(__builtin_amdgcn_fractf(t) * 4294967296.0f);
  return ((unsigned long long)hi << 32) | lo;
}

// After a histogram round: the digit where the weight from the top crosses the target,
// and the weight above it.  On the first round the target is target_of(the histogram's
// total, which is every candidate's weight); it comes back in *target (0: no digit).
template <typename TF>
__device__ __forceinline__ void sel_pick_digit(SelLds& sh, bool first, TF target_of,
                                               unsigned long long* target_io,
                                               unsigned long long above, uint32_t* d_out,
                                               unsigned long long* above_out) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  unsigned long long own = 0;
#pragma unroll
  for (int b = 0; b < SEL_BPT; ++b) own += sh.hist[tid * SEL_BPT + b];
  unsigned long long x = own;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long y = __shfl_down(x, o, 64);
    if (lane + o < 64) x += y;
  }
  if (lane == 0) sh.red64[wave] = x;
  __syncthreads();
  unsigned long long suf = x - own;
  for (int w = wave + 1; w < SEL_NW; ++w) suf += sh.red64[w];
  if (first) {
    unsigned long long tot = 0;
#pragma unroll
    for (int w = 0; w < SEL_NW; ++w) tot += sh.red64[w];
    *target_io = target_of(tot);
  }
  const unsigned long long target = *target_io;
  if (target == 0) return;
  const unsigned long long lo_m = above + suf;
  if (lo_m < target && lo_m + own >= target) {
    unsigned long long cum = lo_m;
    for (int b = SEL_BPT - 1; b >= 0; --b) {
      const unsigned long long nxt = cum + sh.hist[tid * SEL_BPT + b];
      if (nxt >= target) {
        sh.pick_digit = (uint32_t)(tid * SEL_BPT + b);
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

__device__ __forceinline__ uint32_t sel_block_sum_u32(uint32_t v, int* red) {
  v = wave_reduce_u32(v, 0u, [](uint32_t a, uint32_t b) { return a + b; });
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = (int)v;
  __syncthreads();
  uint32_t r = 0;
#pragma unroll
  for (int w = 0; w < SEL_NW; ++w) r += (uint32_t)red[w];
  return r;
}

// Zero the histogram between two barriers.
__device__ __forceinline__ void sel_clear_hist(SelLds& sh) {
  __syncthreads();                   // earlier readers of the LDS scratch are done
#pragma unroll
  for (int b = 0; b < SEL_BPT; ++b) sh.hist[threadIdx.x * SEL_BPT + b] = 0ull;
  __syncthreads();
}

// Stage the candidates whose bits from `pos` up equal `prefix` into the list (it holds
// every slot); returns their number.
template <int EPT>
__device__ __forceinline__ int sel_stage_list(const KeyView<EPT>& key, uint32_t cbits, int pos,
                                              uint32_t prefix, uint32_t* list, SelLds& sh) {
  const uint32_t m2 = ~((1u << pos) - 1u);
  const uint32_t cb = sel_opaque(cbits);
  uint32_t inb = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    if (((cb >> i) & 1u) && (sel_opaque(key[i]) & m2) == prefix) inb |= 1u << i;
  const int2 sc = block_exscan_int(__popc(inb), sh.redi);
  int off = sc.x;
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    if ((inb >> i) & 1u) list[off++] = key[i];
  return sc.y;
}

// Largest candidate key v with W(key >= v) >= target, where W sums weight(key) over the
// candidates and target = target_of(W(all candidates)) (at most that total); the target
// comes back in *target_out, and for a target of 0 nothing else is computed.  The bits
// above the first one where the candidates' keys differ are common to all of them; below
// them v is found SEL_RADIX_BITS at a time from a histogram of weights per digit (LDS
// atomics) and a suffix scan over the digits.  The first round reads the keys in
// registers (outside the loop, so the compiler does not keep the EPT weights, which no
// later round changes, in registers of their own); the candidates that share the
// digits found are then packed into the LDS list, which the remaining rounds read.
// Returns v and, in *above, W(key > v).
template <int EPT, typename WF, typename TF>
__device__ __forceinline__ uint32_t sel_radix_threshold(const KeyView<EPT>& key, uint32_t cbits,
                                                        TF target_of, WF weight, uint32_t kmin,
                                                        uint32_t kmax, uint32_t* list, SelLds& sh,
                                                        unsigned long long* target_out,
                                                        unsigned long long* above_out) {
  const int tid = threadIdx.x;
  *above_out = 0;
  if (kmin == kmax) {
    // one key value: the total is the candidates' count times its weight
    const int cnt = block_sum_int<SEL_NT>(__popc(cbits), sh.redi);
    *target_out = target_of((unsigned long long)cnt * weight(kmin));
    return kmin;
  }
  int pos = 32 - __clz((int)(kmin ^ kmax));
  uint32_t prefix = pos >= 32 ? 0u : (kmin & ~((1u << pos) - 1u));
  unsigned long long above = 0, target = 0;
  int n_list;
  {
    // every candidate shares the prefix: its digit is its key minus the prefix, shifted
    const int nb = min(SEL_RADIX_BITS, pos), lo = pos - nb;
    sel_clear_hist(sh);
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if ((cbits >> i) & 1u) atomicAdd(&sh.hist[(key[i] - prefix) >> lo], weight(key[i]));
    __syncthreads();
    uint32_t d;
    sel_pick_digit(sh, true, target_of, &target, above, &d, &above);
    if (target == 0) {
      *target_out = 0;
      return prefix;
    }
    prefix |= d << lo;
    pos = lo;
    n_list = pos > 0 ? sel_stage_list<EPT>(key, cbits, pos, prefix, list, sh) : 0;
  }
  while (pos > 0) {
    const int nb = min(SEL_RADIX_BITS, pos), lo = pos - nb;
    const uint32_t hi_mask = ~((1u << pos) - 1u);
    const uint32_t dmask = (1u << nb) - 1u;
    sel_clear_hist(sh);
    for (int j = tid; j < n_list; j += SEL_NT) {
      const uint32_t k = list[j];
      if ((k & hi_mask) == prefix) atomicAdd(&sh.hist[(k >> lo) & dmask], weight(k));
    }
    __syncthreads();
    uint32_t d;
    sel_pick_digit(sh, false, target_of, &target, above, &d, &above);
    prefix |= d << lo;
    pos = lo;
  }
  *target_out = target;
  *above_out = above;
  return prefix;
}

// `val` holds the thread's EPT values; they are clamped in place, and their bit patterns
// (non-negative floats order as integers) are the ordering keys.
template <int EPT>
__device__ __forceinline__ void topp_core(float* val, uint32_t cbits, int p_q, int k_min, int k_max,
                          uint32_t* __restrict__ brow, int S_max, int32_t* __restrict__ k_out,
                          float* __restrict__ sel_mass, int32_t* __restrict__ status, int h,
                          uint32_t* list, SelLds& sh, int* tiecnt) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int flags = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    float v = val[i];
    if ((cbits >> i) & 1u) {
      if (v != v) { v = 0.f; flags |= HK_FLAG_NAN; }
      if (v > 1.f) { v = 1.f; flags |= HK_FLAG_RANGE; }
      if (v < 0.f) { v = 0.f; flags |= HK_FLAG_RANGE; }
      if (v == 0.f) v = 0.f;                      // canonical +0
    } else {
      v = 0.f;
    }
    val[i] = v;
  }
  const KeyView<EPT> key{val};
  // __syncthreads_or returns a predicate, so each flag bit is reduced on its own
  const int any_nan = __syncthreads_or(flags & HK_FLAG_NAN);
  const int any_range = __syncthreads_or(flags & HK_FLAG_RANGE);
  flags = (any_nan ? HK_FLAG_NAN : 0) | (any_range ? HK_FLAG_RANGE : 0);
  if (tid == 0 && flags && status) atomicOr(status, flags);

  const int n_cand = block_sum_int<SEL_NT>(__popc(cbits), sh.redi);
  const unsigned long long pq = (unsigned long long)p_q;
  // target = ceil(p_q * Total / 10^6) without overflow (Total from the first search round)
  const auto target_of = [pq](unsigned long long tot) {
    return pq * (tot / 1000000ull) + (pq * (tot % 1000000ull) + 999999ull) / 1000000ull;
  };

  // the bits above the first one where the candidates' keys differ are common to all of
  // them: the searches start below them
  uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    if ((cbits >> i) & 1u) {
      kmin = min(kmin, key[i]);
      kmax = max(kmax, key[i]);
    }
  kmin = block_min_u32(kmin, sh.redi);
  kmax = block_max_u32(kmax, sh.redi);

  // mass rule: v = value of the crossing element, the elements above it all taken, and
  // `take` of those equal to it
  uint32_t v = 0xffffffffu;
  int take = 0;
  unsigned long long target = 0, mass_gt = 0, wv = 0;
  if (n_cand > 0) {
    v = sel_radix_threshold<EPT>(key, cbits, target_of, [](uint32_t kk) { return weight_u64(kk); },
                                 kmin, kmax, list, sh, &target, &mass_gt);
    v = __builtin_amdgcn_readfirstlane(v);
    target = uniform_u64(target);
    mass_gt = uniform_u64(mass_gt);
    if (target > 0) {
      wv = uniform_u64(weight_u64(v));             // > 0: the crossing element weighs
      take = (int)((target - mass_gt + wv - 1) / wv);
    } else {
      v = 0xffffffffu;
    }
  }
  // selection flags: keys above v and keys equal to it; both counts in one reduction
  uint32_t sel = 0, tie = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    if ((cbits >> i) & 1u) {
      if (v != 0xffffffffu && key[i] > v) sel |= 1u << i;
      if (key[i] == v) tie |= 1u << i;
    }
  }
  // (each count is at most 32768, so the packed sum fits 32 unsigned bits)
  const uint32_t both = sel_block_sum_u32((uint32_t)__popc(sel) | ((uint32_t)__popc(tie) << 16), sh.redi);
  const int n_gt = (int)(both & 0xffffu);
  int n_tie = (int)(both >> 16);
  const int k = target > 0 ? n_gt + take : 0;
  const int lo = min(max(k_min, 0), n_cand);
  const int hi = (k_max > 0) ? min(k_max, n_cand) : n_cand;
  const int kf = max(lo, min(k, hi));
  const bool by_mass = kf == k && target > 0;
  if (!by_mass) {
    if (kf == 0) {
      v = 0xffffffffu;
      take = 0;
      sel = 0;
      tie = 0;
      n_tie = 0;
    } else {
      // the kf largest keys: the same search on counts
      unsigned long long t_cnt = 0, cnt_gt = 0;
      v = sel_radix_threshold<EPT>(key, cbits, [kf](unsigned long long) { return (unsigned long long)kf; },
                                   [](uint32_t) { return 1ull; }, kmin, kmax, list, sh, &t_cnt, &cnt_gt);
      v = __builtin_amdgcn_readfirstlane(v);
      take = kf - (int)uniform_u64(cnt_gt);
      sel = 0;
      tie = 0;
#pragma unroll
      for (int i = 0; i < EPT; ++i) {
        if ((cbits >> i) & 1u) {
          if (key[i] > v) sel |= 1u << i;
          if (key[i] == v) tie |= 1u << i;
        }
      }
      n_tie = block_sum_int<SEL_NT>(__popc(tie), sh.redi);
    }
  }
  // keys above v, plus the `take` most recent slots equal to v
  if (take >= n_tie) sel |= tie;
  else if (take > 0) sel |= take_top_ties<EPT>(tie, take, tiecnt);

  // the selected mass: by the mass rule it is W(key > v) + take * w(v) exactly; after a
  // count clamp it is summed
  unsigned long long msel;
  if (by_mass) {
    msel = mass_gt + (unsigned long long)take * wv;
  } else {
    double msel_d = 0.0;
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if ((sel >> i) & 1u) msel_d += (double)fixed_weight(key[i]);
    msel = block_sum_u64<SEL_NT>((unsigned long long)msel_d, sh.red64);
  }

#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const unsigned long long b = __ballot((sel >> i) & 1u);
    const int j0 = SEL_NT * i + 64 * wave;
    if (lane == 0 && j0 < S_max) {
      brow[j0 / 32] = (uint32_t)b;
      if (j0 + 32 < S_max) brow[j0 / 32 + 1] = (uint32_t)(b >> 32);
    }
  }
  if (tid == 0) {
    k_out[h] = kf;
    if (sel_mass) sel_mass[h] = (float)((double)msel / (double)kMassOne);
  }
}

template <int EPT>
__global__ __launch_bounds__(SEL_NT) void topp_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const float* __restrict__ c, int p_q, int k_min, int k_max, uint32_t* __restrict__ sel_bits,
    int32_t* __restrict__ k_out, float* __restrict__ sel_mass, int32_t* __restrict__ status) {
  extern __shared__ uint32_t list[];
  __shared__ SelLds sh;
  __shared__ int tiecnt[EPT * SEL_NW];
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint32_t cbits = cand_bits<EPT>(h, S_max, cand_len, mask);
  const float* crow = c + (size_t)h * S_max;
  float val[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const float v = crow[min(tid + SEL_NT * i, S_max - 1)];   // unconditional: loads overlap
    val[i] = ((cbits >> i) & 1u) ? v : 0.f;
  }
  topp_core<EPT>(val, cbits, p_q, k_min, k_max, sel_bits + (size_t)h * (S_max / 32), S_max, k_out,
                 sel_mass, status, h, list, sh, tiecnt);
}

// a2 + a3 in one launch: calibrate, then Top-p on the calibrated values in registers
template <int EPT>
__global__ __launch_bounds__(SEL_NT) void calib_topp_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask, int n_metrics,
    const float* __restrict__ x0, const float* __restrict__ x1, const float* __restrict__ T0,
    const float* __restrict__ T1, float w0, float w1, int p_q, int k_min, int k_max,
    float* __restrict__ c_out, float* __restrict__ lse_out, uint32_t* __restrict__ sel_bits,
    int32_t* __restrict__ k_out, float* __restrict__ sel_mass, int32_t* __restrict__ status) {
  extern __shared__ uint32_t list[];
  __shared__ SelLds sh;
  __shared__ float red[SEL_NW];
  __shared__ int tiecnt[EPT * SEL_NW];
  const int h = blockIdx.x, tid = threadIdx.x;
  const uint32_t cbits = cand_bits<EPT>(h, S_max, cand_len, mask);
  float c[EPT];
  // the key list of the Top-p search is not live yet: it holds the metric rows meanwhile
  calib_values<EPT>(h, S_max, cbits, n_metrics, x0, x1, T0, T1, w0, w1, lse_out, red,
                    reinterpret_cast<float*>(list), c);
  if (c_out) {
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
      const int j = tid + SEL_NT * i;
      if (j < S_max) c_out[(size_t)h * S_max + j] = c[i];
    }
  }
  topp_core<EPT>(c, cbits, p_q, k_min, k_max, sel_bits + (size_t)h * (S_max / 32), S_max, k_out,
                 sel_mass, status, h, list, sh, tiecnt);
}

// ------------------------------------------------------------------ a2 pooling
// Order-preserving pooling before calibration (Solution 1, SnapKV form): candidate j gets
// the maximum candidate score within `radius` slots on either side.  One 256-thread
// workgroup per (head, 1024-slot tile); the tile and its halo are staged in LDS with
// non-candidates as -inf, so a window never picks one.
constexpr int POOL_NT = 256, POOL_TILE = 1024, POOL_RMAX = 64;

__global__ __launch_bounds__(POOL_NT) void pool_max_kernel(int S_max, const int32_t* __restrict__ cand_len,
                                                           const uint16_t* __restrict__ mask,
                                                           const float* __restrict__ x, int radius,
                                                           float* __restrict__ out) {
  __shared__ float tile[POOL_TILE + 2 * POOL_RMAX];
  const int h = blockIdx.y, j0 = blockIdx.x * POOL_TILE;
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  const float* xr = x + (size_t)h * S_max;
  for (int i = threadIdx.x; i < POOL_TILE + 2 * radius; i += POOL_NT) {
    const int j = j0 - radius + i;
    tile[i] = (j >= 0 && j < S_max && is_cand(mrow, cl, j)) ? xr[j] : -INFINITY;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < POOL_TILE; i += POOL_NT) {
    const int j = j0 + i;
    if (j >= S_max) break;
    float m = -INFINITY;
    if (is_cand(mrow, cl, j))
      for (int d = 0; d <= 2 * radius; ++d) m = fmaxf(m, tile[i + d]);
    out[(size_t)h * S_max + j] = m;
  }
}

// ------------------------------------------------------------------ a2': temperature
// Bisection on log T for M_k(Softmax(x/T)) = target (App. D.1; order invariance App. D.2).
__device__ __forceinline__ uint32_t ordered_key(float x) {
  uint32_t b = __float_as_uint(x);
  if (x != x) return 0u;                         // NaN below everything
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Top-k set of x among the candidates (keys = order-preserving bits of x): keys above the
// k-th largest plus, among the keys equal to it, the most recent slots.
template <int EPT>
__device__ __forceinline__ uint32_t topk_set(const uint32_t* key, uint32_t cbits, int kk, int* redi,
                                             int* tiecnt) {
  uint32_t top = 0;
  if (kk <= 0) return 0;
  uint32_t v = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t t = v | (1u << b);
    if (block_sum_int<SEL_NT>(count_ge<EPT>(key, cbits, t), redi) >= kk) v = t;
  }
  const int cnt_gt = (v == 0xffffffffu) ? 0 : block_sum_int<SEL_NT>(count_ge<EPT>(key, cbits, v + 1), redi);
  const int take = kk - cnt_gt;
  uint32_t tie = 0;
#pragma unroll
  for (int i = 0; i < EPT; ++i)
    if ((cbits >> i) & 1u) {
      if (v != 0xffffffffu && key[i] > v) top |= 1u << i;
      if (key[i] == v) tie |= 1u << i;
    }
  const int n_tie = block_sum_int<SEL_NT>(__popc(tie), redi);
  if (take >= n_tie) top |= tie;
  else if (take > 0) top |= take_top_ties<EPT>(tie, take, tiecnt);
  return top;
}

template <int EPT>
__global__ __launch_bounds__(SEL_NT) void solve_T_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const float* __restrict__ x, const int32_t* __restrict__ k_arr, const float* __restrict__ target,
    float T_lo, float T_hi, int iters, float* __restrict__ T_out) {
  __shared__ float red[SEL_NW];
  __shared__ int redi[SEL_NW];
  __shared__ int tiecnt[EPT * SEL_NW];
  const int h = blockIdx.x, tid = threadIdx.x;
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  const float* xrow = x + (size_t)h * S_max;
  uint32_t cbits = 0, key[EPT];
  float xv[EPT];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = tid + SEL_NT * i;
    key[i] = 0;
    xv[i] = -INFINITY;
    if (j < S_max && is_cand(mrow, cl, j)) {
      cbits |= 1u << i;
      xv[i] = xrow[j];
      key[i] = ordered_key(xv[i]);
      mx = fmaxf(mx, xv[i]);
    }
  }
  mx = block_max<SEL_NT>(mx, red);
  const int n_cand = block_sum_int<SEL_NT>(__popc(cbits), redi);
  const int kk = min(max(k_arr[h], 0), n_cand);
  const uint32_t top = topk_set<EPT>(key, cbits, kk, redi, tiecnt);
  const float tgt = target[h];
  float a = logf(T_lo), b = logf(T_hi);
  for (int it = 0; it < iters; ++it) {
    const float mid = 0.5f * (a + b);
    const float invT = expf(-mid);
    float s_all = 0.f, s_top = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int i = 0; i < EPT; ++i)
        if ((cbits >> i) & 1u) {
          const float e = expf((xv[i] - mx) * invT);
          s_all += e;
          if ((top >> i) & 1u) s_top += e;
        }
    }
    s_all = block_sum<SEL_NT>(s_all, red);
    s_top = block_sum<SEL_NT>(s_top, red);
    const float mass = (s_all > 0.f) ? s_top / s_all : 0.f;
    if (mass - tgt > 0.f) a = mid;
    else b = mid;
  }
  if (tid == 0) T_out[h] = expf(0.5f * (a + b));
}

// The same rule for rows longer than one workgroup holds in registers (S_max > 32768): the
// row is streamed from memory in every sweep.  The k-th largest key comes from an 8-bit
// radix search (four sweeps, each a 256-bin count histogram of the keys that share the
// digits found so far), the ties it leaves are cut by slot from per-thread counts over
// contiguous runs of slots (the most recent slots are taken), and each bisection step is one
// sweep of two block sums.  Only the summation order differs from solve_T_kernel.
__device__ __forceinline__ int wave_incl_scan_i(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

// Shared state of the streamed Top-k search.
struct LongTopK {
  uint32_t hist[256];
  uint32_t digit;
  int above, tie_from;
};

// The Top-k set of a streamed row as (v, tie_from): candidates with key > v, and those with
// key == v at slots >= tie_from (v = 0xffffffff and tie_from = S_max for kk = 0).  Every
// thread of the block calls it; `redi` holds one int per wave.
__device__ __forceinline__ void long_topk(int S_max, const uint16_t* mrow, int cl, const float* xrow,
                                          int kk, uint32_t& v, int& tie_from, LongTopK& sh, int* redi) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  v = 0xffffffffu;
  tie_from = S_max;
  if (kk <= 0) return;
  uint32_t prefix = 0;
  int above = 0, n_tie = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += SEL_NT) sh.hist[i] = 0u;
    __syncthreads();
    for (int j = tid; j < S_max; j += SEL_NT)
      if (is_cand(mrow, cl, j)) {
        const uint32_t key = ordered_key(xrow[j]);
        if (shift == 24 || (key >> (shift + 8)) == (prefix >> (shift + 8)))
          atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
      }
    __syncthreads();
    if (tid == 0) {
      int cum = above;
      uint32_t d = 0;
      for (int b = 255; b >= 0; --b) {
        if (cum + (int)sh.hist[b] >= kk) {
          d = (uint32_t)b;
          break;
        }
        cum += (int)sh.hist[b];
      }
      sh.digit = d;
      sh.above = cum;
    }
    __syncthreads();
    prefix |= sh.digit << shift;
    above = sh.above;
    n_tie = (int)sh.hist[sh.digit];
    __syncthreads();                   // every thread has read the histogram
  }
  v = prefix;
  const int take = kk - above;         // >= 1
  if (take >= n_tie) {
    tie_from = 0;
    return;
  }
  // ties in this thread's run of slots, then the runs above it (higher slots)
  const int P = (S_max + SEL_NT - 1) / SEL_NT, j0 = tid * P, j1 = min(j0 + P, S_max);
  int cnt = 0;
  for (int j = j0; j < j1; ++j)
    if (is_cand(mrow, cl, j) && ordered_key(xrow[j]) == v) ++cnt;
  const int incl = wave_incl_scan_i(cnt);
  __syncthreads();
  if (lane == 63) redi[wave] = incl;
  __syncthreads();
  int before = incl - cnt, total = 0;  // ties in runs below this one, in all runs
#pragma unroll
  for (int w = 0; w < SEL_NW; ++w) {
    if (w < wave) before += redi[w];
    total += redi[w];
  }
  const int after = total - before - cnt;     // ties in runs above this one
  if (after < take && after + cnt >= take) {
    int r = take - after;
    int cut = j0;
    for (int j = j1 - 1; j >= j0; --j)
      if (is_cand(mrow, cl, j) && ordered_key(xrow[j]) == v && --r == 0) {
        cut = j;
        break;
      }
    sh.tie_from = cut;
  }
  __syncthreads();
  tie_from = sh.tie_from;
}

__device__ __forceinline__ bool long_in_top(uint32_t key, int j, uint32_t v, int tie_from) {
  return (v != 0xffffffffu && key > v) || (key == v && j >= tie_from);
}

__global__ __launch_bounds__(SEL_NT) void solve_T_long_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const float* __restrict__ x, const int32_t* __restrict__ k_arr, const float* __restrict__ target,
    float T_lo, float T_hi, int iters, float* __restrict__ T_out) {
  __shared__ float red[SEL_NW];
  __shared__ int redi[SEL_NW];
  __shared__ LongTopK sh;
  const int h = blockIdx.x, tid = threadIdx.x;
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  const float* xrow = x + (size_t)h * S_max;

  float mx = -INFINITY;
  int nc = 0;
  for (int j = tid; j < S_max; j += SEL_NT)
    if (is_cand(mrow, cl, j)) {
      ++nc;
      mx = fmaxf(mx, xrow[j]);
    }
  mx = block_max<SEL_NT>(mx, red);
  const int n_cand = block_sum_int<SEL_NT>(nc, redi);
  const int kk = min(max(k_arr[h], 0), n_cand);
  uint32_t v;
  int tie_from;
  long_topk(S_max, mrow, cl, xrow, kk, v, tie_from, sh, redi);

  const float tgt = target[h];
  float a = logf(T_lo), b = logf(T_hi);
  for (int it = 0; it < iters; ++it) {
    const float mid = 0.5f * (a + b);
    const float invT = expf(-mid);
    float s_all = 0.f, s_top = 0.f;
    if (mx != -INFINITY)
      for (int j = tid; j < S_max; j += SEL_NT)
        if (is_cand(mrow, cl, j)) {
          const float xv = xrow[j];
          const float e = expf((xv - mx) * invT);
          s_all += e;
          if (kk > 0 && long_in_top(ordered_key(xv), j, v, tie_from)) s_top += e;
        }
    s_all = block_sum<SEL_NT>(s_all, red);
    s_top = block_sum<SEL_NT>(s_top, red);
    const float mass = (s_all > 0.f) ? s_top / s_all : 0.f;
    if (mass - tgt > 0.f) a = mid;
    else b = mid;
  }
  if (tid == 0) T_out[h] = expf(0.5f * (a + b));
}

// a2': temperature by gradient descent (Alg. 1, Solution 2 form).  theta = log T, loss
// (M_k(Softmax(x/T)) - target)^2, Adam (0.9 / 0.999 / 1e-8, bias-corrected, no weight
// decay).  M_k and its derivative come from four block sums per iteration:
// with u = 1/T and e = exp(u (x - max x)), M = sum_top e / sum e and
// dM/dtheta = -u M (E_top[x] - E_all[x]).
template <int EPT>
__global__ __launch_bounds__(SEL_NT) void solve_T_gd_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const float* __restrict__ x, const int32_t* __restrict__ k_arr, const float* __restrict__ target,
    float T_init, float lr, int iters, float tol, float* __restrict__ T_out, float* __restrict__ loss_out) {
  __shared__ float red[SEL_NW];
  __shared__ float red4[4][SEL_NW];
  __shared__ int redi[SEL_NW];
  __shared__ int tiecnt[EPT * SEL_NW];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  const float* xrow = x + (size_t)h * S_max;
  uint32_t cbits = 0, key[EPT];
  float xv[EPT];
  float mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < EPT; ++i) {
    const int j = tid + SEL_NT * i;
    key[i] = 0;
    xv[i] = -INFINITY;
    if (j < S_max && is_cand(mrow, cl, j)) {
      cbits |= 1u << i;
      xv[i] = xrow[j];
      key[i] = ordered_key(xv[i]);
      mx = fmaxf(mx, xv[i]);
    }
  }
  mx = block_max<SEL_NT>(mx, red);
  const int n_cand = block_sum_int<SEL_NT>(__popc(cbits), redi);
  const int kk = min(max(k_arr[h], 0), n_cand);
  const uint32_t top = topk_set<EPT>(key, cbits, kk, redi, tiecnt);
  const float tgt = target[h];
  // M_k and dM/dtheta at theta (uniform across the block)
  auto mass_grad = [&](float theta, float& M, float& dM) {
    M = 0.f;
    dM = 0.f;
    if (kk <= 0 || mx == -INFINITY) return;
    const float u = expf(-theta);
    float q[4] = {0.f, 0.f, 0.f, 0.f};    // sum e, sum_top e, sum x e, sum_top x e
#pragma unroll
    for (int i = 0; i < EPT; ++i)
      if ((cbits >> i) & 1u) {
        const float e = expf((xv[i] - mx) * u);
        const float xe = e > 0.f ? xv[i] * e : 0.f;
        q[0] += e;
        q[2] += xe;
        if ((top >> i) & 1u) {
          q[1] += e;
          q[3] += xe;
        }
      }
#pragma unroll
    for (int c = 0; c < 4; ++c) q[c] = wave_sum(q[c]);
    __syncthreads();
    if (lane == 0)
#pragma unroll
      for (int c = 0; c < 4; ++c) red4[c][wave] = q[c];
    __syncthreads();
    float t4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < SEL_NW; ++w)
#pragma unroll
      for (int c = 0; c < 4; ++c) t4[c] += red4[c][w];
    if (t4[1] == 0.f) return;
    M = t4[1] / t4[0];
    dM = -u * M * (t4[3] / t4[1] - t4[2] / t4[0]);
  };
  float theta = logf(T_init), m = 0.f, v = 0.f, b1t = 1.f, b2t = 1.f, loss = 0.f;
  for (int t = 1; t <= iters; ++t) {
    float M, dM;
    mass_grad(theta, M, dM);
    const float gap = M - tgt;
    loss = gap * gap;
    if (loss < tol) break;
    const float g = 2.f * gap * dM;
    m = 0.9f * m + 0.1f * g;
    v = 0.999f * v + 0.001f * g * g;
    b1t *= 0.9f;
    b2t *= 0.999f;
    theta -= lr * (m / (1.f - b1t)) / (sqrtf(v / (1.f - b2t)) + 1e-8f);
  }
  if (iters > 0) {
    float M, dM;
    mass_grad(theta, M, dM);
    loss = (M - tgt) * (M - tgt);
  }
  if (tid == 0) {
    T_out[h] = expf(theta);
    if (loss_out) loss_out[h] = loss;
  }
}

// The gradient-descent temperature for rows longer than 32768 slots: the same Adam steps on
// the same loss, the Top-k set from long_topk and each step's four sums from one sweep of
// the row in memory.
__global__ __launch_bounds__(SEL_NT) void solve_T_gd_long_kernel(
    int S_max, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    const float* __restrict__ x, const int32_t* __restrict__ k_arr, const float* __restrict__ target,
    float T_init, float lr, int iters, float tol, float* __restrict__ T_out, float* __restrict__ loss_out) {
  __shared__ float red[SEL_NW];
  __shared__ float red4[4][SEL_NW];
  __shared__ int redi[SEL_NW];
  __shared__ LongTopK sh;
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cl = cand_len[h];
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  const float* xrow = x + (size_t)h * S_max;
  float mx = -INFINITY;
  int nc = 0;
  for (int j = tid; j < S_max; j += SEL_NT)
    if (is_cand(mrow, cl, j)) {
      ++nc;
      mx = fmaxf(mx, xrow[j]);
    }
  mx = block_max<SEL_NT>(mx, red);
  const int n_cand = block_sum_int<SEL_NT>(nc, redi);
  const int kk = min(max(k_arr[h], 0), n_cand);
  uint32_t vthr;
  int tie_from;
  long_topk(S_max, mrow, cl, xrow, kk, vthr, tie_from, sh, redi);
  const float tgt = target[h];
  // M_k and dM/dtheta at theta (uniform across the block)
  auto mass_grad = [&](float theta, float& M, float& dM) {
    M = 0.f;
    dM = 0.f;
    if (kk <= 0 || mx == -INFINITY) return;
    const float u = expf(-theta);
    float q[4] = {0.f, 0.f, 0.f, 0.f};    // sum e, sum_top e, sum x e, sum_top x e
    for (int j = tid; j < S_max; j += SEL_NT)
      if (is_cand(mrow, cl, j)) {
        const float xv = xrow[j];
        const float e = expf((xv - mx) * u);
        const float xe = e > 0.f ? xv * e : 0.f;
        q[0] += e;
        q[2] += xe;
        if (long_in_top(ordered_key(xv), j, vthr, tie_from)) {
          q[1] += e;
          q[3] += xe;
        }
      }
#pragma unroll
    for (int c = 0; c < 4; ++c) q[c] = wave_sum(q[c]);
    __syncthreads();
    if (lane == 0)
#pragma unroll
      for (int c = 0; c < 4; ++c) red4[c][wave] = q[c];
    __syncthreads();
    float t4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < SEL_NW; ++w)
#pragma unroll
      for (int c = 0; c < 4; ++c) t4[c] += red4[c][w];
    if (t4[1] == 0.f) return;
    M = t4[1] / t4[0];
    dM = -u * M * (t4[3] / t4[1] - t4[2] / t4[0]);
  };
  float theta = logf(T_init), m = 0.f, v = 0.f, b1t = 1.f, b2t = 1.f, loss = 0.f;
  for (int t = 1; t <= iters; ++t) {
    float M, dM;
    mass_grad(theta, M, dM);
    const float gap = M - tgt;
    loss = gap * gap;
    if (loss < tol) break;
    const float g = 2.f * gap * dM;
    m = 0.9f * m + 0.1f * g;
    v = 0.999f * v + 0.001f * g * g;
    b1t *= 0.9f;
    b2t *= 0.999f;
    theta -= lr * (m / (1.f - b1t)) / (sqrtf(v / (1.f - b2t)) + 1e-8f);
  }
  if (iters > 0) {
    float M, dM;
    mass_grad(theta, M, dM);
    loss = (M - tgt) * (M - tgt);
  }
  if (tid == 0) {
    T_out[h] = expf(theta);
    if (loss_out) loss_out[h] = loss;
  }
}

static int ept_for(int S_max) {
  const int e = (S_max + SEL_NT - 1) / SEL_NT;
  if (e <= 1) return 1;
  if (e <= 2) return 2;
  if (e <= 4) return 4;
  if (e <= 8) return 8;
  if (e <= 16) return 16;
  return 32;
}

#define HK_EPT_SWITCH(S_max, CALL)        \
  switch (ept_for(S_max)) {               \
    case 1: { constexpr int E = 1; CALL; break; } \
    case 2: { constexpr int E = 2; CALL; break; } \
    case 4: { constexpr int E = 4; CALL; break; } \
    case 8: { constexpr int E = 8; CALL; break; } \
    case 16: { constexpr int E = 16; CALL; break; } \
    default: { constexpr int E = 32; CALL; break; } \
  }

}  // namespace hk

using namespace hk;

hipError_t hk_launch_calibrate(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                               int n_metrics, const float* x0, const float* x1, const float* T0,
                               const float* T1, float w0, float w1, float* c_out, float* lse_out,
                               hipStream_t st) {
  TimedLaunch t(HK_TK_CALIBRATE, st);
  HK_EPT_SWITCH(S_max, {
    const size_t lds = (size_t)E * SEL_NT * sizeof(float);   // dynamic LDS: a metric's row
    allow_dynamic_lds<calibrate_kernel<E>>(lds);
    hipLaunchKernelGGL((calibrate_kernel<E>), dim3(n_heads), dim3(SEL_NT), lds, st, S_max, cand_len,
                       mask, n_metrics, x0, x1, T0, T1, w0, w1, c_out, lse_out);
  });
  return hipGetLastError();
}

// (dynamic LDS of the Top-p kernels: the packed key list of the low-bit search)
hipError_t hk_launch_topp(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                          const float* c, int p_q, int k_min, int k_max, uint32_t* sel_bits,
                          int32_t* k_out, float* sel_mass, int32_t* status, hipStream_t st) {
  const size_t lds = (size_t)S_max * sizeof(uint32_t);
  TimedLaunch t(HK_TK_TOPP, st);
  HK_EPT_SWITCH(S_max, {
    allow_dynamic_lds<topp_kernel<E>>(lds);
    hipLaunchKernelGGL((topp_kernel<E>), dim3(n_heads), dim3(SEL_NT), lds, st, S_max, cand_len, mask,
                       c, p_q, k_min, k_max, sel_bits, k_out, sel_mass, status);
  });
  return hipGetLastError();
}

hipError_t hk_launch_calib_topp(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                                int n_metrics, const float* x0, const float* x1, const float* T0,
                                const float* T1, float w0, float w1, int p_q, int k_min, int k_max,
                                float* c_out, float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                                float* sel_mass, int32_t* status, hipStream_t st) {
  TimedLaunch t(HK_TK_CALIB_TOPP, st);
  HK_EPT_SWITCH(S_max, {
    // the key list, and before it a metric's row (EPT * SEL_NT floats >= S_max)
    const size_t lds = (size_t)E * SEL_NT * sizeof(uint32_t);
    allow_dynamic_lds<calib_topp_kernel<E>>(lds);
    hipLaunchKernelGGL((calib_topp_kernel<E>), dim3(n_heads), dim3(SEL_NT), lds, st, S_max, cand_len,
                       mask, n_metrics, x0, x1, T0, T1, w0, w1, p_q, k_min, k_max, c_out, lse_out,
                       sel_bits, k_out, sel_mass, status);
  });
  return hipGetLastError();
}

hipError_t hk_launch_pool_max(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                              const float* x, int radius, float* out, hipStream_t st) {
  hipLaunchKernelGGL(pool_max_kernel, dim3((S_max + POOL_TILE - 1) / POOL_TILE, n_heads), dim3(POOL_NT),
                     0, st, S_max, cand_len, mask, x, radius, out);
  return hipGetLastError();
}

hipError_t hk_launch_solve_T_gd(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                                const float* x, const int32_t* k, const float* target, float T_init,
                                float lr, int iters, float tol, float* T_out, float* loss_out,
                                hipStream_t st) {
  TimedLaunch t(HK_TK_SOLVE_T, st);
  if (S_max > SEL_NT * 32) {
    hipLaunchKernelGGL(solve_T_gd_long_kernel, dim3(n_heads), dim3(SEL_NT), 0, st, S_max, cand_len, mask,
                       x, k, target, T_init, lr, iters, tol, T_out, loss_out);
    return hipGetLastError();
  }
  HK_EPT_SWITCH(S_max, hipLaunchKernelGGL((solve_T_gd_kernel<E>), dim3(n_heads), dim3(SEL_NT), 0, st,
                                          S_max, cand_len, mask, x, k, target, T_init, lr, iters, tol,
                                          T_out, loss_out));
  return hipGetLastError();
}

hipError_t hk_launch_solve_T(int n_heads, int S_max, const int32_t* cand_len, const uint16_t* mask,
                             const float* x, const int32_t* k, const float* target, float T_lo,
                             float T_hi, int iters, float* T_out, hipStream_t st) {
  TimedLaunch t(HK_TK_SOLVE_T, st);
  if (S_max > SEL_NT * 32) {
    hipLaunchKernelGGL(solve_T_long_kernel, dim3(n_heads), dim3(SEL_NT), 0, st, S_max, cand_len, mask,
                       x, k, target, T_lo, T_hi, iters, T_out);
    return hipGetLastError();
  }
  HK_EPT_SWITCH(S_max, hipLaunchKernelGGL((solve_T_kernel<E>), dim3(n_heads), dim3(SEL_NT), 0, st,
                                          S_max, cand_len, mask, x, k, target, T_lo, T_hi, iters,
                                          T_out));
  return hipGetLastError();
}

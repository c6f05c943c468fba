// a2 + a3 with every head spread over many workgroups: Logits Calibration (Sec. 3.2,
// Solution 2) and head-adaptive Top-p (Sec. 3.2, Problem 1) for caches longer than one
// workgroup holds in registers, and so that a batch of heads fills every compute unit.
//
//   prep    one workgroup per (head, 2048-slot chunk): the chunk's max and sum of exp per
//           metric, the pieces of the head's log-sum-exp.
//   chunk   one workgroup per (head, chunk): the calibrated value c of each slot (written to
//           c_out when asked for) and its Top-p key, the bits of c clamped to [0, 1]; the
//           chunk's histogram by the key's top 9 bits (fixed-point weight and count per
//           digit, one packed LDS atomic per key, whose return value is the key's rank in
//           its digit), and the chunk's keys sorted by digit, descending (a counting sort:
//           digit offset + rank, staged in LDS, stored whole), each stored as its low 21
//           key bits and its 11-bit slot.
//   finish  one workgroup per head: sums the chunk histograms, picks the level-1 digit,
//           gathers that digit's keys from the chunks' sorted segments (into LDS when they
//           fit: always for heads of up to 32768 slots), refines the threshold over the low
//           21 bits in levels of 11 and 10 bits, applies the count clamp and breaks the ties
//           at the threshold toward the later slots (ties counted per 128-slot block, then
//           the cut found inside one block); writes the count, the selected mass and the
//           head's threshold.
//   bitmap  one workgroup per (head, chunk): every key of a higher digit is selected, the
//           keys of the threshold digit by the threshold rule, the rest not.
// The launches hand their results over through memory in stream order: no workgroup waits
// for another and no cross-die fence is needed.
//
// The rule is the one of the single-workgroup selector: weights w = floor(c * 2^40),
// target = ceil(p_q * Total / 10^6), the smallest set in (key desc, slot desc) order whose
// weight reaches the target, then the count clamp; every quantity is an exact integer, so
// the result does not depend on how the work is split.
#include "hk_internal.h"

namespace hk {
namespace {

constexpr int SW_NT = 256;                     // threads of a chunk workgroup
constexpr int SW_NW = SW_NT / 64;
constexpr int SW_CH = 2048;                    // slots per chunk
constexpr int SW_CS = 11;                      // bits of a chunk-local slot
constexpr int SW_FT = 1024;                    // threads of the finishing workgroup
constexpr int SW_FW = SW_FT / 64;
constexpr int SW_B1 = 512, SW_SH1 = 21;        // level 1: key bits 29..21
constexpr int SW_B2 = 2048, SW_SH2 = 10;       // level 2: bits 20..10
constexpr int SW_B3 = 1024;                    // level 3: bits 9..0
constexpr uint32_t SW_LOW = (1u << SW_SH1) - 1u;
constexpr int SW_TSH = 7;                      // ties counted per block of 128 slots
constexpr int SW_LIST = 32768;                 // keys of one digit the finishing workgroup holds
constexpr int SW_CMAX = 128;                   // chunks per head at most (S_max <= 262144)
constexpr uint32_t SW_NONE = 0xffffffffu;      // key of a non-candidate / no threshold
// a packed histogram entry: count << 52 | weight (a chunk's count <= 2048 < 2^12 and its
// weight <= 2048 * 2^40 < 2^52, so neither field overflows into the other)
constexpr int SW_CNT_SH = 52;
constexpr unsigned long long SW_WMASK = (1ull << SW_CNT_SH) - 1ull;
constexpr size_t SW_LDS = (size_t)SW_LIST * 4 + SW_B2 * 12;   // dynamic LDS of finish
static_assert(SW_B1 == 2 * SW_NT && SW_B1 * 2 == SW_FT && SW_B2 == 2 * SW_FT && SW_B3 == SW_FT,
              "bins per thread");
static_assert(SW_CH == 2 * 4 * SW_NT, "two float4 per thread and chunk");

// Fixed-point weight floor(v * 2^40) of a value v in [0, 1] from its bits, as its two exact
// 32-bit halves: with t = v * 2^8 (exact, t <= 256) the high half is floor(t) and the low
// half floor(fract(t) * 2^32).
__device__ __forceinline__ unsigned long long sw_weight(uint32_t key) {
  const float t = __uint_as_float(key) * 256.0f;
  const uint32_t hi = (uint32_t)t;
  const uint32_t lo = (uint32_t)(__builtin_amdgcn_fractf(t) * 4294967296.0f);
  return ((unsigned long long)hi << 32) | lo;
}

// Inclusive prefix sum of a 64-bit value over the wave's lanes: row shifts by 1, 2, 4, 8
// within each 16-lane row, then the row broadcasts of lanes 15 and 31 (DPP lane moves, no
// LDS round trip), on the two 32-bit halves with the carry.
__device__ __forceinline__ unsigned long long sw_wave_scan(unsigned long long x) {
  uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
#define SW_SCAN_STEP(CTRL, RM)                                                                    \
  {                                                                                               \
    const uint32_t tl = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)lo, CTRL, RM, 0xf, false);  \
    const uint32_t th = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)hi, CTRL, RM, 0xf, false);  \
    const unsigned long long r = (((unsigned long long)hi << 32) | lo) +                          \
                                 (((unsigned long long)th << 32) | tl);                           \
    lo = (uint32_t)r;                                                                             \
    hi = (uint32_t)(r >> 32);                                                                     \
  }
  SW_SCAN_STEP(0x111, 0xf)                 // row_shr:1
  SW_SCAN_STEP(0x112, 0xf)                 // row_shr:2
  SW_SCAN_STEP(0x114, 0xf)                 // row_shr:4
  SW_SCAN_STEP(0x118, 0xf)                 // row_shr:8
  SW_SCAN_STEP(0x142, 0xa)                 // row_bcast:15 into rows 1 and 3
  SW_SCAN_STEP(0x143, 0xc)                 // row_bcast:31 into rows 2 and 3
#undef SW_SCAN_STEP
  return ((unsigned long long)hi << 32) | lo;
}

// A value every lane holds alike, moved to scalar registers.
__device__ __forceinline__ unsigned long long sw_uniform(unsigned long long x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(x >> 32));
  return ((unsigned long long)hi << 32) | lo;
}

// The thread's four consecutive slots of half r of chunk c start at this slot.
__device__ __forceinline__ int sw_group(int c, int r) {
  return c * SW_CH + r * (SW_CH / 2) + (int)threadIdx.x * 4;
}

// Candidate bits of the thread's 8 slots (bit 4 r + e: slot sw_group(c, r) + e).  Four
// consecutive slots share one page-mask word.
__device__ __forceinline__ uint32_t sw_cand(int h, int c, int S_max, const int32_t* __restrict__ cand_len,
                                            const uint16_t* __restrict__ mask) {
  const int cl = min(cand_len[h], S_max);
  const uint16_t* mrow = mask ? mask + (size_t)h * (S_max / HK_PAGE) : nullptr;
  uint32_t cb = 0;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int j0 = sw_group(c, r);
    const uint32_t mw = mrow ? (uint32_t)mrow[min(j0, S_max - 1) >> 4] : 0xffffu;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = j0 + e;
      if (j < cl && ((mw >> (j & 15)) & 1u)) cb |= 1u << (4 * r + e);
    }
  }
  return cb;
}

// The 8 values of the thread (two float4 loads; a group past the row's end is read from the
// row's last group, and its slots are not candidates).
__device__ __forceinline__ void sw_load8(const float* __restrict__ row, int c, int S_max, float (&v)[8]) {
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const float4 q = *reinterpret_cast<const float4*>(row + min(sw_group(c, r), S_max - 4));
    v[4 * r + 0] = q.x;
    v[4 * r + 1] = q.y;
    v[4 * r + 2] = q.z;
    v[4 * r + 3] = q.w;
  }
}

__global__ __launch_bounds__(SW_NT) void sw_prep_kernel(
    int S_max, int C, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    int n_metrics, const float* __restrict__ x0, const float* __restrict__ x1,
    const float* __restrict__ T0, const float* __restrict__ T1, float2* __restrict__ part) {
  __shared__ float red[2][SW_NW];
  const int c = (int)blockIdx.x % C, h = (int)blockIdx.x / C, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t cb = sw_cand(h, c, S_max, cand_len, mask);
  for (int m = 0; m < n_metrics; ++m) {
    const float* Tp = (m == 0 ? T0 : T1);
    const float T = Tp ? Tp[h] : 1.0f;
    float t[8];
    sw_load8((m == 0 ? x0 : x1) + (size_t)h * S_max, c, S_max, t);
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      t[i] = t[i] / T;
      if ((cb >> i) & 1u) mx = fmaxf(mx, t[i]);
    }
    mx = wave_max(mx);
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    float sm = 0.f;
    if (mx != -INFINITY)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if ((cb >> i) & 1u) sm += expf(t[i] - mx);
    sm = wave_sum(sm);
    if (lane == 0) red[1][wave] = sm;
    __syncthreads();
    if (tid == 0)
      part[((size_t)h * C + c) * 2 + m] = make_float2(mx, (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]));
    __syncthreads();                     // red is reused by the next metric
  }
}

template <bool CALIB>
__global__ __launch_bounds__(SW_NT) void sw_chunk_kernel(
    int S_max, int C, const int32_t* __restrict__ cand_len, const uint16_t* __restrict__ mask,
    int n_metrics, const float* __restrict__ x0, const float* __restrict__ x1,
    const float* __restrict__ T0, const float* __restrict__ T1, float w0, float w1,
    const float2* __restrict__ part, const float* __restrict__ c_in, float* __restrict__ c_out,
    float* __restrict__ lse_out, unsigned long long* __restrict__ hp, uint16_t* __restrict__ ho,
    uint32_t* __restrict__ sorted, int32_t* __restrict__ status) {
  __shared__ unsigned long long hist[SW_B1];
  __shared__ uint32_t offs[SW_B1];
  __shared__ __align__(16) uint32_t stage[SW_CH];
  __shared__ uint32_t wsum[SW_NW];
  __shared__ float s_lse[2];
  const int c = (int)blockIdx.x % C, h = (int)blockIdx.x / C, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const uint32_t cb = sw_cand(h, c, S_max, cand_len, mask);
  hist[tid] = 0ull;
  hist[tid + SW_NT] = 0ull;

  float cv[8];
  if constexpr (CALIB) {
    float t[2][8];
#pragma unroll
    for (int m = 0; m < 2; ++m)
      if (m < n_metrics) sw_load8((m == 0 ? x0 : x1) + (size_t)h * S_max, c, S_max, t[m]);
    if (wave < n_metrics) {
      // the head's log-sum-exp of metric `wave` from its C chunk pieces (lanes q, q + 64)
      const float2* pp = part + (size_t)h * C * 2 + wave;
      const float2 a = lane < C ? pp[lane * 2] : make_float2(-INFINITY, 0.f);
      const float2 b = lane + 64 < C ? pp[(lane + 64) * 2] : make_float2(-INFINITY, 0.f);
      const float M = wave_max(fmaxf(a.x, b.x));
      float L = 0.f;
      if (M != -INFINITY) {
        if (a.x != -INFINITY) L += a.y * expf(a.x - M);
        if (b.x != -INFINITY) L += b.y * expf(b.x - M);
      }
      L = wave_sum(L);
      const float lse = M == -INFINITY ? -INFINITY : M + logf(L);
      if (lane == 0) {
        s_lse[wave] = lse;
        if (lse_out && c == 0) lse_out[(size_t)h * n_metrics + wave] = lse;
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) cv[i] = 0.f;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      if (m >= n_metrics) break;
      const float* Tp = (m == 0 ? T0 : T1);
      const float T = Tp ? Tp[h] : 1.0f;
      const float wm = m == 0 ? w0 : w1, lse = s_lse[m];
      if (lse != -INFINITY)
#pragma unroll
        for (int i = 0; i < 8; ++i)
          if ((cb >> i) & 1u) cv[i] = fmaf(wm, expf(t[m][i] / T - lse), cv[i]);
    }
    if (c_out)
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int j0 = sw_group(c, r);
        if (j0 < S_max)
          *reinterpret_cast<float4*>(c_out + (size_t)h * S_max + j0) =
              make_float4(cv[4 * r], cv[4 * r + 1], cv[4 * r + 2], cv[4 * r + 3]);
      }
  } else {
    sw_load8(c_in + (size_t)h * S_max, c, S_max, cv);
    __syncthreads();                     // the cleared histogram is visible
  }

  // keys, and the packed histogram: the returned count is the key's rank in its digit
  int flags = 0;
  uint32_t key[8], rank[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float v = cv[i];
    key[i] = SW_NONE;
    rank[i] = 0;
    if ((cb >> i) & 1u) {
      if (v != v) { v = 0.f; flags |= HK_FLAG_NAN; }
      if (v > 1.f) { v = 1.f; flags |= HK_FLAG_RANGE; }
      if (v < 0.f) { v = 0.f; flags |= HK_FLAG_RANGE; }
      if (v == 0.f) v = 0.f;                      // canonical +0
      key[i] = __float_as_uint(v);
      const unsigned long long old =
          atomicAdd(&hist[key[i] >> SW_SH1], (1ull << SW_CNT_SH) | sw_weight(key[i]));
      rank[i] = (uint32_t)(old >> SW_CNT_SH);
    }
  }
  __syncthreads();
  // digit offsets of the sort, digits descending: thread t holds digits 511 - 2t - b
  uint32_t cnt[2], own = 0;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    cnt[b] = (uint32_t)(hist[SW_B1 - 1 - 2 * tid - b] >> SW_CNT_SH);
    own += cnt[b];
  }
  const uint32_t incl = (uint32_t)sw_wave_scan(own);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  uint32_t off = incl - own;
#pragma unroll
  for (int w = 0; w < SW_NW; ++w)
    if (w < wave) off += wsum[w];
  const size_t hb = ((size_t)h * C + c) * SW_B1;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int d = SW_B1 - 1 - 2 * tid - b;
    offs[d] = off;
    hp[hb + d] = hist[d];
    ho[hb + d] = (uint16_t)off;
    off += cnt[b];
  }
  __syncthreads();
  const uint32_t n_keys = offs[0] + (uint32_t)(hist[0] >> SW_CNT_SH);
#pragma unroll
  for (int i = 0; i < 8; ++i)
    if (key[i] != SW_NONE) {
      const uint32_t local = (uint32_t)((i >> 2) * (SW_CH / 2) + tid * 4 + (i & 3));
      stage[offs[key[i] >> SW_SH1] + rank[i]] = ((key[i] & SW_LOW) << SW_CS) | local;
    }
  __syncthreads();
  // the sorted keys, whole 16-byte pieces (the tail past n_keys is never read)
  uint32_t* srow = sorted + (size_t)h * S_max + (size_t)c * SW_CH;
  const uint32_t n_vec = (n_keys + 3) / 4;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const uint32_t q = (uint32_t)(r * SW_NT + tid);
    if (q < n_vec)
      reinterpret_cast<uint4*>(srow)[q] = reinterpret_cast<const uint4*>(stage)[q];
  }
  const int any_nan = __syncthreads_or(flags & HK_FLAG_NAN);
  const int any_range = __syncthreads_or(flags & HK_FLAG_RANGE);
  if (tid == 0 && status && (any_nan || any_range))
    atomicOr(status, (any_nan ? HK_FLAG_NAN : 0) | (any_range ? HK_FLAG_RANGE : 0));
}

// ------------------------------------------------------------------ the finishing workgroup
struct SwSh {
  unsigned long long rw[SW_FW], rc[SW_FW];
  unsigned long long p_aw, p_ac, p_w, p_c;
  uint32_t p_d;
  uint32_t seg_off[SW_CMAX], seg_pre[SW_CMAX];
  uint32_t seg_tot0;
  uint32_t tie_from;
  uint32_t tmask[4];
};

struct SwPick {
  uint32_t d;                              // the digit
  unsigned long long aw, ac;               // weight and count above it (including the caller's)
  unsigned long long w, c;                 // its own weight and count
};

// After a histogram level of NB bins: the digit where the criterion (weight, or count)
// summed from the top crosses the target.  Thread t holds BPT bins, digits D(t, b) = NB - 1 -
// (BPT * t + b) (threads past the bins hold zeros), so the digits descend with the thread
// and "above" is a prefix over the threads.  The totals are made wave-uniform, so the
// target's 64-bit arithmetic runs on the scalar unit.  aw0 / ac0 are the weight and count above this level's bins.  The target is
// target_of(total weight, total count) of the level (returned in *target, with the totals);
// for a target of 0 no digit is picked.  Two barriers; the results come back through LDS.
template <int BPT, int NB, typename TF>
__device__ __forceinline__ SwPick sw_pick(const unsigned long long (&bw)[BPT],
                                          const unsigned long long (&bc)[BPT], bool by_count,
                                          TF target_of, unsigned long long aw0,
                                          unsigned long long ac0, unsigned long long* target,
                                          unsigned long long* tot_w, unsigned long long* tot_c,
                                          SwSh& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  unsigned long long ow = 0, oc = 0;
#pragma unroll
  for (int b = 0; b < BPT; ++b) {
    ow += bw[b];
    oc += bc[b];
  }
  const unsigned long long iw = sw_wave_scan(ow), ic = sw_wave_scan(oc);
  if (lane == 63) {
    sh.rw[wave] = iw;
    sh.rc[wave] = ic;
  }
  __syncthreads();
  unsigned long long pw = 0, pc = 0, tw = 0, tc = 0;
#pragma unroll
  for (int w = 0; w < SW_FW; ++w) {
    const unsigned long long a = sh.rw[w], n = sh.rc[w];
    if (w < wave) {
      pw += a;
      pc += n;
    }
    tw += a;
    tc += n;
  }
  tw = sw_uniform(tw);
  tc = sw_uniform(tc);
  const unsigned long long tg = target_of(tw, tc);
  *target = tg;
  *tot_w = tw;
  *tot_c = tc;
  unsigned long long cw = aw0 + pw + iw - ow, cc = ac0 + pc + ic - oc;
  const unsigned long long lo = by_count ? cc : cw, own = by_count ? oc : ow;
  if (tg > 0 && lo < tg && lo + own >= tg) {
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
      const unsigned long long nxt = by_count ? cc + bc[b] : cw + bw[b];
      if (nxt >= tg) {
        sh.p_d = (uint32_t)(NB - 1 - (BPT * tid + b));
        sh.p_aw = cw;
        sh.p_ac = cc;
        sh.p_w = bw[b];
        sh.p_c = bc[b];
        break;
      }
      cw += bw[b];
      cc += bc[b];
    }
  }
  __syncthreads();
  return SwPick{sh.p_d, sh.p_aw, sh.p_ac, sh.p_w, sh.p_c};
}

struct SwFixed {
  unsigned long long t;
  __device__ unsigned long long operator()(unsigned long long, unsigned long long) const { return t; }
};

// The elements of the level-1 digit d1 of a head: the chunks' sorted segments, numbered
// 0 .. n - 1 in chunk order (seg_pre is the prefix of the segment lengths, seg_off their
// starts in the chunks' sorted keys).
struct SwSeg {
  const uint32_t* srow;                    // the head's sorted keys
  uint32_t d1;
  uint32_t n;
  int C;
  __device__ __forceinline__ uint32_t key_of(uint32_t p) const { return (d1 << SW_SH1) | (p >> SW_CS); }
};

struct SwFound {
  uint32_t v;                            // threshold key (SW_NONE: none)
  uint32_t d1;
  unsigned long long aw, ac;             // weight and count of the keys above v
  unsigned long long ntie;               // candidates with key == v
  bool list_mode;
  SwSeg seg;
};

// Calls f(key, i, p, q) for the elements i of digit d1 (p: the element as stored, q: its
// chunk), from the LDS list or from the chunks' segments.  With BY_CHUNK (or from the
// segments) one wave walks one chunk's elements at a time, which gives q; otherwise the
// list is walked flat and q is -1.
template <bool BY_CHUNK, typename F>
__device__ __forceinline__ void sw_for_each(const SwFound& r, const uint32_t* list, const SwSh& sh,
                                            F f) {
  if (r.list_mode && !BY_CHUNK) {
    for (uint32_t i = threadIdx.x; i < r.seg.n; i += SW_FT) {
      const uint32_t p = list[i];
      f(r.seg.key_of(p), i, p, -1);
    }
    return;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int q = wave; q < r.seg.C; q += SW_FW) {
    const uint32_t pre = sh.seg_pre[q];
    const uint32_t n = (q + 1 < r.seg.C ? sh.seg_pre[q + 1] : r.seg.n) - pre;
    const uint32_t* src = r.list_mode ? list + pre : r.seg.srow + (size_t)q * SW_CH + sh.seg_off[q];
    for (uint32_t i0 = 0; i0 < n; i0 += 64 * 4) {
      uint32_t p[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t i = i0 + u * 64 + lane;
        p[u] = i < n ? src[i] : 0u;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t i = i0 + u * 64 + lane;
        if (i < n) f(r.seg.key_of(p[u]), pre + i, p[u], q);
      }
    }
  }
}

// One lower level: the histogram of the NB = 2^bits key values at `shift` over the elements
// whose bits above them equal `prefix`, then the pick against the fixed target.
template <int NB>
__device__ __forceinline__ SwPick sw_level(const SwFound& r, const uint32_t* list, uint32_t prefix,
                                           int shift,
                                           bool by_count, unsigned long long target,
                                           const SwPick& above, unsigned long long* hw2,
                                           uint32_t* hc2, SwSh& sh) {
  constexpr int BPT = NB / SW_FT, BITS = NB == 2048 ? 11 : 10;
  const int tid = threadIdx.x;
#pragma unroll
  for (int b = 0; b < BPT; ++b) {
    hw2[b * SW_FT + tid] = 0ull;
    hc2[b * SW_FT + tid] = 0u;
  }
  __syncthreads();
  sw_for_each<false>(r, list, sh, [&](uint32_t k, uint32_t, uint32_t, int) {
    if ((k >> (shift + BITS)) == prefix) {
      const uint32_t b = (k >> shift) & (NB - 1);
      atomicAdd(&hw2[b], sw_weight(k));
      atomicAdd(&hc2[b], 1u);
    }
  });
  __syncthreads();
  unsigned long long bw[BPT], bc[BPT];
#pragma unroll
  for (int b = 0; b < BPT; ++b) {
    bw[b] = hw2[NB - 1 - (BPT * tid + b)];
    bc[b] = hc2[NB - 1 - (BPT * tid + b)];
  }
  unsigned long long tg, tw, tc;
  return sw_pick<BPT, NB>(bw, bc, by_count, SwFixed{target}, above.aw, above.ac, &tg, &tw, &tc, sh);
}

// The largest key v whose criterion summed over keys >= v reaches the target (weights, or
// counts when by_count), target = target_of(total weight, total count) -- returned in
// *target with the totals -- from the head's level-1 histogram (bw1 / bc1: this thread's
// digit) and the chunks' sorted segments of the picked digit.
template <typename TF>
__device__ __forceinline__ SwFound sw_search(const unsigned long long (&bw1)[1],
                                             const unsigned long long (&bc1)[1], bool by_count,
                                             TF target_of, unsigned long long* target,
                                             unsigned long long* tot_w, unsigned long long* tot_c,
                                             const unsigned long long* __restrict__ hprow,
                                             const uint16_t* __restrict__ horow,
                                             const uint32_t* __restrict__ srow, int C,
                                             uint32_t* list, unsigned long long* hw2,
                                             uint32_t* hc2, SwSh& sh) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  SwFound r;
  r.v = SW_NONE;
  r.d1 = 0;
  r.aw = r.ac = r.ntie = 0;
  r.list_mode = false;
  r.seg = SwSeg{srow, 0u, 0u, C};
  const SwPick p1 = sw_pick<1, SW_B1>(bw1, bc1, by_count, target_of, 0ull, 0ull, target, tot_w,
                                      tot_c, sh);
  const unsigned long long tg = *target;
  if (tg == 0) return r;
  const uint32_t d1 = p1.d;
  r.d1 = d1;
  // the digit's segment in every chunk and the prefix of their lengths (waves 0 and 1 hold
  // chunks q = 64 * wave + lane < 128)
  if (wave < 2) {
    const int q = wave * 64 + lane;
    const uint32_t n = q < C ? (uint32_t)(hprow[(size_t)q * SW_B1 + d1] >> SW_CNT_SH) : 0u;
    const uint32_t incl = (uint32_t)sw_wave_scan(n);
    sh.seg_off[q] = q < C ? (uint32_t)horow[(size_t)q * SW_B1 + d1] : 0u;
    sh.seg_pre[q] = incl - n;
    if (wave == 0 && lane == 63) sh.seg_tot0 = incl;
  }
  __syncthreads();
  if (wave == 1) sh.seg_pre[64 + lane] += sh.seg_tot0;
  __syncthreads();
  r.seg = SwSeg{srow, d1, (uint32_t)p1.c, C};
  r.list_mode = p1.c <= SW_LIST;
  if (r.list_mode) {
    // one wave per chunk: its segment, contiguous, into the list at the segment's prefix
    r.list_mode = false;
    sw_for_each<true>(r, list, sh, [&](uint32_t, uint32_t i, uint32_t p, int) { list[i] = p; });
    r.list_mode = true;
    __syncthreads();
  }
  const SwPick p2 = sw_level<SW_B2>(r, list, d1, SW_SH2, by_count, tg, p1, hw2, hc2, sh);
  const uint32_t pre = (d1 << 11) | p2.d;
  const SwPick p3 = sw_level<SW_B3>(r, list, pre, 0, by_count, tg, p2, hw2, hc2, sh);
  r.v = (pre << 10) | p3.d;
  r.aw = p3.aw;
  r.ac = p3.ac;
  r.ntie = p3.c;
  return r;
}

__global__ __launch_bounds__(SW_FT) void sw_finish_kernel(
    int S_max, int C, const unsigned long long* __restrict__ hp, const uint16_t* __restrict__ ho,
    const uint32_t* __restrict__ sorted, int p_q, int k_min, int k_max, uint4* __restrict__ params,
    int32_t* __restrict__ k_out, float* __restrict__ sel_mass) {
  extern __shared__ __align__(16) unsigned char sw_dyn[];
  __shared__ SwSh sh;
  const int h = blockIdx.x, tid = threadIdx.x;
  uint32_t* list = reinterpret_cast<uint32_t*>(sw_dyn);
  unsigned long long* hw2 = reinterpret_cast<unsigned long long*>(sw_dyn + (size_t)SW_LIST * 4);
  uint32_t* hc2 = reinterpret_cast<uint32_t*>(sw_dyn + (size_t)SW_LIST * 4 + SW_B2 * 8);
  // the halves of the level-1 sums, in the list's space before the list is used
  unsigned long long(*s_half)[SW_B1] = reinterpret_cast<unsigned long long(*)[SW_B1]>(sw_dyn);
  const unsigned long long* hprow = hp + (size_t)h * C * SW_B1;
  const uint16_t* horow = ho + (size_t)h * C * SW_B1;
  const uint32_t* srow = sorted + (size_t)h * S_max;

  // the head's level-1 histogram: threads t and t + 512 sum digit 511 - t over the even and
  // the odd chunks; thread t < 512 then holds the digit's total
  unsigned long long bw1[1] = {0ull}, bc1[1] = {0ull};
  {
    const int d = SW_B1 - 1 - (tid & (SW_B1 - 1)), half = tid >> 9;
    const unsigned long long* pp = hprow + d;
    for (int q0 = half; q0 < C; q0 += 32) {
      unsigned long long a[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int q = q0 + 2 * u;
        a[u] = q < C ? pp[(size_t)q * SW_B1] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        bw1[0] += a[u] & SW_WMASK;
        bc1[0] += a[u] >> SW_CNT_SH;
      }
    }
    if (half) {
      s_half[0][tid - SW_B1] = bw1[0];
      s_half[1][tid - SW_B1] = bc1[0];
    }
    __syncthreads();
    if (half) {
      bw1[0] = 0ull;
      bc1[0] = 0ull;
    } else {
      bw1[0] += s_half[0][tid];
      bc1[0] += s_half[1][tid];
    }
  }

  // mass rule: target = ceil(p_q * Total / 10^6) (the level-1 pick computes it from the total)
  const unsigned long long pq = (unsigned long long)p_q;
  const auto mass_target = [pq](unsigned long long tw, unsigned long long) {
    return pq * (tw / 1000000ull) + (pq * (tw % 1000000ull) + 999999ull) / 1000000ull;
  };
  unsigned long long target, tot_w, tot_c;
  SwFound f = sw_search(bw1, bc1, false, mass_target, &target, &tot_w, &tot_c, hprow, horow,
                        srow, C, list, hw2, hc2, sh);
  const int n_cand = (int)tot_c;
  unsigned long long take = 0, wv = 0;
  long long k = 0;
  if (target > 0) {
    // block-uniform values: the 64-bit division runs on the scalar unit
    wv = sw_uniform(sw_weight(f.v));     // > 0: the crossing key weighs
    take = (sw_uniform(target) - sw_uniform(f.aw) + wv - 1) / wv;
    k = (long long)(sw_uniform(f.ac) + take);
  }
  // count clamp
  const int lo = min(max(k_min, 0), n_cand);
  const int hi = (k_max > 0) ? min(k_max, n_cand) : n_cand;
  const int kf = (int)max((long long)lo, min(k, (long long)hi));
  const bool by_mass = kf == k && target > 0;
  if (!by_mass) {
    if (kf == 0) {
      f.v = SW_NONE;
      f.aw = f.ac = f.ntie = 0;
      take = 0;
      wv = 0;
    } else {
      unsigned long long t2, w2, c2;
      f = sw_search(bw1, bc1, true, SwFixed{(unsigned long long)kf}, &t2, &w2, &c2, hprow, horow,
                    srow, C, list, hw2, hc2, sh);
      wv = sw_weight(f.v);
      take = (unsigned long long)kf - f.ac;
    }
  }
  const unsigned long long msel = f.aw + take * wv;

  // ties at v: the `take` with the largest slots, i.e. those at or after tie_from
  uint32_t tie_from = take >= f.ntie ? 0u : (uint32_t)S_max;
  const auto slot = [](uint32_t p, int q) { return (uint32_t)q * SW_CH + (p & (SW_CH - 1)); };
  if (take > 0 && take < f.ntie && S_max <= 32 * SW_FT) {
    // rows of up to 32768 slots: one pass sets the ties' bits in a slot bitmap (one word per
    // thread), a suffix count of the words from the top finds the word holding the cut, and
    // the cut inside it comes from registers
    uint32_t* tb = reinterpret_cast<uint32_t*>(hw2);     // [S_max / 32] words
    tb[tid] = 0u;
    __syncthreads();
    const uint32_t v = f.v;
    sw_for_each<true>(f, list, sh, [&](uint32_t kk, uint32_t, uint32_t p, int q) {
      if (kk == v) {
        const uint32_t j = slot(p, q);
        atomicOr(&tb[j >> 5], 1u << (j & 31));
      }
    });
    __syncthreads();
    // thread t takes word W - 1 - t, so the words descend with the thread and "above" is a
    // prefix over the threads
    const int nwords = S_max / 32;
    const int wd = nwords - 1 - tid;
    const uint32_t word = wd >= 0 ? tb[wd] : 0u;
    const uint32_t cnt = (uint32_t)__popc(word);
    const unsigned long long incl = sw_wave_scan((unsigned long long)cnt);
    if ((tid & 63) == 63) sh.rc[tid >> 6] = incl;
    __syncthreads();
    unsigned long long above = incl - cnt;
#pragma unroll
    for (int w = 0; w < SW_FW; ++w)
      if (w < (tid >> 6)) above += sh.rc[w];
    if (above < take && above + cnt >= take) {
      // the (take - above)-th set bit from the top of this word
      uint32_t x = word;
      for (unsigned long long i = 1; i < take - above; ++i) x &= ~(0x80000000u >> __clz(x));
      sh.tie_from = (uint32_t)wd * 32u + (uint32_t)(31 - __clz(x));
    }
    __syncthreads();
    tie_from = sh.tie_from;
  } else if (take > 0 && take < f.ntie) {
    uint32_t* th = reinterpret_cast<uint32_t*>(hw2);     // ties per 128-slot block (<= 2048)
    th[2 * tid] = 0u;
    th[2 * tid + 1] = 0u;
    if (tid < 4) sh.tmask[tid] = 0u;
    __syncthreads();
    const uint32_t v = f.v;
    sw_for_each<true>(f, list, sh, [&](uint32_t kk, uint32_t, uint32_t p, int q) {
      if (kk == v) atomicAdd(&th[slot(p, q) >> SW_TSH], 1u);
    });
    __syncthreads();
    const unsigned long long bw[2] = {0ull, 0ull};
    const unsigned long long bc[2] = {th[2 * SW_FT - 1 - 2 * tid], th[2 * SW_FT - 2 - 2 * tid]};
    unsigned long long tg, tw, tc;
    const SwPick pb = sw_pick<2, 2 * SW_FT>(bw, bc, true, SwFixed{take}, 0ull, 0ull, &tg, &tw, &tc, sh);
    const uint32_t blk = pb.d;
    const uint32_t rem = (uint32_t)(take - pb.ac);     // ties to take inside block blk, >= 1
    sw_for_each<true>(f, list, sh, [&](uint32_t kk, uint32_t, uint32_t p, int q) {
      if (kk == v) {
        const uint32_t j = slot(p, q);
        if ((j >> SW_TSH) == blk) atomicOr(&sh.tmask[(j & 127) >> 5], 1u << (j & 31));
      }
    });
    __syncthreads();
    if (tid == 0) {
      // the rem-th set bit from the top of the block's 128-bit tie mask, from registers:
      // whole words are skipped by their population counts, then the word's higher set
      // bits are cleared one at a time
      const uint32_t m[4] = {sh.tmask[0], sh.tmask[1], sh.tmask[2], sh.tmask[3]};
      uint32_t need = rem, pos = 0;
      for (int wd = 3; wd >= 0; --wd) {
        const uint32_t c = (uint32_t)__popc(m[wd]);
        if (need > c) {
          need -= c;
          continue;
        }
        uint32_t x = m[wd];
        for (uint32_t i = 1; i < need; ++i) x &= ~(0x80000000u >> __clz(x));
        pos = (uint32_t)(wd * 32 + 31 - __clz(x));
        break;
      }
      sh.tie_from = (blk << SW_TSH) + pos;
    }
    __syncthreads();
    tie_from = sh.tie_from;
  }
  if (tid == 0) {
    params[h] = make_uint4(f.v, tie_from, f.d1, 0u);
    k_out[h] = kf;
    if (sel_mass) sel_mass[h] = (float)((double)msel / (double)(1ull << 40));
  }
}

// One workgroup per (head, chunk): the chunk's words of the selection bitmap.
__global__ __launch_bounds__(SW_NT) void sw_bitmap_kernel(
    int S_max, int C, const unsigned long long* __restrict__ hp, const uint16_t* __restrict__ ho,
    const uint32_t* __restrict__ sorted, const uint4* __restrict__ params,
    uint32_t* __restrict__ sel_bits) {
  __shared__ uint32_t bits[SW_CH / 32];
  const int c = (int)blockIdx.x % C, h = (int)blockIdx.x / C, tid = threadIdx.x;
  if (tid < SW_CH / 32) bits[tid] = 0u;
  const uint4 p = params[h];
  const uint32_t v = p.x, tie_from = p.y, d1 = p.z;
  __syncthreads();
  if (v != SW_NONE) {
    const size_t at = ((size_t)h * C + c) * SW_B1 + d1;
    const uint32_t off = ho[at], end = off + (uint32_t)(hp[at] >> SW_CNT_SH);
    const uint32_t* srow = sorted + (size_t)h * S_max + (size_t)c * SW_CH;
    uint32_t q[SW_CH / SW_NT];
#pragma unroll
    for (int u = 0; u < SW_CH / SW_NT; ++u) {
      const uint32_t i = (uint32_t)(u * SW_NT + tid);
      q[u] = i < end ? srow[i] : 0u;
    }
#pragma unroll
    for (int u = 0; u < SW_CH / SW_NT; ++u) {
      const uint32_t i = (uint32_t)(u * SW_NT + tid);
      if (i < end) {
        const uint32_t local = q[u] & (SW_CH - 1);
        bool s = i < off;                                // a higher digit: selected
        if (!s) {
          const uint32_t kk = (d1 << SW_SH1) | (q[u] >> SW_CS);
          s = kk > v || (kk == v && (uint32_t)c * SW_CH + local >= tie_from);
        }
        if (s) atomicOr(&bits[local >> 5], 1u << (local & 31));
      }
    }
  }
  __syncthreads();
  if (tid < SW_CH / 32) {
    const int j0 = c * SW_CH + tid * 32;
    if (j0 < S_max) sel_bits[(size_t)h * (S_max / 32) + j0 / 32] = bits[tid];
  }
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

struct SwWs {
  size_t part, hp, ho, sorted, params, total;
};
SwWs sw_ws(int n_heads, int S_max) {
  const size_t H = (size_t)n_heads, C = (size_t)(S_max + SW_CH - 1) / SW_CH;
  SwWs w;
  w.part = 0;
  w.hp = w.part + al256(H * C * 2 * sizeof(float2));
  w.ho = w.hp + al256(H * C * SW_B1 * 8);
  w.sorted = w.ho + al256(H * C * SW_B1 * 2);
  w.params = w.sorted + al256(H * (size_t)S_max * 4);
  w.total = w.params + al256(H * sizeof(uint4));
  return w;
}

}  // namespace
}  // namespace hk

using namespace hk;

size_t hk_select_wide_ws(int n_heads, int S_max) { return sw_ws(n_heads, S_max).total; }

hipError_t hk_launch_select_wide(int n_heads, int S_max, const int32_t* cand_len,
                                 const uint16_t* mask, int n_metrics, const float* x0,
                                 const float* x1, const float* T0, const float* T1, float w0,
                                 float w1, const float* c_in, int p_q, int k_min, int k_max,
                                 float* c_out, float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                                 float* sel_mass, int32_t* status, void* ws, hipStream_t st) {
  const SwWs w = sw_ws(n_heads, S_max);
  char* base = static_cast<char*>(ws);
  float2* part = reinterpret_cast<float2*>(base + w.part);
  unsigned long long* hp = reinterpret_cast<unsigned long long*>(base + w.hp);
  uint16_t* ho = reinterpret_cast<uint16_t*>(base + w.ho);
  uint32_t* sorted = reinterpret_cast<uint32_t*>(base + w.sorted);
  uint4* params = reinterpret_cast<uint4*>(base + w.params);
  const int C = (S_max + SW_CH - 1) / SW_CH;
  const dim3 chunks(C * n_heads), block(SW_NT);
  TimedLaunch t(n_metrics > 0 ? HK_TK_CALIB_TOPP : HK_TK_TOPP, st);
  if (n_metrics > 0) {
    hipLaunchKernelGGL(sw_prep_kernel, chunks, block, 0, st, S_max, C, cand_len, mask, n_metrics,
                       x0, x1, T0, T1, part);
    hipLaunchKernelGGL(sw_chunk_kernel<true>, chunks, block, 0, st, S_max, C, cand_len, mask,
                       n_metrics, x0, x1, T0, T1, w0, w1, part, c_in, c_out, lse_out, hp, ho,
                       sorted, status);
  } else {
    hipLaunchKernelGGL(sw_chunk_kernel<false>, chunks, block, 0, st, S_max, C, cand_len, mask, 0,
                       x0, x1, T0, T1, w0, w1, part, c_in, c_out, lse_out, hp, ho, sorted, status);
  }
  allow_dynamic_lds<sw_finish_kernel>(SW_LDS);
  hipLaunchKernelGGL(sw_finish_kernel, dim3(n_heads), dim3(SW_FT), SW_LDS, st, S_max, C, hp, ho,
                     sorted, p_q, k_min, k_max, params, k_out, sel_mass);
  hipLaunchKernelGGL(sw_bitmap_kernel, chunks, block, 0, st, S_max, C, hp, ho, sorted, params,
                     sel_bits);
  return hipGetLastError();
}

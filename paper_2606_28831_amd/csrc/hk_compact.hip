// a4: Cascade-Cache rewrite into dense / sparse / condensed tiers (gfx950).
//
// Sec. 3.1 Step 3 and Sec. 3.3.1: the condensed band is rewritten (Rewrite Cache), the
// sparse band keeps its pages under a selection mask (Sparse Loading), the dense band is
// untouched.  Five stream-ordered kernels, all with static shapes:
//   plan    per head: tier sizes, per-page count of selected valid slots in the condensed
//           band and its exclusive prefix, kept sparse pages, pages to release;
//   alloc   one workgroup: head-order prefix sums of pages needed / released, bounds check
//           against the free list, pop of the needed ids (stack top moves down);
//   gather  one wave per condensed source page: every selected valid slot's K and V rows
//           go to their destination rank, 16-byte lanes, bit-exact;
//   table   per head: new row [condensed][sparse][dense], masks, n_pages, released ids;
//   push    released ids go back on the free list (after every pop has been consumed).
// When the free list is too short, alloc raises HK_FLAG_NOSPACE and the rest do nothing.
// Bands are age bands (dense / sparse / condensed by page position), or, under the hard
// budget (Sec. 3.1 Step 4), set per head by its state: all older pages condensed
// (rewrite), all sparse (sparse loading), or none (the row is kept).
#include "hk_internal.h"

namespace hk {

struct HeadPlan {
  int nc, ns, nd;      // tier sizes in pages (condensed, sparse, dense)
  int cnt_c;           // selected valid slots in the condensed band
  int npc;             // new condensed pages = ceil(cnt_c / 16)
  int nsk;             // sparse pages kept
  int n_free;          // pages released
  int pad;
};

struct CompactGlobals {
  int ok;              // 1: proceed
  int base;            // first popped index in free_ids
  int total_need;
  int total_free;
};

struct CompactWs {
  HeadPlan* plan;
  int* alloc_off;
  int* free_off;
  int* page_off;       // [n_heads][max_pages]
  int* freed;          // [n_heads * max_pages]
  CompactGlobals* g;
};

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline CompactWs carve(void* ws, int n_heads, int max_pages) {
  char* p = static_cast<char*>(ws);
  CompactWs w;
  w.plan = reinterpret_cast<HeadPlan*>(p);
  p += align256(sizeof(HeadPlan) * (size_t)n_heads);
  w.alloc_off = reinterpret_cast<int*>(p);
  p += align256(sizeof(int) * (size_t)n_heads);
  w.free_off = reinterpret_cast<int*>(p);
  p += align256(sizeof(int) * (size_t)n_heads);
  w.page_off = reinterpret_cast<int*>(p);
  p += align256(sizeof(int) * (size_t)n_heads * max_pages);
  w.freed = reinterpret_cast<int*>(p);
  p += align256(sizeof(int) * (size_t)n_heads * max_pages);
  w.g = reinterpret_cast<CompactGlobals*>(p);
  return w;
}

__device__ __forceinline__ uint32_t sel_word16(const uint32_t* srow, int pp) {
  return (srow[pp >> 1] >> ((pp & 1) * 16)) & 0xffffu;
}

// exclusive block scan of one int per thread (NT = 256); returns prefix, total via *tot
template <int NT>
__device__ __forceinline__ int block_exscan(int v, int* lds, int* tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) lds[wave] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const int t = lds[w];
    if (w < wave) before += t;
    all += t;
  }
  *tot = all;
  return before + x - v;
}

constexpr int CP_NT = 256;
constexpr int CP_PPT = 8;     // pages per thread in the plan's prefix (2048 pages per scan)

__global__ __launch_bounds__(CP_NT) void compact_plan_kernel(
    const int32_t* __restrict__ n_pages, const uint16_t* __restrict__ masks,
    const uint32_t* __restrict__ sel_bits, int max_pages, int L_dense, int L_sparse,
    const int32_t* __restrict__ head_mode, CompactWs w) {
  __shared__ int lds[CP_NT / 64];
  const int h = blockIdx.x;
  const int n = n_pages[h];
  int nd = min(n, dense_pages(L_dense));
  int ns = min(n - nd, L_sparse / HK_PAGE);
  if (head_mode) {
    // bands from the head's budget state: every older page condensed, every older page
    // sparse, or the whole row left in place (as if all dense)
    const int mode = head_mode[h];
    if (mode == HK_BUDGET_KEEP) {
      nd = n;
      ns = 0;
    } else {
      ns = (mode == HK_BUDGET_SPARSE) ? n - nd : 0;
    }
  }
  const int nc = n - nd - ns;
  const uint16_t* mrow = masks + (size_t)h * max_pages;
  const uint32_t* srow = sel_bits + (size_t)h * (max_pages / 2);
  int* off = w.page_off + (size_t)h * max_pages;
  // selected slots per condensed page and their exclusive prefix: each thread takes CP_PPT
  // consecutive pages (every load issued before any is used), one block scan per
  // CP_NT * CP_PPT pages
  int carry = 0;
  for (int base = 0; base < nc; base += CP_NT * CP_PPT) {
    const int p0 = base + (int)threadIdx.x * CP_PPT;
    uint32_t m[CP_PPT], sw[CP_PPT];
#pragma unroll
    for (int k = 0; k < CP_PPT; ++k) {
      const int pp = min(p0 + k, nc - 1);
      m[k] = mrow[pp];
      sw[k] = sel_word16(srow, pp);
    }
    int c[CP_PPT], mine = 0;
#pragma unroll
    for (int k = 0; k < CP_PPT; ++k) {
      c[k] = (p0 + k < nc) ? __popc(m[k] & sw[k]) : 0;
      mine += c[k];
    }
    int tot;
    int run = carry + block_exscan<CP_NT>(mine, lds, &tot);
#pragma unroll
    for (int k = 0; k < CP_PPT; ++k) {
      if (p0 + k < nc) off[p0 + k] = run;
      run += c[k];
    }
    carry += tot;
  }
  int kept = 0;
  for (int pp = nc + threadIdx.x; pp < nc + ns; pp += CP_NT)
    kept += (((uint32_t)mrow[pp] & sel_word16(srow, pp)) != 0u) ? 1 : 0;
  int tot;
  block_exscan<CP_NT>(kept, lds, &tot);
  if (threadIdx.x == 0) {
    HeadPlan p;
    p.nc = nc;
    p.ns = ns;
    p.nd = nd;
    p.cnt_c = carry;
    p.npc = (carry + HK_PAGE - 1) / HK_PAGE;
    p.nsk = tot;
    p.n_free = nc + (ns - tot);
    p.pad = 0;
    w.plan[h] = p;
  }
}

constexpr int AL_NT = 1024;

__global__ __launch_bounds__(AL_NT) void compact_alloc_kernel(int n_heads, const int32_t* free_top,
                                                              int32_t* status, CompactWs w) {
  __shared__ int lds[AL_NT / 64];
  const int per = (n_heads + AL_NT - 1) / AL_NT;
  const int h0 = threadIdx.x * per;
  int need = 0, fr = 0;
  for (int h = h0; h < min(h0 + per, n_heads); ++h) {
    need += w.plan[h].npc;
    fr += w.plan[h].n_free;
  }
  int tot_need, tot_free;
  int ex_need = block_exscan<AL_NT>(need, lds, &tot_need);
  int ex_free = block_exscan<AL_NT>(fr, lds, &tot_free);
  for (int h = h0; h < min(h0 + per, n_heads); ++h) {
    w.alloc_off[h] = ex_need;
    w.free_off[h] = ex_free;
    ex_need += w.plan[h].npc;
    ex_free += w.plan[h].n_free;
  }
  if (threadIdx.x == 0) {
    const int top = *free_top;
    CompactGlobals g;
    g.ok = (tot_need <= top) ? 1 : 0;
    g.base = top - tot_need;
    g.total_need = tot_need;
    g.total_free = tot_free;
    *w.g = g;
    if (!g.ok && status) atomicOr(status, HK_FLAG_NOSPACE);
  }
}

// Source rows are read once and rewritten rows are not read again by this step:
// nontemporal (streaming) loads and stores for both.
__device__ __forceinline__ uint4 load16(const char* p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}
__device__ __forceinline__ void store16(char* p, uint4 v) {
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), reinterpret_cast<u32x4*>(p));
}

// Source-driven gather: one wave per condensed source page, whose selected rows are
// packed densely onto lane groups (row k of the selection goes to group k % RPI), all
// loads issued before any store.  A selected slot of rank r (within the head's condensed
// band) lands in slot r % 16 of new page r / 16, so consecutive ranks fill pages in order.
template <int ROW_BYTES>
__global__ __launch_bounds__(256) void compact_gather_kernel(
    char* __restrict__ k_pool, char* __restrict__ v_pool, const int32_t* __restrict__ table,
    const uint16_t* __restrict__ masks, const uint32_t* __restrict__ sel_bits,
    const int32_t* __restrict__ free_ids, int max_pages, CompactWs w) {
  if (!w.g->ok) return;
  const int h = blockIdx.y;
  const int pp = blockIdx.x * 4 + (threadIdx.x >> 6);
  const HeadPlan p = w.plan[h];
  if (pp >= p.nc) return;
  const uint32_t m = (uint32_t)masks[(size_t)h * max_pages + pp] &
                     sel_word16(sel_bits + (size_t)h * (max_pages / 2), pp);
  if (m == 0u) return;
  const int lane = threadIdx.x & 63;
  constexpr int LPR = ROW_BYTES / 16;        // lanes per row
  constexpr int RPI = 64 / LPR;              // rows per instruction
  constexpr int NI = HK_PAGE / RPI;          // instructions per page
  const int sub = lane / LPR, chunk = lane % LPR;
  const size_t src_page = (size_t)table[(size_t)h * max_pages + pp];
  const int rank0 = w.page_off[(size_t)h * max_pages + pp];
  const int* popped = free_ids + w.g->base + w.alloc_off[h];
  const int nsel = __popc(m);
  uint4 kv[NI], vv[NI];
  int dst_slot[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int k = i * RPI + sub;             // k-th selected slot of the page
    dst_slot[i] = -1;
    if (k < nsel) {
      uint32_t mm = m;
      for (int j = 0; j < k; ++j) mm &= mm - 1u;
      const int t = __ffs(mm) - 1;
      const size_t src = (src_page * HK_PAGE + t) * ROW_BYTES + chunk * 16;
      kv[i] = load16(k_pool + src);
      vv[i] = load16(v_pool + src);
      dst_slot[i] = rank0 + k;
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int rank = dst_slot[i];
    if (rank >= 0) {
      const size_t dst = ((size_t)popped[rank >> 4] * HK_PAGE + (rank & 15)) * ROW_BYTES + chunk * 16;
      store16(k_pool + dst, kv[i]);
      store16(v_pool + dst, vv[i]);
    }
  }
}

__global__ __launch_bounds__(CP_NT) void compact_table_kernel(
    int32_t* __restrict__ table, uint16_t* __restrict__ masks, int32_t* __restrict__ n_pages,
    const uint32_t* __restrict__ sel_bits, const int32_t* __restrict__ free_ids, int max_pages,
    CompactWs w) {
  extern __shared__ __align__(16) char smem[];
  __shared__ int lds[CP_NT / 64];
  if (!w.g->ok) return;
  const int h = blockIdx.x;
  const HeadPlan p = w.plan[h];
  const int n = p.nc + p.ns + p.nd;
  int32_t* trow = table + (size_t)h * max_pages;
  uint16_t* mrow = masks + (size_t)h * max_pages;
  const uint32_t* srow = sel_bits + (size_t)h * (max_pages / 2);
  int32_t* old_id = reinterpret_cast<int32_t*>(smem);
  uint16_t* old_m = reinterpret_cast<uint16_t*>(old_id + max_pages);
  // the old row staged in LDS, CP_PPT pages per thread per pass, loads issued first
  for (int b0 = 0; b0 < n; b0 += CP_NT * CP_PPT) {
    int32_t id[CP_PPT];
    uint16_t mk[CP_PPT];
#pragma unroll
    for (int k = 0; k < CP_PPT; ++k) {
      const int pp = min(b0 + k * CP_NT + (int)threadIdx.x, n - 1);
      id[k] = trow[pp];
      mk[k] = mrow[pp];
    }
#pragma unroll
    for (int k = 0; k < CP_PPT; ++k) {
      const int pp = b0 + k * CP_NT + (int)threadIdx.x;
      if (pp < n) {
        old_id[pp] = id[k];
        old_m[pp] = mk[k];
      }
    }
  }
  __syncthreads();
  const int* popped = free_ids + w.g->base + w.alloc_off[h];
  int* freed = w.freed + w.free_off[h];
  // condensed: fresh pages, full but the last
  const int last = p.cnt_c & 15;
  for (int i = threadIdx.x; i < p.npc; i += CP_NT) {
    trow[i] = popped[i];
    mrow[i] = (i == p.npc - 1 && last) ? (uint16_t)((1u << last) - 1u) : (uint16_t)0xffffu;
  }
  // old condensed pages are released
  for (int pp = threadIdx.x; pp < p.nc; pp += CP_NT) freed[pp] = old_id[pp];
  // sparse: keep in order under the selection mask, release emptied pages
  int kept_before = 0, drop_before = 0;
  for (int base = 0; base < p.ns; base += CP_NT) {
    const int pp = p.nc + base + threadIdx.x;
    uint32_t m2 = 0;
    if (base + (int)threadIdx.x < p.ns) m2 = (uint32_t)old_m[pp] & sel_word16(srow, pp);
    const int keep = (base + (int)threadIdx.x < p.ns && m2) ? 1 : 0;
    const int drop = (base + (int)threadIdx.x < p.ns && !m2) ? 1 : 0;
    int tk, td;
    const int ek = block_exscan<CP_NT>(keep, lds, &tk);
    const int ed = block_exscan<CP_NT>(drop, lds, &td);
    if (keep) {
      trow[p.npc + kept_before + ek] = old_id[pp];
      mrow[p.npc + kept_before + ek] = (uint16_t)m2;
    }
    if (drop) freed[p.nc + drop_before + ed] = old_id[pp];
    kept_before += tk;
    drop_before += td;
  }
  // dense: shifted down, unchanged
  const int dst0 = p.npc + p.nsk, src0 = p.nc + p.ns;
  for (int i = threadIdx.x; i < p.nd; i += CP_NT) {
    trow[dst0 + i] = old_id[src0 + i];
    mrow[dst0 + i] = old_m[src0 + i];
  }
  const int n_new = p.npc + p.nsk + p.nd;
  for (int i = n_new + threadIdx.x; i < n; i += CP_NT) {
    trow[i] = -1;
    mrow[i] = 0;
  }
  if (threadIdx.x == 0) n_pages[h] = n_new;
}

__global__ __launch_bounds__(256) void compact_push_kernel(int32_t* __restrict__ free_ids,
                                                           int32_t* __restrict__ free_top, CompactWs w) {
  const CompactGlobals g = *w.g;
  if (!g.ok) return;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < g.total_free; i += gridDim.x * blockDim.x)
    free_ids[g.base + i] = w.freed[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) *free_top = g.base + g.total_free;
}

// Fresh allocator: free_ids[i] = first_free + i for the n free pages, top = n.
__global__ __launch_bounds__(256) void alloc_init_kernel(int32_t* __restrict__ free_ids,
                                                        int32_t* __restrict__ free_top, int first_free,
                                                        int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    free_ids[i] = first_free + i;
  if (blockIdx.x == 0 && threadIdx.x == 0) *free_top = n;
}

}  // namespace hk

using namespace hk;

hipError_t hk_launch_alloc_init(int32_t* free_ids, int32_t* free_top, int first_free, int n,
                                hipStream_t st) {
  const int blocks = max(1, min((n + 255) / 256, 1024));
  hipLaunchKernelGGL(alloc_init_kernel, dim3(blocks), dim3(256), 0, st, free_ids, free_top, first_free, n);
  return hipGetLastError();
}

size_t hk_compact_ws(int n_heads, int max_pages) {
  return align256(sizeof(HeadPlan) * (size_t)n_heads) + 2 * align256(sizeof(int) * (size_t)n_heads) +
         2 * align256(sizeof(int) * (size_t)n_heads * max_pages) + align256(sizeof(CompactGlobals));
}

hipError_t hk_launch_compact(int n_heads, int D, const hk_paged_kv* kv, const uint32_t* sel_bits,
                             int L_dense, int L_sparse, const int32_t* head_mode,
                             const hk_allocator* alloc, int32_t* status, void* ws, hipStream_t st) {
  const CompactWs w = carve(ws, n_heads, kv->max_pages);
  const int mp = kv->max_pages;
  {
    TimedLaunch t(HK_TK_COMPACT_META, st);
    hipLaunchKernelGGL(compact_plan_kernel, dim3(n_heads), dim3(CP_NT), 0, st, kv->n_pages,
                       kv->page_mask, sel_bits, mp, L_dense, L_sparse, head_mode, w);
  }
  {
    TimedLaunch t(HK_TK_COMPACT_META, st);
    hipLaunchKernelGGL(compact_alloc_kernel, dim3(1), dim3(AL_NT), 0, st, n_heads, alloc->free_top,
                       status, w);
  }
  const int row_bytes = D * (kv->dtype == HK_BF16 ? 2 : 4);
  dim3 gg((mp + 3) / 4, n_heads);
  char* kp = static_cast<char*>(kv->k_pool);
  char* vp = static_cast<char*>(kv->v_pool);
  {
  TimedLaunch t(HK_TK_COMPACT_GATHER, st);
  switch (row_bytes) {
    case 128: hipLaunchKernelGGL((compact_gather_kernel<128>), gg, dim3(256), 0, st, kp, vp, kv->page_table, kv->page_mask, sel_bits, alloc->free_ids, mp, w); break;
    case 256: hipLaunchKernelGGL((compact_gather_kernel<256>), gg, dim3(256), 0, st, kp, vp, kv->page_table, kv->page_mask, sel_bits, alloc->free_ids, mp, w); break;
    default: hipLaunchKernelGGL((compact_gather_kernel<512>), gg, dim3(256), 0, st, kp, vp, kv->page_table, kv->page_mask, sel_bits, alloc->free_ids, mp, w); break;
  }
  }
  const size_t lds = (size_t)mp * (sizeof(int32_t) + sizeof(uint16_t));
  allow_dynamic_lds<compact_table_kernel>(lds);
  {
    TimedLaunch t(HK_TK_COMPACT_META, st);
    hipLaunchKernelGGL(compact_table_kernel, dim3(n_heads), dim3(CP_NT), lds, st, kv->page_table,
                       kv->page_mask, kv->n_pages, sel_bits, alloc->free_ids, mp, w);
  }
  {
    TimedLaunch t(HK_TK_COMPACT_META, st);
    hipLaunchKernelGGL(compact_push_kernel, dim3(256), dim3(256), 0, st, alloc->free_ids,
                       alloc->free_top, w);
  }
  return hipGetLastError();
}

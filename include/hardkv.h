/*
 * hardkv.h -- C ABI of the Hard-KV decoding-time KV-compression step on MI355X (gfx950).
 *
 * Paper: "Hard-KV: Head-Adaptive Regularization for Decoding-time KV Compression".
 * The step (Sec. 3.1, continuous compression pipeline, Steps 1-3) is
 *   hk_score          importance of every cached key against an observation window
 *   hk_calibrate      Logits Calibration into one probability space (Sec. 3.2, Solution 2)
 *   hk_calibrate_solve_T  per-head temperature for Problem 1 (App. D.1, binary search)
 *   hk_calibrate_solve_T_gd  the same temperature by gradient descent (Alg. 1)
 *   hk_topp_select    head-adaptive Top-p budget (Sec. 3.2, Problem 1)
 *   hk_calibrate_topp hk_calibrate followed by hk_topp_select in one launch
 *   hk_topp_select_ws / hk_calibrate_topp_ws  the same with each head spread over many
 *                     workgroups (long caches, small batches)
 *   hk_compress       score -> calibrate + Top-p -> compact in one call
 *   hk_pool_max       order-preserving max-pooling of scores before calibration
 *                     (Sec. 3.2 Solution 1, SnapKV form)
 *   hk_compact        Cascade-Cache rewrite into dense / sparse / condensed tiers
 *                     (Sec. 3.1 Step 3; Sec. 3.3.1 Rewrite Cache and Sparse Loading)
 *   hk_decode_attn    paged decode attention over the variable-budget cache with the
 *                     attention-state merge (App. F)
 *   hk_append_kv      append-only dense-tier write of one decode step (Sec. 3.1 Step 1)
 *   hk_alloc_init     a fresh device page allocator
 * Step 4 (Sec. 3.1, hard budget; Sec. 3.3.1 budget thresholds L_lower / L_upper):
 *   hk_score_rows     each window row's own attention probabilities over the candidates
 *   hk_vote_topp      Cautious Update: every row's own Top-p set, counted as votes
 *   hk_budget_plan    per-head budget state (keep / sparse loading / rewrite) and cap
 *   hk_budget_select  selection under the cap, ranked by votes, with attention sinks
 *   hk_compact_modes  hk_compact driven by the per-head budget state
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  The library never
 *     allocates, frees or synchronises; it only enqueues kernels on `stream`.
 *   - Scratch memory is a caller-provided device `workspace` of at least
 *     hk_workspace_size(op, ...) bytes, 256-byte aligned.
 *   - Shapes are static: no entry point changes a tensor's size; counts that change
 *     (pages per head, free-list top) live in device memory and are updated in place.
 *   - The return value reports argument validation and launch errors synchronously.
 *     Conditions found while running (page pool exhausted, NaN inputs) are OR-ed as
 *     HK_FLAG_* bits into a caller-provided device int32 `status` word, which the
 *     caller clears and reads after its own synchronisation.
 *   - Calls on one stream run in order; calls that touch the same cache from
 *     different streams without ordering race.
 *
 * Paged Cascade Cache (head-flattened block table, Sec. 3.3.2 P2; App. B.1):
 *   one "head" = (sequence, KV head); with NS sequences and Hkv KV heads there are
 *   n_heads = NS * Hkv rows.  Logical slot j of head h lives in physical page
 *   page_table[h][j / 16], slot j % 16, and is valid when bit (j % 16) of
 *   page_mask[h][j / 16] is set.  Pages are ordered oldest first; rows hold
 *   n_pages[h] pages and -1 past them.  S_max = 16 * max_pages logical slots per head.
 *   Page contents: k_pool / v_pool [num_pages][16][D] in `dtype`.
 *
 * Window queries (observation window of the W most recent queries) are window-major:
 *   q_obs[W][NS][Hq][D].  Query head g belongs to KV head g / G, G = Hq / Hkv.
 *   The R = G * W rows of a KV head are its G query heads at every window position.
 */
#ifndef HARDKV_H_
#define HARDKV_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
typedef int32_t hk_status;
enum {
  HK_OK = 0,
  HK_ERR_ARG = 1,        /* null pointer, non-positive size, scalar out of range      */
  HK_ERR_DTYPE = 2,      /* dtype is not HK_F32 or HK_BF16                             */
  HK_ERR_SHAPE = 3,      /* unsupported shape: D not 64/128, Hq % Hkv != 0,
                            G*W > 256, S_max > 32768, ...                              */
  HK_ERR_ALIGN = 4,      /* a pointer is not 16-byte aligned (256 for workspace)       */
  HK_ERR_WORKSPACE = 5,  /* workspace smaller than hk_workspace_size()                 */
  HK_ERR_HIP = 6,        /* a kernel launch failed                                     */
  HK_ERR_SCRATCH = 7     /* hk_decode_attn_noalloc: more than its static scratch       */
};
/* bits OR-ed into the device status word */
enum {
  HK_FLAG_NOSPACE = 1,   /* hk_compact / hk_append_kv: free list too short; cache left unchanged */
  HK_FLAG_NAN = 2,       /* a NaN probability was met and given weight 0               */
  HK_FLAG_RANGE = 4      /* a probability outside [0,1] was clamped                    */
};

typedef enum { HK_F32 = 0, HK_BF16 = 1 } hk_dtype;

/* One paged Cascade Cache (any number of heads; layers may share one pool). */
typedef struct {
  void* k_pool;          /* [num_pages][16][D]                                          */
  void* v_pool;          /* [num_pages][16][D]                                          */
  int32_t* page_table;   /* [n_heads][max_pages] physical ids, -1 past n_pages          */
  uint16_t* page_mask;   /* [n_heads][max_pages] bit t = slot t valid                   */
  int32_t* n_pages;      /* [n_heads] pages in use                                      */
  int32_t num_pages;     /* pool capacity (pages)                                       */
  int32_t max_pages;     /* table width                                                 */
  hk_dtype dtype;
} hk_paged_kv;

/* Device page allocator: a stack of free page ids. */
typedef struct {
  int32_t* free_ids;     /* [capacity] device; entries [0, *free_top) are free          */
  int32_t* free_top;     /* device int32                                                */
  int32_t capacity;
} hk_allocator;

typedef struct {
  int32_t NS;            /* sequences in this call (batch x layers)                     */
  int32_t Hq;            /* query heads per sequence                                    */
  int32_t Hkv;           /* KV heads per sequence                                       */
  int32_t D;             /* head dimension: 64 or 128                                   */
  int32_t W;             /* observation-window length                                   */
} hk_dims;

enum { HK_OP_SCORE = 0, HK_OP_COMPACT = 1, HK_OP_DECODE = 2, HK_OP_APPEND = 3, HK_OP_COMPRESS = 4,
       HK_OP_SELECT = 5 };

/* Bytes of workspace entry point `op` needs for these dims and table width (HK_OP_SELECT:
 * hk_select_workspace_size(dims->NS * dims->Hkv, 16 * max_pages)). */
size_t hk_workspace_size(int32_t op, const hk_dims* dims, int32_t max_pages);

/* Name of a hk_status code (flags = 0) or of a single HK_FLAG_* bit (flags = 1). */
const char* hk_status_string(int32_t code, int32_t flags);

/* ------------------------------------------------------------------ a1: score
 * Importance of every candidate slot of every KV head against its observation window
 * (Reduce step of the three-step selection framework, App. E, applied to the raw
 * attention distribution S of Problem 1, Sec. 3.2; Vanilla/H2O-style attention mass,
 * Sec. 4 baseline adaptations):
 *   z[r][j]  = sm_scale * <q_r, k_j>                     (App. F standard attention)
 *   LSE_r    = log sum_{j valid} exp z[r][j]             computed here, or row_lse_in
 *   s[h][j]  = log( (1/R) sum_r exp(z[r][j] - LSE_r) )   for candidate slots j
 *            = -inf for every other slot
 * Candidates of head h are valid slots older than the dense tier: j < cand_len[h] with
 * cand_len[h] = 16 * max(0, n_pages[h] - ceil(L_dense / 16)).
 * Optional redundancy metric (R-KV style pairwise key similarity as a logit-level
 * transform, Sec. 4; Solution 2 form): with n_ref reference slots ref_slots[h][0..n_ref)
 * (valid logical slots of head h),
 *   x_red[h][j] = -max_{i in ref, i != j} cos(k_i, k_j)  for candidates (-inf elsewhere);
 *   a zero-norm key has cosine 0; an empty reference set gives +1.
 * Arguments
 *   q_obs        [W][NS][Hq][D] in kv->dtype
 *   row_lse_in   [W][NS][Hq] fp32 or NULL (then computed: two passes over K)
 *   row_lse_out  [W][NS][Hq] fp32 or NULL
 *   s_attn       [n_heads][S_max] fp32 (written in full), or NULL to compute only the row
 *                LSEs and cand_len_out (pass 1; row_lse_in must then be NULL, row_lse_out
 *                given and x_red NULL)
 *   cand_len_out [n_heads] int32
 *   ref_slots    [n_heads][n_ref] int32 or NULL; n_ref in [0, 256]; x_red likewise
 * Errors: HK_ERR_SHAPE unless D in {64,128}, Hq % Hkv == 0 and G*W <= 256.
 */
hk_status hk_score(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv,
                   int32_t L_dense, float sm_scale, const float* row_lse_in,
                   float* row_lse_out, float* s_attn, int32_t* cand_len_out,
                   const int32_t* ref_slots, int32_t n_ref, float* x_red,
                   void* workspace, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ a2: calibrate
 * Logits Calibration, Solution 2 (Sec. 3.2): each metric m is mapped to a distribution
 * over the candidates of head h,
 *   c_m[j] = exp(x_m[j] / T_m[h] - lse_m[h]),  lse_m[h] = log sum_{cand} exp(x_m / T_m[h]),
 * and the output is the mixture c = sum_m w_m c_m (0 outside candidates).
 * Candidates: j < cand_len[h] and (page_mask == NULL or bit j%16 of page_mask[h][j/16]).
 * Arguments
 *   x[m]    host array of n_metrics device pointers, each [n_heads][S_max] fp32
 *   T[m]    host array of n_metrics device pointers to [n_heads] fp32, or T == NULL /
 *           T[m] == NULL for T = 1; every T must be > 0
 *   w       host array of n_metrics mixture weights
 *   c_out   [n_heads][S_max] fp32;  lse_out [n_heads][n_metrics] fp32 or NULL
 * n_metrics in [1, 2].  All -inf candidates give c = 0 and lse = -inf.
 */
hk_status hk_calibrate(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                       const uint16_t* page_mask, int32_t n_metrics,
                       const float* const* x, const float* const* T, const float* w,
                       float* c_out, float* lse_out, hipStream_t stream);

/* ------------------------------------------------------------------ a3: Top-p
 * Head-adaptive Top-p budget (Sec. 3.2, Problem 1): per head, the smallest prefix of the
 * candidates ordered by c descending -- ties to the larger slot index, i.e. the more
 * recent token -- whose mass reaches p.  Fixed-point rule (exact, order-free):
 *   w_j = floor(c_j * 2^40), Total = sum w, p_q = round(p * 1e6),
 *   target = ceil(p_q * Total / 1e6), k = min{k : mass of the first k >= target}
 *   (k = 0 if target = 0), then clamped to [min(k_min, n_cand), min(k_max, n_cand)]
 *   (k_max <= 0: no cap).  NaN c counts as 0 (HK_FLAG_NAN); c outside [0,1] is clamped
 *   (HK_FLAG_RANGE).
 * Outputs
 *   sel_bits [n_heads][S_max/32] uint32, bit j%32 of word j/32 = slot j selected
 *   k_out    [n_heads] int32
 *   sel_mass_out [n_heads] fp32 = (mass of the selected set) / 2^40, or NULL
 * p in [0, 1].  S_max must be a multiple of 32 and at most 32768.
 */
hk_status hk_topp_select(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                         const uint16_t* page_mask, const float* c, double p,
                         int32_t k_min, int32_t k_max, uint32_t* sel_bits, int32_t* k_out,
                         float* sel_mass_out, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------ a2 + a3 fused
 * hk_calibrate followed by hk_topp_select on its output, in one launch: the calibrated
 * values stay on chip, and c_out, lse_out, sel_bits, k_out and sel_mass_out receive
 * exactly what the two separate calls would write (same arithmetic, bit for bit).
 * c_out and lse_out may be NULL (then nothing is written there); sel_mass_out and status
 * may be NULL.  Arguments and limits as for hk_calibrate and hk_topp_select.
 */
hk_status hk_calibrate_topp(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                            const uint16_t* page_mask, int32_t n_metrics,
                            const float* const* x, const float* const* T, const float* w,
                            double p, int32_t k_min, int32_t k_max, float* c_out,
                            float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                            float* sel_mass_out, int32_t* status, hipStream_t stream);

/* ------------------------------------------------------------------ a2 + a3, wide
 * hk_topp_select and hk_calibrate_topp with every head spread over ceil(S_max / 4096)
 * workgroups (Sec. 3.2, Problem 1 and Solution 2): for caches longer than 32768 slots, and
 * so that a batch of few heads still fills the chip.  The Top-p rule is the one stated for
 * hk_topp_select, in the same exact integers, so for the same c the selection, k_out and
 * sel_mass_out are those hk_topp_select writes, bit for bit.  hk_calibrate_topp_ws
 * assembles each head's log-sum-exp from 4096-slot pieces: its c_out and lse_out agree
 * with hk_calibrate's to fp32 rounding, and its selection is the exact Top-p of the c it
 * computed (which it writes to c_out when given).
 * Arguments as for hk_topp_select / hk_calibrate_topp, plus
 *   workspace  device, 256-byte aligned, >= hk_select_workspace_size(n_heads, S_max)
 *              bytes, used for the calibration pieces, the per-head histograms and
 *              counters and each slot's key; overwritten by every call (calls that overlap
 *              on one workspace race).
 * S_max must be a multiple of 32 and at most 262144; x[m], c and c_out must be 16-byte
 * aligned (HK_ERR_ALIGN).  HK_ERR_WORKSPACE for a workspace that is too small, HK_ERR_ALIGN
 * for one not 256-byte aligned.
 */
size_t hk_select_workspace_size(int32_t n_heads, int32_t S_max);
hk_status hk_topp_select_ws(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                            const uint16_t* page_mask, const float* c, double p, int32_t k_min,
                            int32_t k_max, uint32_t* sel_bits, int32_t* k_out,
                            float* sel_mass_out, int32_t* status, void* workspace,
                            size_t ws_bytes, hipStream_t stream);
hk_status hk_calibrate_topp_ws(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                               const uint16_t* page_mask, int32_t n_metrics,
                               const float* const* x, const float* const* T, const float* w,
                               double p, int32_t k_min, int32_t k_max, float* c_out,
                               float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                               float* sel_mass_out, int32_t* status, void* workspace,
                               size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ a2 pooling
 * Order-preserving transform g of Solution 1 (Sec. 3.2, S_hat = S(g(z / T))) in the
 * SnapKV form used by the paper's baselines: for every candidate j of head h,
 *   x_out[h][j] = max { x[h][i] : i candidate, |i - j| <= radius },
 * and x_out = -inf at non-candidates (candidates as for hk_calibrate).  Max commutes with
 * the logarithm, so pooling log scores pools the underlying masses.  x, x_out
 * [n_heads][S_max] fp32 device arrays, distinct (no in-place); radius in [0, 64]
 * (radius 0 copies the candidates).  HK_ERR_ARG for a null or aliased pointer,
 * HK_ERR_SHAPE for a radius outside [0, 64] or an S_max that is not a multiple of 32 or
 * exceeds 262144 (the wide selector's limit: one workgroup per 1024-slot tile, so the
 * length is not bound by a workgroup).
 */
hk_status hk_pool_max(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                      const uint16_t* page_mask, const float* x, int32_t radius, float* x_out,
                      hipStream_t stream);

/* ------------------------------------------------------------------ a2': temperature
 * Temperature of Problem 1 (Sec. 3.2) by bisection (App. D.1, binary search on T):
 *   f(T) = M_k(Softmax(x / T)) - target_mass[h], M_k = mass of the Top-k set of x
 *   (order c desc, ties to the larger slot; invariant in T, App. D.2 theorem).
 *   Search on log T in [T_lo, T_hi] for `iters` halvings: f(T_mid) > 0 raises the lower
 *   end, otherwise the upper end comes down; T_out = exp(midpoint of the final bracket).
 * Arguments: x [n_heads][S_max] fp32; k [n_heads] int32 (the Top-p count of the target
 * distribution); target_mass [n_heads] fp32; T_out [n_heads] fp32.
 * 0 < T_lo < T_hi; iters in [1, 64]; S_max a multiple of 32, at most 262144 (rows longer
 * than 32768 slots are streamed from memory in each sweep instead of held in registers).
 */
hk_status hk_calibrate_solve_T(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                               const uint16_t* page_mask, const float* x, const int32_t* k,
                               const float* target_mass, float T_lo, float T_hi,
                               int32_t iters, float* T_out, hipStream_t stream);

/* Temperature of Problem 1 by gradient descent (Alg. 1, Solution 2 form): theta = log T
 * starts at log(T_init) and takes Adam steps (beta1 0.9, beta2 0.999, eps 1e-8,
 * bias-corrected, no weight decay, step size lr) on the loss
 *   l(theta) = (M_k(Softmax(x / T)) - target_mass[h])^2,
 * the Top-k set being that of x (invariant in T, App. D.2 theorem; ties to the larger
 * slot), with the exact derivative dM/dtheta = -(1/T) M (E_top[x] - E_all[x]); it stops
 * when l < tol or after `iters` steps.  T_out [n_heads] fp32; loss_out [n_heads] fp32 (the
 * loss at the returned T) or NULL.  Other arguments as for hk_calibrate_solve_T.
 * T_init > 0, lr > 0, iters in [0, 100000], tol >= 0.
 */
hk_status hk_calibrate_solve_T_gd(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                                  const uint16_t* page_mask, const float* x, const int32_t* k,
                                  const float* target_mass, float T_init, float lr, int32_t iters,
                                  float tol, float* T_out, float* loss_out, hipStream_t stream);

/* ------------------------------------------------------------------ the whole step
 * One compression step (Sec. 3.1 Steps 2-3) in one call: hk_score (attention mass; row
 * LSEs computed, or taken from row_lse_in) -> hk_calibrate_topp_ws (one metric, T = 1;
 * the calibrated probabilities are not written out) -> hk_compact, on `stream`, in that
 * order.  The
 * scores, candidate counts, row LSEs and every stage's scratch live in `workspace`
 * (>= hk_workspace_size(HK_OP_COMPRESS, dims, max_pages) bytes, 256-byte aligned).
 * Outputs: k_out [n_heads] (the Top-p counts), sel_bits_out [n_heads][S_max/32] or NULL
 * (the selection is then kept in the workspace), status (HK_FLAG_* of every stage).
 * Arguments and errors as for the three calls it makes; alloc->capacity >= kv->num_pages,
 * S_max = 16 * max_pages <= 262144 and at most 2^20 heads are checked before anything is
 * launched (HK_ERR_ARG, HK_ERR_SHAPE).
 */
hk_status hk_compress(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv,
                      int32_t L_dense, int32_t L_sparse, float sm_scale, const float* row_lse_in,
                      double p, int32_t k_min, int32_t k_max, const hk_allocator* alloc,
                      uint32_t* sel_bits_out, int32_t* k_out, int32_t* status, void* workspace,
                      size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ a4: compact
 * Cascade-Cache rewrite (Sec. 3.1 Step 3; Sec. 3.3.1).  Per head, page positions are
 * split into age bands: dense = the newest ceil(L_dense/16) pages, sparse = the
 * floor(L_sparse/16) pages before them, condensed = all older pages.
 *   condensed: every selected valid slot is copied (K and V rows, bit-exact), in
 *              ascending logical order, into freshly popped pages filled 16 at a time
 *              (all full except the last) -- Rewrite Cache; the old pages are pushed back;
 *   sparse:    pages stay in place with mask &= selection -- Sparse Loading; a page left
 *              empty is pushed back;
 *   dense:     untouched.
 * The new row is [condensed][sparse][dense], still oldest first; n_pages is updated.
 * Page ids are popped in head order before any is pushed, so the rewrite is out of place
 * and deterministic.  If the free list is too short, HK_FLAG_NOSPACE is raised and the
 * cache is left exactly as it was.
 * alloc->capacity must be at least kv->num_pages (HK_ERR_ARG otherwise): the pages the
 * rewrite frees are pushed onto the stack, which can then list every page of the pool.
 */
hk_status hk_compact(const hk_dims* dims, const hk_paged_kv* kv, const uint32_t* sel_bits,
                     int32_t L_dense, int32_t L_sparse, const hk_allocator* alloc,
                     int32_t* status, void* workspace, size_t ws_bytes, hipStream_t stream);

/* Fresh device page allocator (the free-page stack the rewrite and the append pop from,
 * Sec. 3.3.2 metadata management): pages [first_free, num_pages) become free, listed in
 * ascending order (free_ids[i] = first_free + i), and *free_top = num_pages - first_free;
 * pages below first_free are taken (e.g. by the prompt).  Entries of free_ids past the
 * top are not written.  HK_ERR_ARG unless 0 <= first_free <= num_pages and
 * num_pages - first_free <= alloc->capacity.  (A stack that hk_compact,
 * hk_compact_modes or hk_compress push onto needs capacity >= the pool's page count.)
 */
hk_status hk_alloc_init(const hk_allocator* alloc, int32_t first_free, int32_t num_pages,
                        hipStream_t stream);

/* ------------------------------------------------------------------ a5: decode
 * One decode step of attention for every query head over its KV head's valid slots
 * (App. F):  o = sum_j Softmax_j(sm_scale q.k_j) v_j,  lse = log sum_j exp(sm_scale q.k_j).
 * Split-K partial states over page ranges are combined with the merge operator of App. F.
 * q [NS][Hq][D] in kv->dtype; o [NS][Hq][D] fp32; lse [NS][Hq] fp32 (may point into a
 * window ring).  A head with no valid slot gives o = 0, lse = -inf.
 */
hk_status hk_decode_attn(const hk_dims* dims, const void* q, const hk_paged_kv* kv,
                         float sm_scale, float* o, float* lse, void* workspace,
                         size_t ws_bytes, hipStream_t stream);

/* hk_decode_attn for callers that cannot allocate or pass a workspace: code recorded under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.  Same arguments
 * (minus the workspace), kernels and results as hk_decode_attn, bit for bit.  The split
 * partial states go to a static device array of the library (16 MiB, one per GPU the library
 * runs on, held until the process ends); the call allocates nothing.  Limit: the call needs
 * hk_decode_noalloc_scratch_bytes(dims, kv->max_pages) bytes of it =
 * NS * Hkv * n_split * (Hq / Hkv) * (D + 2) * 4 with n_split from hk_decode_plan (about
 * 6.4 MB for 64 sequences x 8 KV heads, G 4, D 128, a 768-page table); a larger call returns
 * HK_ERR_SCRATCH without launching.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (different streams, or different host threads without ordering)
 * race, and the array keeps the last call's contents.  Other errors as for hk_decode_attn.
 */
hk_status hk_decode_attn_noalloc(const hk_dims* dims, const void* q, const hk_paged_kv* kv,
                                 float sm_scale, float* o, float* lse, hipStream_t stream);
size_t hk_decode_noalloc_scratch_bytes(const hk_dims* dims, int32_t max_pages);

/* The split hk_decode_attn uses for these dims and table width (host only, no launch):
 * every head's pages are shared by *n_split workgroups, none of which walks more than
 * *pages_per_split pages (a full-width row is split into ranges of that many pages;
 * shorter rows are spread over the same number of splits, at least 16 pages each).
 * Larger head counts take longer splits (up to 128 pages) so that one launch offers the
 * chip about 2048 workgroups.  HK_ERR_ARG for null outputs or max_pages <= 0; dims as for
 * hk_decode_attn.
 */
hk_status hk_decode_plan(const hk_dims* dims, int32_t max_pages, int32_t* n_split,
                         int32_t* pages_per_split);

/* ------------------------------------------------------------------ a6: append
 * Append-only write of one decode step's K and V into the dense tier (Sec. 3.1 Step 1):
 * for each head the new token goes one past the highest valid slot of its newest page,
 * or into slot 0 of a page popped from the allocator when that page is full (or the
 * row is empty).  k_new, v_new [NS][Hkv][D] in kv->dtype.  Pops happen in head order.
 * If the free list is too short or a row is full (n_pages == max_pages) the step is
 * skipped for every head and HK_FLAG_NOSPACE is raised.
 * workspace: device, 256-B aligned, >= hk_workspace_size(HK_OP_APPEND) bytes (a few int32
 * per 64 heads), caller-owned, overwritten by the call.
 */
hk_status hk_append_kv(const hk_dims* dims, const hk_paged_kv* kv, const void* k_new,
                       const void* v_new, const hk_allocator* alloc, int32_t* status,
                       void* workspace, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ Step 4: hard budget
 * The hard budget of the continuous compression pipeline (Sec. 3.1 Step 4 and the Condensed
 * tier; Sec. 3.3.1 budget thresholds): a head whose memory exceeds L_upper is rewritten under
 * a capped selection, one whose valid slots exceed L_lower is thinned by sparse loading, any
 * other head is kept.  The Cautious Update strategy (Sec. 3.1) replaces the window's mean
 * attention by votes: every window query keeps its own selection, and under a strict budget
 * the candidates are ranked by their votes.
 */
enum { HK_BUDGET_KEEP = 0, HK_BUDGET_SPARSE = 1, HK_BUDGET_REWRITE = 2 };

/* Per-row attention probabilities of the R = G * W window rows of every head:
 *   a_rows[h][r][j] = exp(z[r][j] - LSE_r)   for candidate slots j (as in hk_score),
 *                   = 0                       for every other j < S_max,
 * z and the row order r = w * G + g as in hk_score; row_lse [W][NS][Hq] fp32 holds LSE_r
 * (hk_score's row_lse_out, or the decode step's LSEs).  a_rows [n_heads][R][S_max] fp32,
 * written in full: n_heads * R * S_max * 4 bytes.  Errors as for hk_score.
 */
hk_status hk_score_rows(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv,
                        int32_t L_dense, float sm_scale, const float* row_lse, float* a_rows,
                        hipStream_t stream);

/* Cautious Update votes (Sec. 3.1): row r of head h selects its own head-adaptive Top-p set
 * of the candidates under a_rows[h][r] -- the rule of hk_topp_select with k_min = 1 and no
 * cap, same fixed-point mass, tie order, NaN and range handling -- and
 *   votes[h][j] = number of rows r whose set holds j   (uint16, <= R).
 * The cumulative selection mask of the strategy is votes >= 1.
 * Arguments
 *   a_rows   [n_heads][R][S_max] fp32 (e.g. from hk_score_rows)
 *   votes    [n_heads][S_max] uint16, 16-byte aligned
 *   row_sel  [n_heads][R][S_max/32] uint32, caller-owned: every row's selection bitmap
 *   row_k    [n_heads][R] int32 or NULL: every row's selection size
 * R in [1, 256]; p in [0, 1]; S_max a multiple of 32, at most 65536.
 */
hk_status hk_vote_topp(int32_t n_heads, int32_t R, int32_t S_max, const int32_t* cand_len,
                       const uint16_t* page_mask, const float* a_rows, double p, uint16_t* votes,
                       uint32_t* row_sel, int32_t* row_k, int32_t* status, hipStream_t stream);

/* Budget state of every head at a compression point:
 *   used = 16 * n_pages[h], valid = number of set page_mask bits of the head,
 *   HK_BUDGET_REWRITE if used > L_upper,  HK_BUDGET_SPARSE else if valid > L_lower,
 *   HK_BUDGET_KEEP otherwise;
 *   k_cap[h] = max(0, 16 * floor(L_upper / 16) - 16 * nd) for REWRITE heads (nd = the
 *   dense pages, min(n_pages, ceil(L_dense / 16))), -1 otherwise: the rewritten candidates
 *   then fit the pages L_upper leaves beside the dense tier.
 * head_mode, k_cap [n_heads] int32 (device).  0 <= L_lower <= L_upper; L_dense >= 0.
 */
hk_status hk_budget_plan(const hk_dims* dims, const hk_paged_kv* kv, int32_t L_dense,
                         int32_t L_lower, int32_t L_upper, int32_t* head_mode, int32_t* k_cap,
                         hipStream_t stream);

/* Selection under the budget, per head:
 *   KEEP heads: every candidate.
 *   other heads: the sinks -- candidates j < n_sink, the attention sinks (Sec. 3.1 Tier 1;
 *   Sec. 4 baselines) -- are always kept; the base set is the other candidates with
 *   votes[h][j] >= 1 (if votes) and bit j of sel_in (if sel_in); it is ranked by
 *   (votes desc, c desc, slot desc) -- a NULL votes or c counts as 0, c is clamped to [0, 1]
 *   with NaN as 0 -- and its first min(|base|, cap) slots are kept,
 *   cap = max(0, k_cap[h] - |sinks|), no cap when k_cap is NULL or k_cap[h] < 0.
 * head_mode NULL treats every head as REWRITE.  Outputs sel_out [n_heads][S_max/32] uint32
 * (16-byte aligned) and k_out [n_heads] = number of selected slots.  n_sink >= 0; S_max a
 * multiple of 32, at most 65536.
 */
hk_status hk_budget_select(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                           const uint16_t* page_mask, const uint16_t* votes, const float* c,
                           const uint32_t* sel_in, const int32_t* head_mode, const int32_t* k_cap,
                           int32_t n_sink, uint32_t* sel_out, int32_t* k_out, hipStream_t stream);

/* hk_compact with the bands set per head by its budget state instead of L_sparse:
 *   REWRITE  every page before the dense tier is condensed (rewritten);
 *   SPARSE   every page before the dense tier is sparse (kept under the mask);
 *   KEEP     the row is left as it is (sel_bits is not read for it).
 * Workspace, allocator, ordering and HK_FLAG_NOSPACE behaviour as for hk_compact
 * (hk_workspace_size(HK_OP_COMPACT)), alloc->capacity >= kv->num_pages as there.
 * head_mode [n_heads] int32 with values HK_BUDGET_*.
 */
hk_status hk_compact_modes(const hk_dims* dims, const hk_paged_kv* kv, const uint32_t* sel_bits,
                           int32_t L_dense, const int32_t* head_mode, const hk_allocator* alloc,
                           int32_t* status, void* workspace, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------ kernel timing
 * Optional HIP-event timing of individual kernels, for measurement harnesses (not part of
 * the method).  hk_timing_enable(mask) selects the kernels to time: bit k of mask stands
 * for kernel id k below (0 turns timing off, the default).  Every launch of a selected
 * kernel is then bracketed by two events recorded on its launch stream.  hk_timing_read
 * waits for the events of one kernel, returns their summed duration (ms) and the number
 * of timed launches since the previous read, and clears them.  Events are recycled
 * between reads.  Thread-safe.  Errors: HK_ERR_ARG for an unknown kernel id or a null
 * output, HK_ERR_HIP if an event could not be read (the sum then omits it).
 */
enum {
  HK_TK_SCORE_PASS1 = 0,   /* hk_score: LSE pass over the window                        */
  HK_TK_SCORE_MERGE = 1,   /* hk_score: chunk partials -> row LSE                        */
  HK_TK_SCORE_PASS2 = 2,   /* hk_score: attention-mass (and redundancy) pass             */
  HK_TK_CALIBRATE = 3,     /* hk_calibrate                                               */
  HK_TK_TOPP = 4,          /* hk_topp_select                                             */
  HK_TK_SOLVE_T = 5,       /* hk_calibrate_solve_T and hk_calibrate_solve_T_gd           */
  HK_TK_COMPACT_GATHER = 6,/* hk_compact: condensed-row gather into fresh pages          */
  HK_TK_COMPACT_META = 7,  /* hk_compact: plan, alloc, table, push (four launches)       */
  HK_TK_DECODE_SPLIT = 8,  /* hk_decode_attn: split-K partial states                     */
  HK_TK_DECODE_MERGE = 9,  /* hk_decode_attn: merge of the partial states                */
  HK_TK_APPEND = 10,       /* hk_append_kv: count + write, timed together                */
  HK_TK_CALIB_TOPP = 11,   /* hk_calibrate_topp                                          */
  HK_TK_SCORE_ROWS = 12,   /* hk_score_rows                                              */
  HK_TK_VOTE = 13,         /* hk_vote_topp: per-row Top-p                                */
  HK_TK_VOTE_COUNT = 14,   /* hk_vote_topp: column counts of the row bitmaps             */
  HK_TK_BUDGET_PLAN = 15,  /* hk_budget_plan                                             */
  HK_TK_BUDGET_SELECT = 16,/* hk_budget_select                                           */
  HK_TK_COUNT = 17
};
hk_status hk_timing_enable(uint32_t kernel_mask);
hk_status hk_timing_read(int32_t kernel, double* total_ms, int64_t* launches);

/* Rate probes behind the score passes' rooflines (measurement only; not a step of the
 * method).  hk_probe launches one throughput kernel of `blocks` workgroups of 256 threads
 * on `stream`:
 *   HK_PROBE_EXP  : every thread runs 8 independent chains of `iters` hardware
 *                   exponentials (v_exp_f32): 8 * iters * 256 * blocks of them;
 *   HK_PROBE_MFMA : every wave runs 4 independent chains of `iters`
 *                   v_mfma_f32_32x32x16_bf16: 16 * iters * blocks MFMAs of 32768 flop;
 *   HK_PROBE_MIX  : the score passes' work mix: every wave runs iters x 4 steps, a step
 *                   being one 32x32x16 bf16 MFMA plus, for two values per lane, an fma, a
 *                   hardware exponential and an add, interleaved one step at a time;
 *   HK_PROBE_SPLIT: the same total work with the MFMAs in the even waves and the VALU
 *                   work in the odd waves of every workgroup (2 iters x 4 steps each);
 *   HK_PROBE_VALU : only the VALU part of HK_PROBE_MIX;
 *   HK_PROBE_MFMA4: only the MFMA part of HK_PROBE_MIX.
 * out: device, >= 256 * blocks floats, caller-owned; receives one value per thread (it
 * keeps the work live).  The caller times the launch.  Errors: HK_ERR_ARG for an unknown
 * kind, blocks < 1 or > 2^20, iters < 1, or a null out.
 */
enum { HK_PROBE_EXP = 0, HK_PROBE_MFMA = 1, HK_PROBE_MIX = 2, HK_PROBE_SPLIT = 3, HK_PROBE_VALU = 4,
       HK_PROBE_MFMA4 = 5 };
hk_status hk_probe(int32_t kind, int32_t blocks, int32_t iters, float* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* HARDKV_H_ */

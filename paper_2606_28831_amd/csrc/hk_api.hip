// C ABI of libhardkv: argument validation and dispatch to the HIP launchers.
// Declarations, argument meaning and error behaviour: include/hardkv.h.
#include <algorithm>
#include <cmath>
#include <cstdint>

#include "hk_internal.h"

bool hk_decode_supports_group(int G);

namespace {

constexpr int kMaxSlots = 32768;   // per-head logical slots held in registers by the selectors
constexpr int kMaxSlotsWide = 262144;   // per-head slots of the multi-workgroup selector
constexpr int kMaxSlotsBudget = 65536;  // per-row slots of the vote and budget selection

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

hk_status check_dims(const hk_dims* d, bool need_w) {
  if (!d) return HK_ERR_ARG;
  if (d->NS <= 0 || d->Hq <= 0 || d->Hkv <= 0 || d->D <= 0) return HK_ERR_ARG;
  if (need_w && d->W <= 0) return HK_ERR_ARG;
  if (d->D != 64 && d->D != 128) return HK_ERR_SHAPE;
  if (d->Hq % d->Hkv != 0) return HK_ERR_SHAPE;
  if ((long long)d->NS * d->Hkv > 65535) return HK_ERR_SHAPE;
  return HK_OK;
}

hk_status check_kv(const hk_paged_kv* kv, bool need_v) {
  if (!kv || !kv->k_pool || !kv->page_table || !kv->page_mask || !kv->n_pages) return HK_ERR_ARG;
  if (need_v && !kv->v_pool) return HK_ERR_ARG;
  if (kv->dtype != HK_F32 && kv->dtype != HK_BF16) return HK_ERR_DTYPE;
  if (kv->num_pages <= 0 || kv->max_pages <= 0) return HK_ERR_ARG;
  if (kv->max_pages % 2 != 0) return HK_ERR_SHAPE;                 // S_max multiple of 32
  if (!aligned16(kv->k_pool) || (need_v && !aligned16(kv->v_pool))) return HK_ERR_ALIGN;
  if (!aligned16(kv->page_table) || !aligned16(kv->page_mask) || !aligned16(kv->n_pages))
    return HK_ERR_ALIGN;
  return HK_OK;
}

hk_status check_rows(int n_heads, int S_max, const int32_t* cand_len, int max_slots = kMaxSlots) {
  if (n_heads <= 0 || S_max <= 0 || !cand_len) return HK_ERR_ARG;
  if (S_max % 32 != 0 || S_max > max_slots) return HK_ERR_SHAPE;
  if (n_heads > 1 << 20) return HK_ERR_SHAPE;
  return HK_OK;
}

hk_status check_rows_wide(int n_heads, int S_max, const int32_t* cand_len) {
  return check_rows(n_heads, S_max, cand_len, kMaxSlotsWide);
}

hk_status launched(hipError_t e) { return e == hipSuccess ? HK_OK : HK_ERR_HIP; }

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace of hk_compress: scores, candidate counts, row LSEs, selection, then the score,
// selection and compaction scratch (the stages run one after the other; they share one
// region).
struct CompressWs {
  size_t s, cand, lse, sel, scratch, total;
};
CompressWs compress_ws(const hk_dims* d, int max_pages) {
  const size_t H = (size_t)d->NS * d->Hkv, S = (size_t)max_pages * HK_PAGE;
  CompressWs w;
  w.s = 0;
  w.cand = w.s + al256(H * S * 4);
  w.lse = w.cand + al256(H * 4);
  w.sel = w.lse + al256((size_t)d->W * d->NS * d->Hq * 4);
  w.scratch = w.sel + al256(H * (S / 32) * 4);
  const size_t a = hk_score_ws(d->NS, d->Hq, d->Hkv, d->D, d->W, max_pages);
  const size_t b = hk_compact_ws((int)H, max_pages);
  const size_t c = hk_select_wide_ws((int)H, (int)S);
  w.total = w.scratch + al256(std::max(a, std::max(b, c)));
  return w;
}

}  // namespace

extern "C" {

size_t hk_workspace_size(int32_t op, const hk_dims* d, int32_t max_pages) {
  if (!d || max_pages <= 0) return 0;
  switch (op) {
    case HK_OP_SCORE: return hk_score_ws(d->NS, d->Hq, d->Hkv, d->D, d->W, max_pages);
    case HK_OP_COMPACT: return hk_compact_ws(d->NS * d->Hkv, max_pages);
    case HK_OP_DECODE: return hk_decode_ws(d->NS, d->Hq, d->Hkv, d->D, max_pages);
    case HK_OP_APPEND: return hk_append_ws(d->NS, d->Hkv);
    case HK_OP_COMPRESS: return compress_ws(d, max_pages).total;
    case HK_OP_SELECT: return hk_select_wide_ws(d->NS * d->Hkv, max_pages * HK_PAGE);
    default: return 0;
  }
}

const char* hk_status_string(int32_t code, int32_t flags) {
  if (flags) {
    switch (code) {
      case HK_FLAG_NOSPACE: return "HK_FLAG_NOSPACE: page pool exhausted, cache left unchanged";
      case HK_FLAG_NAN: return "HK_FLAG_NAN: NaN probability given weight 0";
      case HK_FLAG_RANGE: return "HK_FLAG_RANGE: probability outside [0,1] clamped";
      default: return "unknown flag";
    }
  }
  switch (code) {
    case HK_OK: return "HK_OK";
    case HK_ERR_ARG: return "HK_ERR_ARG: null pointer or size/scalar out of range";
    case HK_ERR_DTYPE: return "HK_ERR_DTYPE: dtype must be HK_F32 or HK_BF16";
    case HK_ERR_SHAPE: return "HK_ERR_SHAPE: unsupported shape";
    case HK_ERR_ALIGN: return "HK_ERR_ALIGN: pointer not 16-byte (workspace: 256-byte) aligned";
    case HK_ERR_WORKSPACE: return "HK_ERR_WORKSPACE: workspace smaller than hk_workspace_size()";
    case HK_ERR_HIP: return "HK_ERR_HIP: kernel launch failed";
    case HK_ERR_SCRATCH:
      return "HK_ERR_SCRATCH: the call needs more than the library's static scratch (16 MiB)";
    default: return "unknown status";
  }
}

hk_status hk_score(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv, int32_t L_dense,
                   float sm_scale, const float* row_lse_in, float* row_lse_out, float* s_attn,
                   int32_t* cand_len_out, const int32_t* ref_slots, int32_t n_ref, float* x_red,
                   void* workspace, size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, true);
  if (e) return e;
  if ((e = check_kv(kv, false))) return e;
  if (!q_obs || !cand_len_out) return HK_ERR_ARG;
  // without s_attn only the row LSEs are computed: they must be computed and returned
  if (!s_attn && (row_lse_in || !row_lse_out || x_red)) return HK_ERR_ARG;
  if (L_dense < 0 || !(sm_scale > 0.f) || !std::isfinite(sm_scale)) return HK_ERR_ARG;
  const int G = dims->Hq / dims->Hkv;
  if (G * dims->W > 256) return HK_ERR_SHAPE;
  if ((x_red != nullptr) != (ref_slots != nullptr)) return HK_ERR_ARG;
  if (x_red && (n_ref < 0 || n_ref > 256)) return HK_ERR_ARG;
  if (!aligned16(q_obs)) return HK_ERR_ALIGN;
  if (hk_score_lds_bytes(dims->Hq / dims->Hkv * dims->W, dims->D, kv->dtype == HK_BF16 ? 2 : 4,
                         x_red != nullptr) > 160 * 1024)
    return HK_ERR_SHAPE;
  const size_t need = hk_score_ws(dims->NS, dims->Hq, dims->Hkv, dims->D, dims->W, kv->max_pages);
  if (!row_lse_in) {
    if (!workspace || ws_bytes < need) return HK_ERR_WORKSPACE;
    if (!aligned256(workspace)) return HK_ERR_ALIGN;
  }
  hk_score_args a;
  a.q_obs = q_obs;
  a.kv = kv;
  a.NS = dims->NS;
  a.Hq = dims->Hq;
  a.Hkv = dims->Hkv;
  a.D = dims->D;
  a.W = dims->W;
  a.L_dense = L_dense;
  a.sm_scale = sm_scale;
  a.row_lse_in = row_lse_in;
  a.row_lse_out = row_lse_out;
  a.s_attn = s_attn;
  a.cand_len = cand_len_out;
  a.ref_slots = ref_slots;
  a.n_ref = x_red ? n_ref : 0;
  a.x_red = x_red;
  a.ws = workspace;
  return launched(hk_launch_score(a, stream));
}

hk_status hk_calibrate(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                       const uint16_t* page_mask, int32_t n_metrics, const float* const* x,
                       const float* const* T, const float* w, float* c_out, float* lse_out,
                       hipStream_t stream) {
  hk_status e = check_rows(n_heads, S_max, cand_len);
  if (e) return e;
  if (n_metrics < 1 || n_metrics > 2 || !x || !w || !c_out) return HK_ERR_ARG;
  for (int m = 0; m < n_metrics; ++m)
    if (!x[m] || !std::isfinite(w[m])) return HK_ERR_ARG;
  const float* T0 = T ? T[0] : nullptr;
  const float* T1 = (T && n_metrics > 1) ? T[1] : nullptr;
  return launched(hk_launch_calibrate(n_heads, S_max, cand_len, page_mask, n_metrics, x[0],
                                      n_metrics > 1 ? x[1] : nullptr, T0, T1, w[0],
                                      n_metrics > 1 ? w[1] : 0.f, c_out, lse_out, stream));
}

hk_status hk_topp_select(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                         const uint16_t* page_mask, const float* c, double p, int32_t k_min,
                         int32_t k_max, uint32_t* sel_bits, int32_t* k_out, float* sel_mass_out,
                         int32_t* status, hipStream_t stream) {
  hk_status e = check_rows(n_heads, S_max, cand_len);
  if (e) return e;
  if (!c || !sel_bits || !k_out) return HK_ERR_ARG;
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  if (!aligned16(sel_bits)) return HK_ERR_ALIGN;
  const int p_q = (int)std::nearbyint(p * 1e6);
  return launched(hk_launch_topp(n_heads, S_max, cand_len, page_mask, c, p_q, k_min, k_max,
                                 sel_bits, k_out, sel_mass_out, status, stream));
}

hk_status hk_calibrate_topp(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                            const uint16_t* page_mask, int32_t n_metrics, const float* const* x,
                            const float* const* T, const float* w, double p, int32_t k_min,
                            int32_t k_max, float* c_out, float* lse_out, uint32_t* sel_bits,
                            int32_t* k_out, float* sel_mass_out, int32_t* status,
                            hipStream_t stream) {
  hk_status e = check_rows(n_heads, S_max, cand_len);
  if (e) return e;
  if (n_metrics < 1 || n_metrics > 2 || !x || !w || !sel_bits || !k_out) return HK_ERR_ARG;
  for (int m = 0; m < n_metrics; ++m)
    if (!x[m] || !std::isfinite(w[m])) return HK_ERR_ARG;
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  if (!aligned16(sel_bits)) return HK_ERR_ALIGN;
  const int p_q = (int)std::nearbyint(p * 1e6);
  const float* T0 = T ? T[0] : nullptr;
  const float* T1 = (T && n_metrics > 1) ? T[1] : nullptr;
  return launched(hk_launch_calib_topp(n_heads, S_max, cand_len, page_mask, n_metrics, x[0],
                                       n_metrics > 1 ? x[1] : nullptr, T0, T1, w[0],
                                       n_metrics > 1 ? w[1] : 0.f, p_q, k_min, k_max, c_out,
                                       lse_out, sel_bits, k_out, sel_mass_out, status, stream));
}

size_t hk_select_workspace_size(int32_t n_heads, int32_t S_max) {
  if (n_heads <= 0 || S_max <= 0) return 0;
  return hk_select_wide_ws(n_heads, S_max);
}

hk_status hk_topp_select_ws(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                            const uint16_t* page_mask, const float* c, double p, int32_t k_min,
                            int32_t k_max, uint32_t* sel_bits, int32_t* k_out,
                            float* sel_mass_out, int32_t* status, void* workspace,
                            size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_rows_wide(n_heads, S_max, cand_len);
  if (e) return e;
  if (!c || !sel_bits || !k_out) return HK_ERR_ARG;
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  if (!aligned16(sel_bits) || !aligned16(c)) return HK_ERR_ALIGN;
  if (!workspace || ws_bytes < hk_select_wide_ws(n_heads, S_max)) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  const int p_q = (int)std::nearbyint(p * 1e6);
  return launched(hk_launch_select_wide(n_heads, S_max, cand_len, page_mask, 0, nullptr, nullptr,
                                        nullptr, nullptr, 0.f, 0.f, c, p_q, k_min, k_max, nullptr,
                                        nullptr, sel_bits, k_out, sel_mass_out, status, workspace,
                                        stream));
}

hk_status hk_calibrate_topp_ws(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                               const uint16_t* page_mask, int32_t n_metrics,
                               const float* const* x, const float* const* T, const float* w,
                               double p, int32_t k_min, int32_t k_max, float* c_out,
                               float* lse_out, uint32_t* sel_bits, int32_t* k_out,
                               float* sel_mass_out, int32_t* status, void* workspace,
                               size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_rows_wide(n_heads, S_max, cand_len);
  if (e) return e;
  if (n_metrics < 1 || n_metrics > 2 || !x || !w || !sel_bits || !k_out) return HK_ERR_ARG;
  for (int m = 0; m < n_metrics; ++m)
    if (!x[m] || !std::isfinite(w[m])) return HK_ERR_ARG;
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  if (!aligned16(sel_bits) || (c_out && !aligned16(c_out))) return HK_ERR_ALIGN;
  for (int m = 0; m < n_metrics; ++m)
    if (!aligned16(x[m])) return HK_ERR_ALIGN;
  if (!workspace || ws_bytes < hk_select_wide_ws(n_heads, S_max)) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  const int p_q = (int)std::nearbyint(p * 1e6);
  const float* T0 = T ? T[0] : nullptr;
  const float* T1 = (T && n_metrics > 1) ? T[1] : nullptr;
  return launched(hk_launch_select_wide(n_heads, S_max, cand_len, page_mask, n_metrics, x[0],
                                        n_metrics > 1 ? x[1] : nullptr, T0, T1, w[0],
                                        n_metrics > 1 ? w[1] : 0.f, nullptr, p_q, k_min, k_max,
                                        c_out, lse_out, sel_bits, k_out, sel_mass_out, status,
                                        workspace, stream));
}

hk_status hk_pool_max(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                      const uint16_t* page_mask, const float* x, int32_t radius, float* x_out,
                      hipStream_t stream) {
  hk_status e = check_rows_wide(n_heads, S_max, cand_len);       // tiled: any length
  if (e) return e;
  if (!x || !x_out || x == x_out) return HK_ERR_ARG;
  if (radius < 0 || radius > 64) return HK_ERR_SHAPE;
  return launched(hk_launch_pool_max(n_heads, S_max, cand_len, page_mask, x, radius, x_out, stream));
}

hk_status hk_calibrate_solve_T(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                               const uint16_t* page_mask, const float* x, const int32_t* k,
                               const float* target_mass, float T_lo, float T_hi, int32_t iters,
                               float* T_out, hipStream_t stream) {
  hk_status e = check_rows_wide(n_heads, S_max, cand_len);       // longer rows are streamed
  if (e) return e;
  if (!x || !k || !target_mass || !T_out) return HK_ERR_ARG;
  if (!(T_lo > 0.f) || !(T_hi > T_lo) || !std::isfinite(T_hi) || iters < 1 || iters > 64)
    return HK_ERR_ARG;
  return launched(hk_launch_solve_T(n_heads, S_max, cand_len, page_mask, x, k, target_mass, T_lo,
                                    T_hi, iters, T_out, stream));
}

hk_status hk_calibrate_solve_T_gd(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                                  const uint16_t* page_mask, const float* x, const int32_t* k,
                                  const float* target_mass, float T_init, float lr, int32_t iters,
                                  float tol, float* T_out, float* loss_out, hipStream_t stream) {
  hk_status e = check_rows_wide(n_heads, S_max, cand_len);    // longer rows are streamed
  if (e) return e;
  if (!x || !k || !target_mass || !T_out) return HK_ERR_ARG;
  if (!(T_init > 0.f) || !std::isfinite(T_init) || !(lr > 0.f) || !std::isfinite(lr)) return HK_ERR_ARG;
  if (iters < 0 || iters > 100000 || !(tol >= 0.f)) return HK_ERR_ARG;
  return launched(hk_launch_solve_T_gd(n_heads, S_max, cand_len, page_mask, x, k, target_mass, T_init,
                                       lr, iters, tol, T_out, loss_out, stream));
}

hk_status hk_compact(const hk_dims* dims, const hk_paged_kv* kv, const uint32_t* sel_bits,
                     int32_t L_dense, int32_t L_sparse, const hk_allocator* alloc, int32_t* status,
                     void* workspace, size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!sel_bits || !alloc || !alloc->free_ids || !alloc->free_top) return HK_ERR_ARG;
  // freed pages are pushed back: the stack must be able to hold every page of the pool
  if (alloc->capacity < kv->num_pages) return HK_ERR_ARG;
  if (L_dense < 0 || L_sparse < 0) return HK_ERR_ARG;
  if ((long long)kv->max_pages * 6 > 160 * 1024) return HK_ERR_SHAPE;   // table row staged in LDS
  const int n_heads = dims->NS * dims->Hkv;
  if (!workspace || ws_bytes < hk_compact_ws(n_heads, kv->max_pages)) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  return launched(hk_launch_compact(n_heads, dims->D, kv, sel_bits, L_dense, L_sparse, nullptr,
                                    alloc, status, workspace, stream));
}

hk_status hk_compress(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv,
                      int32_t L_dense, int32_t L_sparse, float sm_scale, const float* row_lse_in,
                      double p, int32_t k_min, int32_t k_max, const hk_allocator* alloc,
                      uint32_t* sel_bits_out, int32_t* k_out, int32_t* status, void* workspace,
                      size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, true);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!k_out || !workspace) return HK_ERR_ARG;
  if (!alloc || !alloc->free_ids || !alloc->free_top || alloc->capacity < kv->num_pages)
    return HK_ERR_ARG;                                             // checked before any launch
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  // the selection's row limits, checked here so that no launch runs before a refusal
  if (kv->max_pages > kMaxSlotsWide / HK_PAGE || dims->NS * dims->Hkv > (1 << 20)) return HK_ERR_SHAPE;
  const CompressWs cw = compress_ws(dims, kv->max_pages);
  if (ws_bytes < cw.total) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  if (sel_bits_out && !aligned16(sel_bits_out)) return HK_ERR_ALIGN;
  char* ws = static_cast<char*>(workspace);
  float* s = reinterpret_cast<float*>(ws + cw.s);
  int32_t* cand = reinterpret_cast<int32_t*>(ws + cw.cand);
  float* lse = reinterpret_cast<float*>(ws + cw.lse);
  uint32_t* sel = sel_bits_out ? sel_bits_out : reinterpret_cast<uint32_t*>(ws + cw.sel);
  void* scratch = ws + cw.scratch;
  const size_t scratch_bytes = ws_bytes - cw.scratch;
  e = hk_score(dims, q_obs, kv, L_dense, sm_scale, row_lse_in, row_lse_in ? nullptr : lse, s, cand,
               nullptr, 0, nullptr, scratch, scratch_bytes, stream);
  if (e) return e;
  const int n_heads = dims->NS * dims->Hkv, S_max = kv->max_pages * HK_PAGE;
  const float* xs[1] = {s};
  const float w1[1] = {1.0f};
  e = hk_calibrate_topp_ws(n_heads, S_max, cand, kv->page_mask, 1, xs, nullptr, w1, p, k_min,
                           k_max, nullptr, nullptr, sel, k_out, nullptr, status, scratch,
                           scratch_bytes, stream);
  if (e) return e;
  return hk_compact(dims, kv, sel, L_dense, L_sparse, alloc, status, scratch, scratch_bytes, stream);
}

hk_status hk_compact_modes(const hk_dims* dims, const hk_paged_kv* kv, const uint32_t* sel_bits,
                           int32_t L_dense, const int32_t* head_mode, const hk_allocator* alloc,
                           int32_t* status, void* workspace, size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!sel_bits || !head_mode || !alloc || !alloc->free_ids || !alloc->free_top) return HK_ERR_ARG;
  if (alloc->capacity < kv->num_pages) return HK_ERR_ARG;        // as for hk_compact
  if (L_dense < 0) return HK_ERR_ARG;
  if ((long long)kv->max_pages * 6 > 160 * 1024) return HK_ERR_SHAPE;
  const int n_heads = dims->NS * dims->Hkv;
  if (!workspace || ws_bytes < hk_compact_ws(n_heads, kv->max_pages)) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  return launched(hk_launch_compact(n_heads, dims->D, kv, sel_bits, L_dense, 0, head_mode, alloc,
                                    status, workspace, stream));
}

hk_status hk_score_rows(const hk_dims* dims, const void* q_obs, const hk_paged_kv* kv,
                        int32_t L_dense, float sm_scale, const float* row_lse, float* a_rows,
                        hipStream_t stream) {
  hk_status e = check_dims(dims, true);
  if (e) return e;
  if ((e = check_kv(kv, false))) return e;
  if (!q_obs || !row_lse || !a_rows) return HK_ERR_ARG;
  if (L_dense < 0 || !(sm_scale > 0.f) || !std::isfinite(sm_scale)) return HK_ERR_ARG;
  if (dims->Hq / dims->Hkv * dims->W > 256) return HK_ERR_SHAPE;
  if (!aligned16(q_obs)) return HK_ERR_ALIGN;
  if (hk_score_lds_bytes(dims->Hq / dims->Hkv * dims->W, dims->D, kv->dtype == HK_BF16 ? 2 : 4,
                         false) > 160 * 1024)
    return HK_ERR_SHAPE;
  return launched(hk_launch_score_rows(dims->NS, dims->Hq, dims->Hkv, dims->D, dims->W, q_obs, kv,
                                       L_dense, sm_scale, row_lse, a_rows, stream));
}

hk_status hk_vote_topp(int32_t n_heads, int32_t R, int32_t S_max, const int32_t* cand_len,
                       const uint16_t* page_mask, const float* a_rows, double p, uint16_t* votes,
                       uint32_t* row_sel, int32_t* row_k, int32_t* status, hipStream_t stream) {
  hk_status e = check_rows(n_heads, S_max, cand_len, kMaxSlotsBudget);
  if (e) return e;
  if (R < 1 || R > 256) return HK_ERR_SHAPE;
  if (n_heads > 65535) return HK_ERR_SHAPE;
  if (!a_rows || !votes || !row_sel) return HK_ERR_ARG;
  if (!(p >= 0.0 && p <= 1.0)) return HK_ERR_ARG;
  if (!aligned16(votes) || !aligned16(row_sel)) return HK_ERR_ALIGN;
  const int p_q = (int)std::nearbyint(p * 1e6);
  return launched(hk_launch_vote_topp(n_heads, R, S_max, cand_len, page_mask, a_rows, p_q, votes,
                                      row_k, row_sel, status, stream));
}

hk_status hk_budget_plan(const hk_dims* dims, const hk_paged_kv* kv, int32_t L_dense,
                         int32_t L_lower, int32_t L_upper, int32_t* head_mode, int32_t* k_cap,
                         hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, false))) return e;
  if (!head_mode || !k_cap) return HK_ERR_ARG;
  if (L_dense < 0 || L_lower < 0 || L_upper < L_lower) return HK_ERR_ARG;
  return launched(hk_launch_budget_plan(dims->NS * dims->Hkv, kv->max_pages, kv->n_pages,
                                        kv->page_mask, L_dense, L_lower, L_upper, head_mode, k_cap,
                                        stream));
}

hk_status hk_budget_select(int32_t n_heads, int32_t S_max, const int32_t* cand_len,
                           const uint16_t* page_mask, const uint16_t* votes, const float* c,
                           const uint32_t* sel_in, const int32_t* head_mode, const int32_t* k_cap,
                           int32_t n_sink, uint32_t* sel_out, int32_t* k_out, hipStream_t stream) {
  hk_status e = check_rows(n_heads, S_max, cand_len, kMaxSlotsBudget);
  if (e) return e;
  if (!sel_out || !k_out || n_sink < 0) return HK_ERR_ARG;
  if (!aligned16(sel_out)) return HK_ERR_ALIGN;
  return launched(hk_launch_budget_select(n_heads, S_max, cand_len, page_mask, votes, c, sel_in,
                                          head_mode, k_cap, n_sink, sel_out, k_out, stream));
}

hk_status hk_alloc_init(const hk_allocator* alloc, int32_t first_free, int32_t num_pages,
                        hipStream_t stream) {
  if (!alloc || !alloc->free_ids || !alloc->free_top) return HK_ERR_ARG;
  if (first_free < 0 || num_pages < first_free || num_pages - first_free > alloc->capacity)
    return HK_ERR_ARG;
  if (!aligned16(alloc->free_ids)) return HK_ERR_ALIGN;
  return launched(hk_launch_alloc_init(alloc->free_ids, alloc->free_top, first_free,
                                       num_pages - first_free, stream));
}

hk_status hk_decode_attn(const hk_dims* dims, const void* q, const hk_paged_kv* kv, float sm_scale,
                         float* o, float* lse, void* workspace, size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!q || !o || !lse) return HK_ERR_ARG;
  if (!(sm_scale > 0.f) || !std::isfinite(sm_scale)) return HK_ERR_ARG;
  if (!hk_decode_supports_group(dims->Hq / dims->Hkv)) return HK_ERR_SHAPE;
  if (!aligned16(q)) return HK_ERR_ALIGN;
  if (!workspace || ws_bytes < hk_decode_ws(dims->NS, dims->Hq, dims->Hkv, dims->D, kv->max_pages))
    return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  return launched(hk_launch_decode(dims->NS, dims->Hq, dims->Hkv, dims->D, q, kv, sm_scale, o, lse,
                                   workspace, stream));
}

hk_status hk_decode_attn_noalloc(const hk_dims* dims, const void* q, const hk_paged_kv* kv,
                                 float sm_scale, float* o, float* lse, hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!q || !o || !lse) return HK_ERR_ARG;
  if (!(sm_scale > 0.f) || !std::isfinite(sm_scale)) return HK_ERR_ARG;
  if (!hk_decode_supports_group(dims->Hq / dims->Hkv)) return HK_ERR_SHAPE;
  if (!aligned16(q)) return HK_ERR_ALIGN;
  if (hk_decode_noalloc_bytes(dims->NS, dims->Hq, dims->Hkv, dims->D, kv->max_pages) >
      HK_NOALLOC_SCRATCH_BYTES)
    return HK_ERR_SCRATCH;
  void* scratch = nullptr;
  if (hk_noalloc_scratch(&scratch) != hipSuccess) return HK_ERR_HIP;
  return launched(hk_launch_decode(dims->NS, dims->Hq, dims->Hkv, dims->D, q, kv, sm_scale, o, lse,
                                   scratch, stream, /*timed=*/false));
}

size_t hk_decode_noalloc_scratch_bytes(const hk_dims* dims, int32_t max_pages) {
  if (!dims || dims->Hkv <= 0 || dims->NS <= 0 || dims->Hq <= 0 || max_pages <= 0) return 0;
  return hk_decode_noalloc_bytes(dims->NS, dims->Hq, dims->Hkv, dims->D, max_pages);
}

hk_status hk_decode_plan(const hk_dims* dims, int32_t max_pages, int32_t* n_split,
                         int32_t* pages_per_split) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if (max_pages <= 0 || !n_split || !pages_per_split) return HK_ERR_ARG;
  int pps, ns;
  hk_decode_split_plan(dims->NS * dims->Hkv, max_pages, &pps, &ns);
  *n_split = ns;
  *pages_per_split = pps;
  return HK_OK;
}

hk_status hk_append_kv(const hk_dims* dims, const hk_paged_kv* kv, const void* k_new,
                       const void* v_new, const hk_allocator* alloc, int32_t* status,
                       void* workspace, size_t ws_bytes, hipStream_t stream) {
  hk_status e = check_dims(dims, false);
  if (e) return e;
  if ((e = check_kv(kv, true))) return e;
  if (!k_new || !v_new || !alloc || !alloc->free_ids || !alloc->free_top) return HK_ERR_ARG;
  if (!aligned16(k_new) || !aligned16(v_new)) return HK_ERR_ALIGN;
  if (!workspace || ws_bytes < hk_append_ws(dims->NS, dims->Hkv)) return HK_ERR_WORKSPACE;
  if (!aligned256(workspace)) return HK_ERR_ALIGN;
  return launched(hk_launch_append(dims->NS, dims->Hkv, dims->D, kv, k_new, v_new, alloc, status,
                                   workspace, stream));
}

hk_status hk_probe(int32_t kind, int32_t blocks, int32_t iters, float* out, hipStream_t stream) {
  if (kind < HK_PROBE_EXP || kind > HK_PROBE_MFMA4) return HK_ERR_ARG;
  if (blocks < 1 || blocks > (1 << 20) || iters < 1 || !out) return HK_ERR_ARG;
  return launched(hk_launch_probe(kind, blocks, iters, out, stream));
}

}  // extern "C"

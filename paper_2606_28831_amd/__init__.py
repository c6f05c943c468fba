"""Python binding of libhardkv (Hard-KV decoding-time compression step on MI355X).

Argument marshalling only: every step runs in the HIP kernels of libhardkv.so.
Torch tensors provide device memory and the current stream; each wrapper passes
their device pointers to the C entry point of the same name (include/hardkv.h)
and raises HardKVError on a non-zero status.  There is no fallback: if the
library is missing, importing the entry points raises.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

__all__ = ["HardKVError", "lib", "PagedKV", "Allocator", "hk_score", "hk_calibrate",
           "hk_calibrate_solve_T", "hk_topp_select", "hk_compact", "hk_decode_attn",
           "hk_append_kv", "hk_workspace_size", "hk_status_string", "OP_SCORE", "OP_COMPACT",
           "OP_DECODE", "OP_APPEND", "FLAG_NOSPACE", "FLAG_NAN", "FLAG_RANGE", "LIB_PATH",
           "hk_timing_enable", "hk_timing_read", "TIMED_KERNELS", "hk_calibrate_topp",
           "hk_pool_max", "hk_score_rows", "hk_vote_topp", "hk_budget_plan", "hk_budget_select",
           "hk_compact_modes", "hk_calibrate_solve_T_gd", "hk_alloc_init", "hk_compress", "OP_COMPRESS", "BUDGET_KEEP", "BUDGET_SPARSE", "BUDGET_REWRITE",
           "hk_probe", "PROBE_EXP", "PROBE_MFMA", "PROBE_MIX", "PROBE_SPLIT", "PROBE_VALU",
           "PROBE_MFMA4", "hk_decode_plan",
           "hk_decode_attn_noalloc", "hk_decode_noalloc_scratch_bytes", "ERR_SCRATCH",
           "OP_SELECT", "hk_select_workspace_size", "select_workspace", "hk_topp_select_ws",
           "hk_calibrate_topp_ws"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhardkv.so")

HK_F32, HK_BF16 = 0, 1
OP_SCORE, OP_COMPACT, OP_DECODE, OP_APPEND, OP_COMPRESS, OP_SELECT = 0, 1, 2, 3, 4, 5
FLAG_NOSPACE, FLAG_NAN, FLAG_RANGE = 1, 2, 4
ERR_SCRATCH = 7
BUDGET_KEEP, BUDGET_SPARSE, BUDGET_REWRITE = 0, 1, 2
PROBE_EXP, PROBE_MFMA, PROBE_MIX, PROBE_SPLIT, PROBE_VALU, PROBE_MFMA4 = 0, 1, 2, 3, 4, 5
EXPORTED = ["hk_score", "hk_calibrate", "hk_calibrate_solve_T", "hk_topp_select", "hk_compact",
            "hk_decode_attn", "hk_append_kv", "hk_workspace_size", "hk_status_string",
            "hk_timing_enable", "hk_timing_read", "hk_calibrate_topp", "hk_pool_max",
            "hk_score_rows", "hk_vote_topp", "hk_budget_plan", "hk_budget_select",
            "hk_compact_modes", "hk_calibrate_solve_T_gd", "hk_alloc_init", "hk_compress",
            "hk_probe", "hk_decode_plan", "hk_decode_attn_noalloc", "hk_decode_noalloc_scratch_bytes",
            "hk_select_workspace_size", "hk_topp_select_ws", "hk_calibrate_topp_ws"]
# kernel ids of hk_timing_read, in header order
TIMED_KERNELS = ["score_pass1", "score_merge", "score_pass2", "calibrate", "topp", "solve_T",
                 "compact_gather", "compact_meta", "decode_split", "decode_merge", "append",
                 "calib_topp", "score_rows", "vote", "vote_count", "budget_plan", "budget_select"]


class HardKVError(RuntimeError):
    pass


class hk_dims(C.Structure):
    _fields_ = [("NS", C.c_int32), ("Hq", C.c_int32), ("Hkv", C.c_int32), ("D", C.c_int32),
                ("W", C.c_int32)]


class hk_paged_kv(C.Structure):
    _fields_ = [("k_pool", C.c_void_p), ("v_pool", C.c_void_p), ("page_table", C.c_void_p),
                ("page_mask", C.c_void_p), ("n_pages", C.c_void_p), ("num_pages", C.c_int32),
                ("max_pages", C.c_int32), ("dtype", C.c_int32)]


class hk_allocator(C.Structure):
    _fields_ = [("free_ids", C.c_void_p), ("free_top", C.c_void_p), ("capacity", C.c_int32)]


_lib = None


def lib():
    """Load libhardkv.so (built in-tree by paper_2606_28831_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise HardKVError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2606_28831_amd.build` (no fallback exists)")
        L = C.CDLL(LIB_PATH)
        P, I32, SZ, F, D = C.c_void_p, C.c_int32, C.c_size_t, C.c_float, C.c_double
        L.hk_workspace_size.restype = SZ
        L.hk_workspace_size.argtypes = [I32, C.POINTER(hk_dims), I32]
        L.hk_status_string.restype = C.c_char_p
        L.hk_status_string.argtypes = [I32, I32]
        L.hk_score.restype = I32
        L.hk_score.argtypes = [C.POINTER(hk_dims), P, C.POINTER(hk_paged_kv), I32, F, P, P, P, P,
                               P, I32, P, P, SZ, P]
        L.hk_calibrate.restype = I32
        L.hk_calibrate.argtypes = [I32, I32, P, P, I32, C.POINTER(C.c_void_p),
                                   C.POINTER(C.c_void_p), C.POINTER(C.c_float), P, P, P]
        L.hk_topp_select.restype = I32
        L.hk_topp_select.argtypes = [I32, I32, P, P, P, D, I32, I32, P, P, P, P, P]
        L.hk_calibrate_solve_T.restype = I32
        L.hk_calibrate_solve_T.argtypes = [I32, I32, P, P, P, P, P, F, F, I32, P, P]
        L.hk_compact.restype = I32
        L.hk_compact.argtypes = [C.POINTER(hk_dims), C.POINTER(hk_paged_kv), P, I32, I32,
                                 C.POINTER(hk_allocator), P, P, SZ, P]
        L.hk_decode_attn.restype = I32
        L.hk_decode_attn.argtypes = [C.POINTER(hk_dims), P, C.POINTER(hk_paged_kv), F, P, P, P,
                                     SZ, P]
        L.hk_append_kv.restype = I32
        L.hk_append_kv.argtypes = [C.POINTER(hk_dims), C.POINTER(hk_paged_kv), P, P,
                                   C.POINTER(hk_allocator), P, P, SZ, P]
        L.hk_calibrate_topp.restype = I32
        L.hk_calibrate_topp.argtypes = [I32, I32, P, P, I32, C.POINTER(C.c_void_p),
                                        C.POINTER(C.c_void_p), C.POINTER(C.c_float), D, I32, I32,
                                        P, P, P, P, P, P, P]
        L.hk_select_workspace_size.restype = SZ
        L.hk_select_workspace_size.argtypes = [I32, I32]
        L.hk_topp_select_ws.restype = I32
        L.hk_topp_select_ws.argtypes = [I32, I32, P, P, P, D, I32, I32, P, P, P, P, P, SZ, P]
        L.hk_calibrate_topp_ws.restype = I32
        L.hk_calibrate_topp_ws.argtypes = [I32, I32, P, P, I32, C.POINTER(C.c_void_p),
                                           C.POINTER(C.c_void_p), C.POINTER(C.c_float), D, I32,
                                           I32, P, P, P, P, P, P, P, SZ, P]
        L.hk_pool_max.restype = I32
        L.hk_pool_max.argtypes = [I32, I32, P, P, P, I32, P, P]
        L.hk_score_rows.restype = I32
        L.hk_score_rows.argtypes = [C.POINTER(hk_dims), P, C.POINTER(hk_paged_kv), I32, F, P, P, P]
        L.hk_vote_topp.restype = I32
        L.hk_vote_topp.argtypes = [I32, I32, I32, P, P, P, D, P, P, P, P, P]
        L.hk_budget_plan.restype = I32
        L.hk_budget_plan.argtypes = [C.POINTER(hk_dims), C.POINTER(hk_paged_kv), I32, I32, I32, P,
                                     P, P]
        L.hk_budget_select.restype = I32
        L.hk_budget_select.argtypes = [I32, I32, P, P, P, P, P, P, P, I32, P, P, P]
        L.hk_compact_modes.restype = I32
        L.hk_compact_modes.argtypes = [C.POINTER(hk_dims), C.POINTER(hk_paged_kv), P, I32, P,
                                       C.POINTER(hk_allocator), P, P, C.c_size_t, P]
        L.hk_calibrate_solve_T_gd.restype = I32
        L.hk_calibrate_solve_T_gd.argtypes = [I32, I32, P, P, P, P, P, F, F, I32, F, P, P, P]
        L.hk_alloc_init.restype = I32
        L.hk_alloc_init.argtypes = [C.POINTER(hk_allocator), I32, I32, P]
        L.hk_compress.restype = I32
        L.hk_compress.argtypes = [C.POINTER(hk_dims), P, C.POINTER(hk_paged_kv), I32, I32, F, P, D,
                                  I32, I32, C.POINTER(hk_allocator), P, P, P, P, SZ, P]
        L.hk_decode_attn_noalloc.restype = I32
        L.hk_decode_attn_noalloc.argtypes = [C.POINTER(hk_dims), P, C.POINTER(hk_paged_kv), F, P, P, P]
        L.hk_decode_noalloc_scratch_bytes.restype = SZ
        L.hk_decode_noalloc_scratch_bytes.argtypes = [C.POINTER(hk_dims), I32]
        L.hk_decode_plan.restype = I32
        L.hk_decode_plan.argtypes = [C.POINTER(hk_dims), I32, C.POINTER(I32), C.POINTER(I32)]
        L.hk_probe.restype = I32
        L.hk_probe.argtypes = [I32, I32, I32, P, P]
        L.hk_timing_enable.restype = I32
        L.hk_timing_enable.argtypes = [C.c_uint32]
        L.hk_timing_read.restype = I32
        L.hk_timing_read.argtypes = [I32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
        _lib = L
    return _lib


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor")
    if not t.is_contiguous():
        raise HardKVError("tensor arguments must be contiguous")
    return C.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _check(code: int, name: str):
    if code != 0:
        msg = lib().hk_status_string(code, 0).decode()
        raise HardKVError(f"{name}: {msg}")


def hk_status_string(code: int, flags: bool = False) -> str:
    return lib().hk_status_string(int(code), int(bool(flags))).decode()


def dims(NS, Hq, Hkv, D, W=0) -> hk_dims:
    return hk_dims(int(NS), int(Hq), int(Hkv), int(D), int(W))


class PagedKV:
    """Device tensors of one paged Cascade Cache plus its C descriptor."""

    def __init__(self, k_pool, v_pool, page_table, page_mask, n_pages):
        self.k_pool, self.v_pool = k_pool, v_pool
        self.page_table, self.page_mask, self.n_pages = page_table, page_mask, n_pages
        if k_pool.dtype == torch.bfloat16:
            dt = HK_BF16
        elif k_pool.dtype == torch.float32:
            dt = HK_F32
        else:
            raise HardKVError("cache dtype must be bfloat16 or float32")
        self.desc = hk_paged_kv(k_pool.data_ptr(), v_pool.data_ptr() if v_pool is not None else None,
                                page_table.data_ptr(), page_mask.data_ptr(), n_pages.data_ptr(),
                                k_pool.shape[0], page_table.shape[1], dt)

    def rows(self, first_head: int, n_heads: int) -> "PagedKV":
        """A view of heads [first_head, first_head + n_heads) (e.g. one layer)."""
        sl = slice(first_head, first_head + n_heads)
        return PagedKV(self.k_pool, self.v_pool, self.page_table[sl], self.page_mask[sl],
                       self.n_pages[sl])

    @property
    def max_pages(self):
        return self.page_table.shape[1]


class Allocator:
    def __init__(self, free_ids, free_top):
        self.free_ids, self.free_top = free_ids, free_top
        self.desc = hk_allocator(free_ids.data_ptr(), free_top.data_ptr(), free_ids.shape[0])


def hk_workspace_size(op: int, d: hk_dims, max_pages: int) -> int:
    return int(lib().hk_workspace_size(int(op), C.byref(d), int(max_pages)))


def workspace(op: int, d: hk_dims, max_pages: int, device) -> torch.Tensor:
    n = max(256, hk_workspace_size(op, d, max_pages))
    return torch.empty(n, dtype=torch.uint8, device=device)


def hk_score(d: hk_dims, q_obs, kv: PagedKV, L_dense: int, sm_scale: float, s_attn, cand_len,
             row_lse_in=None, row_lse_out=None, ref_slots=None, n_ref: int = 0, x_red=None,
             ws=None, stream=None):
    _check(lib().hk_score(C.byref(d), _ptr(q_obs), C.byref(kv.desc), int(L_dense),
                          float(sm_scale), _ptr(row_lse_in), _ptr(row_lse_out), _ptr(s_attn),
                          _ptr(cand_len), _ptr(ref_slots), int(n_ref), _ptr(x_red), _ptr(ws),
                          ws.numel() if ws is not None else 0, _stream(stream)), "hk_score")


def hk_calibrate(n_heads: int, S_max: int, cand_len, page_mask, xs, Ts, weights, c_out,
                 lse_out=None, stream=None):
    m = len(xs)
    xa = (C.c_void_p * m)(*[t.data_ptr() for t in xs])
    Ta = None
    if Ts is not None:
        Ta = (C.c_void_p * m)(*[(t.data_ptr() if t is not None else None) for t in Ts])
    wa = (C.c_float * m)(*[float(w) for w in weights])
    _check(lib().hk_calibrate(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask), m, xa,
                              Ta, wa, _ptr(c_out), _ptr(lse_out), _stream(stream)), "hk_calibrate")


def hk_topp_select(n_heads: int, S_max: int, cand_len, page_mask, c, p: float, sel_bits, k_out,
                   k_min: int = 1, k_max: int = 0, sel_mass=None, status=None, stream=None):
    _check(lib().hk_topp_select(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask), _ptr(c),
                                float(p), int(k_min), int(k_max), _ptr(sel_bits), _ptr(k_out),
                                _ptr(sel_mass), _ptr(status), _stream(stream)), "hk_topp_select")


def hk_calibrate_topp(n_heads: int, S_max: int, cand_len, page_mask, xs, Ts, weights, p: float,
                      sel_bits, k_out, c_out=None, lse_out=None, k_min: int = 1, k_max: int = 0,
                      sel_mass=None, status=None, stream=None):
    m = len(xs)
    xa = (C.c_void_p * m)(*[t.data_ptr() for t in xs])
    Ta = None
    if Ts is not None:
        Ta = (C.c_void_p * m)(*[(t.data_ptr() if t is not None else None) for t in Ts])
    wa = (C.c_float * m)(*[float(w) for w in weights])
    _check(lib().hk_calibrate_topp(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask), m,
                                   xa, Ta, wa, float(p), int(k_min), int(k_max), _ptr(c_out),
                                   _ptr(lse_out), _ptr(sel_bits), _ptr(k_out), _ptr(sel_mass),
                                   _ptr(status), _stream(stream)), "hk_calibrate_topp")


def hk_select_workspace_size(n_heads: int, S_max: int) -> int:
    return int(lib().hk_select_workspace_size(int(n_heads), int(S_max)))


def select_workspace(n_heads: int, S_max: int, device) -> torch.Tensor:
    """Workspace of hk_topp_select_ws / hk_calibrate_topp_ws for these sizes."""
    n = max(256, hk_select_workspace_size(n_heads, S_max))
    return torch.empty(n, dtype=torch.uint8, device=device)


def hk_topp_select_ws(n_heads: int, S_max: int, cand_len, page_mask, c, p: float, sel_bits, k_out,
                      ws, k_min: int = 1, k_max: int = 0, sel_mass=None, status=None, stream=None):
    _check(lib().hk_topp_select_ws(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask),
                                   _ptr(c), float(p), int(k_min), int(k_max), _ptr(sel_bits),
                                   _ptr(k_out), _ptr(sel_mass), _ptr(status), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)),
           "hk_topp_select_ws")


def hk_calibrate_topp_ws(n_heads: int, S_max: int, cand_len, page_mask, xs, Ts, weights, p: float,
                         sel_bits, k_out, ws, c_out=None, lse_out=None, k_min: int = 1,
                         k_max: int = 0, sel_mass=None, status=None, stream=None):
    m = len(xs)
    xa = (C.c_void_p * m)(*[t.data_ptr() for t in xs])
    Ta = None
    if Ts is not None:
        Ta = (C.c_void_p * m)(*[(t.data_ptr() if t is not None else None) for t in Ts])
    wa = (C.c_float * m)(*[float(w) for w in weights])
    _check(lib().hk_calibrate_topp_ws(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask),
                                      m, xa, Ta, wa, float(p), int(k_min), int(k_max),
                                      _ptr(c_out), _ptr(lse_out), _ptr(sel_bits), _ptr(k_out),
                                      _ptr(sel_mass), _ptr(status), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream(stream)),
           "hk_calibrate_topp_ws")


def hk_pool_max(n_heads: int, S_max: int, cand_len, page_mask, x, radius: int, x_out, stream=None):
    _check(lib().hk_pool_max(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask), _ptr(x),
                             int(radius), _ptr(x_out), _stream(stream)), "hk_pool_max")


def hk_calibrate_solve_T(n_heads: int, S_max: int, cand_len, page_mask, x, k, target_mass, T_out,
                         T_lo: float = 1e-4, T_hi: float = 1e4, iters: int = 40, stream=None):
    _check(lib().hk_calibrate_solve_T(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask),
                                      _ptr(x), _ptr(k), _ptr(target_mass), float(T_lo),
                                      float(T_hi), int(iters), _ptr(T_out), _stream(stream)),
           "hk_calibrate_solve_T")


def hk_calibrate_solve_T_gd(n_heads: int, S_max: int, cand_len, page_mask, x, k, target_mass,
                            T_out, T_init: float = 1.0, lr: float = 0.05, iters: int = 200,
                            tol: float = 0.0, loss_out=None, stream=None):
    _check(lib().hk_calibrate_solve_T_gd(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask),
                                         _ptr(x), _ptr(k), _ptr(target_mass), float(T_init),
                                         float(lr), int(iters), float(tol), _ptr(T_out),
                                         _ptr(loss_out), _stream(stream)), "hk_calibrate_solve_T_gd")


def hk_compress(d: hk_dims, q_obs, kv: PagedKV, L_dense: int, L_sparse: int, sm_scale: float,
                p: float, alloc: Allocator, k_out, ws, status=None, sel_bits_out=None,
                row_lse_in=None, k_min: int = 1, k_max: int = 0, stream=None):
    _check(lib().hk_compress(C.byref(d), _ptr(q_obs), C.byref(kv.desc), int(L_dense), int(L_sparse),
                             float(sm_scale), _ptr(row_lse_in), float(p), int(k_min), int(k_max),
                             C.byref(alloc.desc), _ptr(sel_bits_out), _ptr(k_out), _ptr(status),
                             _ptr(ws), ws.numel(), _stream(stream)), "hk_compress")


def hk_alloc_init(alloc: Allocator, first_free: int, num_pages: int, stream=None):
    _check(lib().hk_alloc_init(C.byref(alloc.desc), int(first_free), int(num_pages),
                               _stream(stream)), "hk_alloc_init")


def hk_compact(d: hk_dims, kv: PagedKV, sel_bits, L_dense: int, L_sparse: int, alloc: Allocator,
               status, ws, stream=None):
    _check(lib().hk_compact(C.byref(d), C.byref(kv.desc), _ptr(sel_bits), int(L_dense),
                            int(L_sparse), C.byref(alloc.desc), _ptr(status), _ptr(ws), ws.numel(),
                            _stream(stream)), "hk_compact")


def hk_decode_attn(d: hk_dims, q, kv: PagedKV, sm_scale: float, o, lse, ws, stream=None):
    _check(lib().hk_decode_attn(C.byref(d), _ptr(q), C.byref(kv.desc), float(sm_scale), _ptr(o),
                                _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)), "hk_decode_attn")


def hk_decode_attn_noalloc(d: hk_dims, q, kv: PagedKV, sm_scale: float, o, lse, stream=None):
    """hk_decode_attn with the split states in the library's static scratch (no workspace)."""
    _check(lib().hk_decode_attn_noalloc(C.byref(d), _ptr(q), C.byref(kv.desc), float(sm_scale),
                                        _ptr(o), _ptr(lse), _stream(stream)), "hk_decode_attn_noalloc")


def hk_decode_noalloc_scratch_bytes(d: hk_dims, max_pages: int) -> int:
    return int(lib().hk_decode_noalloc_scratch_bytes(C.byref(d), int(max_pages)))


def hk_decode_plan(d: hk_dims, max_pages: int):
    """(n_split, pages_per_split) that hk_decode_attn uses for these dims and table width."""
    ns, pps = C.c_int32(0), C.c_int32(0)
    _check(lib().hk_decode_plan(C.byref(d), int(max_pages), C.byref(ns), C.byref(pps)),
           "hk_decode_plan")
    return ns.value, pps.value


def hk_append_kv(d: hk_dims, kv: PagedKV, k_new, v_new, alloc: Allocator, status, ws,
                 stream=None):
    _check(lib().hk_append_kv(C.byref(d), C.byref(kv.desc), _ptr(k_new), _ptr(v_new),
                              C.byref(alloc.desc), _ptr(status), _ptr(ws),
                              ws.numel() if ws is not None else 0, _stream(stream)), "hk_append_kv")


def hk_score_rows(d: hk_dims, q_obs, kv: PagedKV, L_dense: int, sm_scale: float, row_lse, a_rows,
                  stream=None):
    _check(lib().hk_score_rows(C.byref(d), _ptr(q_obs), C.byref(kv.desc), int(L_dense),
                               float(sm_scale), _ptr(row_lse), _ptr(a_rows), _stream(stream)),
           "hk_score_rows")


def hk_vote_topp(n_heads: int, R: int, S_max: int, cand_len, page_mask, a_rows, p: float, votes,
                 row_sel, row_k=None, status=None, stream=None):
    _check(lib().hk_vote_topp(int(n_heads), int(R), int(S_max), _ptr(cand_len), _ptr(page_mask),
                              _ptr(a_rows), float(p), _ptr(votes), _ptr(row_sel), _ptr(row_k),
                              _ptr(status), _stream(stream)), "hk_vote_topp")


def hk_budget_plan(d: hk_dims, kv: PagedKV, L_dense: int, L_lower: int, L_upper: int, head_mode,
                   k_cap, stream=None):
    _check(lib().hk_budget_plan(C.byref(d), C.byref(kv.desc), int(L_dense), int(L_lower),
                                int(L_upper), _ptr(head_mode), _ptr(k_cap), _stream(stream)),
           "hk_budget_plan")


def hk_budget_select(n_heads: int, S_max: int, cand_len, page_mask, sel_out, k_out, votes=None,
                     c=None, sel_in=None, head_mode=None, k_cap=None, n_sink: int = 0,
                     stream=None):
    _check(lib().hk_budget_select(int(n_heads), int(S_max), _ptr(cand_len), _ptr(page_mask),
                                  _ptr(votes), _ptr(c), _ptr(sel_in), _ptr(head_mode), _ptr(k_cap),
                                  int(n_sink), _ptr(sel_out), _ptr(k_out), _stream(stream)),
           "hk_budget_select")


def hk_compact_modes(d: hk_dims, kv: PagedKV, sel_bits, L_dense: int, head_mode, alloc: Allocator,
                     status, ws, stream=None):
    _check(lib().hk_compact_modes(C.byref(d), C.byref(kv.desc), _ptr(sel_bits), int(L_dense),
                                  _ptr(head_mode), C.byref(alloc.desc), _ptr(status), _ptr(ws),
                                  ws.numel(), _stream(stream)), "hk_compact_modes")


def hk_timing_enable(kernels=None):
    """Time the launches of the named kernels (all of them for kernels=None; [] turns
    timing off)."""
    names = TIMED_KERNELS if kernels is None else kernels
    mask = 0
    for k in names:
        mask |= 1 << TIMED_KERNELS.index(k)
    _check(lib().hk_timing_enable(mask), "hk_timing_enable")


def hk_probe(kind: int, blocks: int, iters: int, out, stream=None):
    """One rate-probe launch (a PROBE_* kind); out: >= 256 * blocks floats."""
    _check(lib().hk_probe(int(kind), int(blocks), int(iters), _ptr(out), _stream(stream)),
           "hk_probe")


def hk_timing_read(kernel: str):
    """(summed ms, launches) of one timed kernel since the previous read; clears them."""
    ms, n = C.c_double(0.0), C.c_int64(0)
    _check(lib().hk_timing_read(TIMED_KERNELS.index(kernel), C.byref(ms), C.byref(n)),
           "hk_timing_read")
    return ms.value, n.value

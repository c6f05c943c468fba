"""hk_decode_attn_noalloc -- decode attention for callers that cannot allocate -- against
hk_decode_attn on the same inputs, called through the C ABI: bit for bit on two calls in a
row, the second with a smaller input (fewer heads, another dtype and head dim, a narrower
table), so the static scratch holding the first call's split states must not leak into the
second.  The first call has a config-5 layer's shape (64 sequences x 8 KV heads, G 4, D 128,
768-page table: the 128-page split)."""
import ctypes as C
import math

import pytest
import torch

import workload as WL

pytestmark = pytest.mark.gpu
DEV = "cuda"

CASES = [
    (dict(L=1, B=64, Hq=32, Hkv=8, D=128, N=3000, dtype="bf16", W=1, seed=51, recipe="normal"),
     dict(max_pages=768, hole_prob=0.05)),
    (dict(L=1, B=3, Hq=8, Hkv=2, D=64, N=300, dtype="f32", W=1, seed=52, recipe="normal"),
     dict(max_pages=40, hole_prob=0.2)),
]


def test_noalloc_decode_equals_workspace_decode():
    import paper_2606_28831_amd as hk
    L = hk.lib()
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i, (cfg, kw) in enumerate(CASES):
        w = WL.make_workload(cfg, DEV, **kw)
        kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
        Hq, D = cfg["Hq"], cfg["D"]
        d = hk.dims(w.NS, Hq, cfg["Hkv"], D)
        need = hk.hk_decode_noalloc_scratch_bytes(d, w.max_pages)
        assert 0 < need <= 16 << 20
        g = torch.Generator(device=DEV).manual_seed(60 + i)
        q = torch.randn(w.NS, Hq, D, generator=g, device=DEV).to(w.k_pool.dtype)
        scale = 1 / math.sqrt(D)
        o_ref = torch.full((w.NS, Hq, D), float("nan"), device=DEV)
        lse_ref = torch.full((w.NS, Hq), float("nan"), device=DEV)
        hk.hk_decode_attn(d, q, kv, scale, o_ref, lse_ref, hk.workspace(hk.OP_DECODE, d, w.max_pages, DEV))
        o = torch.full_like(o_ref, float("nan"))
        lse = torch.full_like(lse_ref, float("nan"))
        rc = L.hk_decode_attn_noalloc(C.byref(d), C.c_void_p(q.data_ptr()), C.byref(kv.desc),
                                      C.c_float(scale), C.c_void_p(o.data_ptr()),
                                      C.c_void_p(lse.data_ptr()), st)
        assert rc == 0, hk.hk_status_string(rc)
        torch.cuda.synchronize()
        assert torch.isfinite(o_ref).all() and torch.isfinite(lse_ref).all()
        assert torch.equal(o, o_ref) and torch.equal(lse, lse_ref), f"call {i}"

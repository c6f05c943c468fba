"""End-to-end decode loop (append + paged decode + periodic compression) against an
independent host replay.

The host keeps, per head, the valid K/V rows in logical order.  Every decode step the
oracle's attention over that replay is compared with the GPU output; every compression
the GPU score (single pass, fed the GPU's decode LSEs) is compared with the oracle score
fed the oracle's own decode LSEs; the GPU Top-p selection, made on the GPU's own
probabilities, must satisfy the Top-p rule's defining properties (the stage's parity on
seeded inputs is tested on its own); the replay then keeps the selected rows, and after
the rewrite the GPU cache must hold exactly the replay's rows (bit-exact).
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workload as WL
from hk_testlib import (HostCache, check_lse, check_log_scores, check_prob, check_topp_rule, np64,
                        np_i, unpack_bits)

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _valid_rows(host: HostCache, h):
    K, valid = host.head(h)
    V, _ = host.head_v(h)
    return K[valid], V[valid], valid


@pytest.mark.parametrize("L_dense", [48, 0])
def test_decode_loop_chain(L_dense):
    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import DecodeLoop

    L, B, Hq, Hkv, D, W, T, n_seg, p = 2, 2, 8, 2, 128, 8, 32, 3, 0.9
    G, NS, H = Hq // Hkv, L * B, L * B * Hkv
    cfg = dict(L=L, B=B, Hq=Hq, Hkv=Hkv, D=D, N=200, dtype="bf16", W=W, seed=21, recipe="normal")
    w = WL.make_workload(cfg, DEV, max_pages=20, pool_slack=3.0)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    loop = DecodeLoop(L, B, Hq, Hkv, D, W, kv, alloc, p, L_dense)
    scale = 1 / math.sqrt(D)

    host0 = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    rows = {h: list(_valid_rows(host0, h)[:2]) for h in range(H)}
    for seg in range(n_seg):
        g = torch.Generator(device=DEV).manual_seed(100 + seg)
        q_seg = torch.randn(T, NS, Hq, D, generator=g, device=DEV).to(torch.bfloat16)
        k_seg = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(torch.bfloat16)
        v_seg = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(torch.bfloat16)
        lse_seg = torch.empty(T, NS, Hq, device=DEV)
        qn, kn, vn = np64(q_seg), np64(k_seg), np64(v_seg)
        oracle_lse = np.zeros((T, NS, Hq))
        for t in range(T):
            loop.step(q_seg[t], k_seg[t], v_seg[t], lse_seg[t])
            torch.cuda.synchronize()
            on, ln = np64(loop.o), np64(lse_seg[t])
            for h in range(H):
                s, kvh = divmod(h, Hkv)
                rows[h][0] = np.vstack([rows[h][0], kn[t, s, kvh][None]])
                rows[h][1] = np.vstack([rows[h][1], vn[t, s, kvh][None]])
                Kh, Vh = rows[h]
                o_ref, l_ref = O.decode_head(qn[t, s, kvh * G:(kvh + 1) * G], Kh, Vh,
                                             np.ones(len(Kh), bool), scale)
                oracle_lse[t, s, kvh * G:(kvh + 1) * G] = l_ref
                for gi in range(G):
                    check_prob(on[s, kvh * G + gi], o_ref[gi], 2e-3, f"o seg {seg} t {t} h {h}")
                check_lse(ln[s, kvh * G:(kvh + 1) * G], l_ref, 2e-3, f"lse seg {seg} t {t} h {h}")
        assert int(loop.status.item()) == 0
        # ---- compression
        pre = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
        for h in range(H):   # the GPU cache holds exactly the replay before compressing
            Kg, Vg, _ = _valid_rows(pre, h)
            assert np.array_equal(Kg, rows[h][0]) and np.array_equal(Vg, rows[h][1]), (seg, h)
        loop.compress(q_seg[T - W:], lse_seg[T - W:])
        torch.cuda.synchronize()
        b = loop.comp.buf
        s_gpu, c_gpu, sel_gpu, k_gpu = np64(b.s_attn), b.c.cpu().numpy(), np_i(b.sel_bits), np_i(b.k)
        S = w.S_max
        for h in range(H):
            s, kvh = divmod(h, Hkv)
            n = int(pre.n[h])
            _, valid = pre.head(h)
            nd = O.tier_pages(n, L_dense, 0)[2]
            cand_len = 16 * (n - nd)
            q_rows = qn[T - W:, s, kvh * G:(kvh + 1) * G].reshape(-1, D)
            lse_rows = oracle_lse[T - W:, s, kvh * G:(kvh + 1) * G].reshape(-1)
            Kfull, _ = pre.head(h)
            s_ref, _ = O.score_head(q_rows, Kfull, valid, cand_len, scale, row_lse_in=lse_rows)
            full = np.full(S, -np.inf)
            full[:len(s_ref)] = s_ref
            check_log_scores(s_gpu[h], full, 2e-3, f"score seg {seg} h {h}")
            cand = np.zeros(S, bool)
            cand[:len(valid)] = O.candidate_mask(valid, cand_len)
            sel = unpack_bits(sel_gpu[h], S)
            check_topp_rule(c_gpu[h], sel, int(k_gpu[h]), cand, p, what=f"seg {seg} h {h}")
            # replay: selected candidates, then every dense-tier row, in order
            keep = (sel[:len(valid)] | ~O.candidate_mask(valid, cand_len))[valid]
            rows[h] = [rows[h][0][keep], rows[h][1][keep]]
        post = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
        for h in range(H):
            Kg, Vg, _ = _valid_rows(post, h)
            assert np.array_equal(Kg, rows[h][0]) and np.array_equal(Vg, rows[h][1]), (seg, h)
        assert int(b.status.item()) == 0

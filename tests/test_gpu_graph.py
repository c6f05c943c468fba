"""The config-5 style decode segment (append + per-layer paged decode for every step, then
one compression) recorded once into a HIP graph and replayed over fresh inputs gives the
same results, bit for bit, as the same segments run eagerly: outputs, LSEs, tables, masks,
page counts, allocator and pool contents.  The replays are interleaved with eager work
(input refills) and synchronisations, and every replay is checked."""
import pytest
import torch

import workload as WL

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _loop(hk, DecodeLoop, cfg, L, B, Hq, Hkv, D, W, L_dense):
    w = WL.make_workload(cfg, DEV, max_pages=24, pool_slack=3.0)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    return w, DecodeLoop(L, B, Hq, Hkv, D, W, kv, alloc, 0.9, L_dense)


def test_graph_replay_equals_eager():
    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import DecodeLoop

    L, B, Hq, Hkv, D, W, T, n_seg = 2, 2, 8, 2, 128, 8, 32, 4
    NS = L * B
    cfg = dict(L=L, B=B, Hq=Hq, Hkv=Hkv, D=D, N=200, dtype="bf16", W=W, seed=41, recipe="normal")
    wa, eager = _loop(hk, DecodeLoop, cfg, L, B, Hq, Hkv, D, W, 48)
    wb, graphed = _loop(hk, DecodeLoop, cfg, L, B, Hq, Hkv, D, W, 48)
    bf = torch.bfloat16
    qb = torch.empty(T, NS, Hq, D, device=DEV, dtype=bf)
    kb = torch.empty(T, NS, Hkv, D, device=DEV, dtype=bf)
    vb = torch.empty(T, NS, Hkv, D, device=DEV, dtype=bf)
    lb = torch.empty(T, NS, Hq, device=DEV)
    graph = None
    for seg in range(n_seg):
        g = torch.Generator(device=DEV).manual_seed(500 + seg)
        q = torch.randn(T, NS, Hq, D, generator=g, device=DEV).to(bf)
        k = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf)
        v = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf)
        la = torch.empty(T, NS, Hq, device=DEV)
        eager.segment(q, k, v, la)
        qb.copy_(q)
        kb.copy_(k)
        vb.copy_(v)
        torch.cuda.synchronize()
        if graph is None:
            graph = graphed.capture_segment(qb, kb, vb, lb)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(eager.o, graphed.o), seg
        assert torch.equal(la, lb), seg
        for name in ("page_table", "page_mask", "n_pages", "free_top", "k_pool", "v_pool"):
            assert torch.equal(getattr(wa, name), getattr(wb, name)), (seg, name)
        top = int(wa.free_top.item())
        assert torch.equal(wa.free_ids[:top], wb.free_ids[:top]), seg
        assert torch.equal(eager.comp.buf.sel_bits, graphed.comp.buf.sel_bits), seg
    assert int(eager.status.item()) == int(graphed.status.item()) == 0


def test_graph_replay_matches_oracle():
    """Graph-replayed segments against the oracle, not only against eager runs: a host model
    of every head (tests/hk_testlib.DecodeReplay) checks every step's LSE (the graph's LSE
    buffer holds the whole segment), the last step's decode output, the compression's scores
    and selection, and the rewritten cache (page counts, masks, K/V bytes) after each of four
    replays over fresh inputs, with eager refills and synchronisations between them."""
    import math

    import numpy as np

    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import DecodeLoop
    from hk_testlib import DecodeReplay, check_lse, check_prob, np64, np_i

    L, B, Hq, Hkv, D, W, T, n_seg, L_dense, p = 2, 2, 8, 2, 128, 8, 32, 4, 48, 0.9
    G, NS, H = Hq // Hkv, L * B, L * B * Hkv
    cfg = dict(L=L, B=B, Hq=Hq, Hkv=Hkv, D=D, N=200, dtype="bf16", W=W, seed=43, recipe="normal")
    w, loop = _loop(hk, DecodeLoop, cfg, L, B, Hq, Hkv, D, W, L_dense)
    model = DecodeReplay(w, range(H), Hkv, G, D, 1 / math.sqrt(D), w.max_pages)
    bf = torch.bfloat16
    qb = torch.empty(T, NS, Hq, D, device=DEV, dtype=bf)
    kb = torch.empty(T, NS, Hkv, D, device=DEV, dtype=bf)
    vb = torch.empty(T, NS, Hkv, D, device=DEV, dtype=bf)
    lb = torch.empty(T, NS, Hq, device=DEV)
    graph = loop.capture_segment(qb, kb, vb, lb)     # records only; nothing runs yet
    torch.cuda.synchronize()
    model.check_cache(w, "after capture")
    for seg in range(n_seg):
        g = torch.Generator(device=DEV).manual_seed(900 + seg)
        qb.copy_(torch.randn(T, NS, Hq, D, generator=g, device=DEV).to(bf))
        kb.copy_(torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf))
        vb.copy_(torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf))
        torch.cuda.synchronize()
        qn, kn, vn = np64(qb), np64(kb), np64(vb)
        graph.replay()
        torch.cuda.synchronize()
        ref_lse = {h: np.zeros((T, G)) for h in range(H)}
        for t in range(T):
            ref = model.step(qn[t], kn[t], vn[t])
            for h in range(H):
                ref_lse[h][t] = ref[h][1]
        on, ln = np64(loop.o), np64(lb)
        for h in range(H):
            s, kvh = divmod(h, Hkv)
            check_lse(ln[:, s, kvh * G:(kvh + 1) * G], ref_lse[h], 2e-3, f"graph lse seg {seg} head {h}")
            for gi in range(G):
                check_prob(on[s, kvh * G + gi], ref[h][0][gi], 2e-3, f"graph o seg {seg} head {h}")
        b = loop.comp.buf
        assert int(loop.status.item()) == 0 and int(b.status.item()) == 0
        rows = lambda t_: {h: t_[h].cpu().numpy() for h in range(H)}
        model.compress(qn[T - W:], {h: ref_lse[h][T - W:] for h in range(H)},
                       {h: np64(b.s_attn[h]) for h in range(H)}, rows(b.c), rows(b.sel_bits),
                       np_i(b.k), L_dense, p, w.S_max, f"graph seg {seg}")
        model.check_cache(w, f"graph seg {seg} after the rewrite")

"""Config 5 at its own shape: 32 layers x batch 64, 32 query / 8 KV heads, head_dim 128,
bf16, an 8192-token prompt per head, compression every 128 decode steps at Top-p 0.9 with a
512-token dense tier -- the cache, table width and launches bench.py runs.  Two whole
segments of the decode loop (append + per-layer paged decode attention every step, then
one compression of every layer, Sec. 3.1 Steps 1-3) are checked on sampled heads against a
host replay with the oracle: decode outputs at sampled steps and LSEs at every step (App. F
attention and merge), the single-pass scores over the decode LSEs at each compression, the
selection by the Top-p rule on the GPU's own probabilities, and the rewritten cache rows
byte for byte.  The decode launches must take the 128-page split that the chip-filling rule
picks for 512 heads per layer over a 768-page table.  After each segment's appends and each
rewrite, every page of the pool is listed once or free, never both (all 16384 heads)."""
import math

import numpy as np
import pytest
import torch

import workload as WL
from hk_testlib import DecodeReplay, check_lse, check_prob, np64, np_i

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _check_pages_conserved(w, what):
    """Every page of the pool is either listed once in some head's table (below its page
    count) or on the free list below its top, never both and never twice."""
    tab, n = np_i(w.page_table), np_i(w.n_pages)
    used = tab[np.arange(tab.shape[1])[None, :] < n[:, None]]
    free = np_i(w.free_ids)[:int(np_i(w.free_top).reshape(-1)[0])]
    assert len(np.unique(used)) == len(used), f"{what}: a page listed twice"
    assert len(np.unique(free)) == len(free), f"{what}: a page free twice"
    assert len(np.intersect1d(used, free)) == 0, f"{what}: a listed page is also free"
    assert len(used) + len(free) == w.k_pool.shape[0], f"{what}: pages lost"


@pytest.mark.timeout(900)
def test_config5_two_segments_sampled_heads():
    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import DecodeLoop

    cfg = WL.config(5)
    L, B, Hq, Hkv, D, W = (cfg[k] for k in ("L", "B", "Hq", "Hkv", "D", "W"))
    T, p, L_dense = cfg["compress_every"], cfg["p"], cfg["L_dense"]
    G, NS, H = Hq // Hkv, L * B, L * B * Hkv
    max_pages = (cfg["N"] + cfg["decode_steps"]) // 16
    w = WL.make_workload(cfg, DEV, max_pages=max_pages, pool_pages=H * max_pages + H * 256)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    loop = DecodeLoop(L, B, Hq, Hkv, D, W, kv, alloc, p, L_dense)
    # the launch shape: 6 splits of at most 128 pages per head, 512 heads per layer
    assert hk.hk_decode_plan(loop.d_layer, w.max_pages) == (6, 128)
    scale = 1 / math.sqrt(D)
    rng = np.random.default_rng(5)
    heads = sorted({0, H - 1} | {int(x) for x in rng.choice(H, size=6, replace=False)})
    seqs = sorted({h // Hkv for h in heads})
    sidx = {s: i for i, s in enumerate(seqs)}
    seq_t = torch.tensor(seqs, device=DEV)
    replay = DecodeReplay(w, heads, Hkv, G, D, scale, w.max_pages)
    print(f"config 5: cache ready, heads {heads}", flush=True)
    o_steps = {0, 1, 63, T - 1}
    bf = torch.bfloat16
    for seg in range(2):
        g = torch.Generator(device=DEV).manual_seed(cfg["seed"] * 7919 + seg + 1)
        q_seg = torch.randn(T, NS, Hq, D, generator=g, device=DEV).to(bf)
        k_seg = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf)
        v_seg = torch.randn(T, NS, Hkv, D, generator=g, device=DEV).to(bf)
        lse_seg = torch.empty(T, NS, Hq, device=DEV)
        qn = np64(q_seg.index_select(1, seq_t))
        kn = np64(k_seg.index_select(1, seq_t))
        vn = np64(v_seg.index_select(1, seq_t))
        # the oracle attends at the sampled steps and over the last W steps (whose LSEs the
        # compression reads); every step's rows are appended to the model
        ref_lse = {h: np.zeros((T, G)) for h in heads}
        dec_steps = o_steps | set(range(T - W, T))
        for t in range(T):
            loop.step(q_seg[t], k_seg[t], v_seg[t], lse_seg[t])
            ref = replay.step(qn[t], kn[t], vn[t], sidx, decode=t in dec_steps)
            for h in ref:
                ref_lse[h][t] = ref[h][1]
            if t in o_steps:
                torch.cuda.synchronize()
                o_gpu = np64(loop.o.index_select(0, seq_t))
                for h in heads:
                    s, kvh = divmod(h, Hkv)
                    for gi in range(G):
                        check_prob(o_gpu[sidx[s], kvh * G + gi], ref[h][0][gi], 2e-3,
                                   f"o seg {seg} step {t} head {h} q {gi}")
        torch.cuda.synchronize()
        assert int(loop.status.item()) == 0, "append ran out of pages"
        lse_gpu = np64(lse_seg.index_select(1, seq_t))
        ts = sorted(dec_steps)
        for h in heads:
            s, kvh = divmod(h, Hkv)
            check_lse(lse_gpu[ts, sidx[s], kvh * G:(kvh + 1) * G], ref_lse[h][ts], 2e-3,
                      f"lse seg {seg} head {h}")
        replay.check_cache(w, f"seg {seg} before compression")
        _check_pages_conserved(w, f"seg {seg} after the appends")
        loop.compress(q_seg[T - W:], lse_seg[T - W:])
        torch.cuda.synchronize()
        b = loop.comp.buf
        assert int(b.status.item()) == 0
        rows = lambda t_: {h: t_[h].cpu().numpy() for h in heads}
        replay.compress(qn[T - W:], {h: ref_lse[h][T - W:] for h in heads},
                        {h: np64(b.s_attn[h]) for h in heads}, rows(b.c), rows(b.sel_bits),
                        np_i(b.k), L_dense, p, w.S_max, f"seg {seg}", sidx=sidx)
        replay.check_cache(w, f"seg {seg} after the rewrite")
        _check_pages_conserved(w, f"seg {seg} after the rewrite")
        print(f"config 5: segment {seg} matches the oracle (kept {[replay.nr[h] for h in heads]})",
              flush=True)
        del q_seg, k_seg, v_seg, lse_seg

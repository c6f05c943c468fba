"""Full-size workloads in the launch configuration bench.py times, checked on sampled heads.

Stages whose inputs are the seeded workload are compared with the oracle run on that
workload: scores (rtol 2e-3, log domain), sampled redundancy scores, and (single-metric
configs) calibrated probabilities from the oracle's own scores.  Stages that consume the
GPU's own outputs are checked by their defining properties: the calibrated mixture is a
distribution over the candidates, the temperature solves its equation on the GPU's
inputs, the selection satisfies the Top-p rule on the GPU's probabilities, and the
rewritten cache holds exactly the selected rows in order (bytes) with the sparse and
dense pages in place.  Heads are sampled across the budget range.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workload as WL
from hk_testlib import (HostCache, check_log_scores, check_prob, check_topp_rule, np64, np_i,
                        rewritten_sources, unpack_bits)

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run_full(c):
    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import Compressor
    cfg = WL.config(c)
    w = WL.make_workload(cfg, DEV)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    metric = "attn+red" if cfg.get("n_ref") else "attn"
    comp = Compressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv, alloc, cfg["p"],
                      L_dense=cfg["L_dense"], L_sparse=cfg["L_sparse"], metric=metric,
                      n_ref=cfg.get("n_ref", 0))
    return hk, cfg, w, comp


def _sample_heads(k, n):
    order = np.argsort(k, kind="stable")
    picks = {int(order[0]), int(order[-1]), int(order[len(order) // 2])}
    rng = np.random.default_rng(0)
    picks |= {int(i) for i in rng.choice(len(k), size=n - len(picks), replace=False)}
    return sorted(picks)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("c", [2, 3, 4])
def test_full_size_sampled(c):
    hk, cfg, w, comp = _run_full(c)
    G, D = cfg["Hq"] // cfg["Hkv"], cfg["D"]
    scale = 1 / math.sqrt(D)
    ref = w.ref_slots
    # pristine copies for the sampled heads (taken before the rewrite touches the tables)
    pre = {"table": np_i(w.page_table).copy(), "mask": np_i(w.page_mask).astype(np.int64) & 0xFFFF,
           "n": np_i(w.n_pages).copy()}
    comp.score(w.q_obs, ref_slots=ref)
    comp.select()
    torch.cuda.synchronize()
    b = comp.buf
    k_all = np_i(b.k)
    heads = _sample_heads(k_all, 5)
    host = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages, heads=heads)
    s_gpu = {h: np64(b.s_attn[h]) for h in heads}
    c_gpu = {h: b.c[h].cpu().numpy() for h in heads}
    sel_gpu = {h: np_i(b.sel_bits[h]) for h in heads}
    xr_gpu = {h: np64(b.x_red[h]) for h in heads} if b.x_red is not None else None
    T_gpu = np64(b.T_red) if b.T_red is not None else None
    src_rows = {}
    for h in heads:
        rows, valid = host.head(h)
        vrows, _ = host.head_v(h)
        src_rows[h] = (rows, vrows, valid)
    comp.compact()
    torch.cuda.synchronize()
    assert int(b.status.item()) == 0
    qn = w.q_obs
    S = w.S_max
    for h in heads:
        rows, vrows, valid = src_rows[h]
        n = int(pre["n"][h])
        nc, ns, nd = O.tier_pages(n, cfg["L_dense"], cfg["L_sparse"])
        cand_len = 16 * (n - nd)
        s, kvh = divmod(h, cfg["Hkv"])
        q = qn[:, s, kvh * G:(kvh + 1) * G].float().cpu().numpy().astype(np.float64).reshape(-1, D)
        s_ref, _ = O.score_head(q, rows, valid, cand_len, scale)
        full = np.full(S, -np.inf)
        full[:len(s_ref)] = s_ref
        check_log_scores(s_gpu[h], full, 2e-3, f"cfg{c} score head {h}")
        cand = np.zeros(S, bool)
        cand[:len(valid)] = O.candidate_mask(valid, cand_len)
        if xr_gpu is not None:
            # redundancy on a sample of candidate slots (the oracle is a double loop)
            rng = np.random.default_rng(h)
            sample = rng.choice(np.nonzero(cand)[0], size=300, replace=False)
            only = np.zeros(len(valid), bool)
            only[sample] = True
            xr_ref = O.redundancy_head(rows, only, len(valid), np_i(ref[h]))
            err = np.abs(xr_gpu[h][sample] - xr_ref[sample])
            assert err.max() <= 2e-3, f"cfg{c} x_red head {h}: {err.max()}"
            # temperature: M_k(Softmax(x_red / T)) meets the target mass on the GPU's inputs
            k_a, m_a = int(np_i(b.k_attn)[h]), float(np64(b.mass_attn)[h])
            xs = xr_gpu[h][cand] / float(T_gpu[h])
            top = np.sort(xs)[::-1][:k_a]
            mk = math.exp(np.logaddexp.reduce(top) - np.logaddexp.reduce(xs))
            assert abs(mk - m_a) <= 2e-3, f"cfg{c} T head {h}: M_k {mk} vs target {m_a}"
            # the mixture is a distribution over the candidates
            cg = c_gpu[h].astype(np.float64)
            assert np.all(cg[~cand] == 0) and np.all(cg >= 0) and abs(cg.sum() - 1) <= 1e-4, h
        else:
            c_ref, _ = O.calibrate_head(full, cand)
            check_prob(c_gpu[h], c_ref, 2e-3, f"cfg{c} c head {h}")
        sel = unpack_bits(sel_gpu[h], S)
        check_topp_rule(c_gpu[h], sel, int(k_all[h]), cand, cfg["p"], what=f"cfg{c} head {h}")
        # rewrite: condensed band -> the selected rows in order; sparse pages in place under
        # the selection; dense pages unchanged
        new_table = np_i(w.page_table[h])
        new_mask = np_i(w.page_mask[h]).astype(np.int64) & 0xFFFF
        want = rewritten_sources(pre["table"][h], pre["mask"][h], n, sel, nc)
        npc = -(-len(want) // 16)
        sparse = []
        for pp in range(nc, nc + ns):
            word = sum(1 << t for t in range(16) if sel[pp * 16 + t])
            m2 = int(pre["mask"][h][pp]) & word
            if m2:
                sparse.append((int(pre["table"][h][pp]), m2))
        dense = [(int(pre["table"][h][pp]), int(pre["mask"][h][pp])) for pp in range(nc + ns, n)]
        assert int(w.n_pages[h]) == npc + len(sparse) + nd, f"cfg{c} n_pages head {h}"
        pos_of = {int(pid): i for i, pid in enumerate(pre["table"][h][:n])}
        for i in range(npc):
            chunk = want[16 * i:16 * (i + 1)]
            assert new_mask[i] == (1 << len(chunk)) - 1, f"cfg{c} mask head {h} page {i}"
            got = w.k_pool[int(new_table[i])][:len(chunk)].float().cpu().numpy()
            gotv = w.v_pool[int(new_table[i])][:len(chunk)].float().cpu().numpy()
            wk = np.stack([rows[pos_of[ph] * 16 + t] for ph, t in chunk])
            wv = np.stack([vrows[pos_of[ph] * 16 + t] for ph, t in chunk])
            assert np.array_equal(got, wk) and np.array_equal(gotv, wv), f"cfg{c} bytes head {h} page {i}"
        for i, (pid, m) in enumerate(sparse + dense):
            assert new_table[npc + i] == pid and new_mask[npc + i] == m, f"cfg{c} kept page head {h}"

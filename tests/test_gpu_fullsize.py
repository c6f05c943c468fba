"""Full-size workloads in the launch configuration bench.py times, checked on sampled heads.

For each sampled head the oracle is fed the GPU's own stage inputs: scores against the
oracle score (rtol 2e-3, log domain), calibrated probabilities, Top-p selection and
count (bit-exact), the solved temperature (config 4), and the rewritten cache layout
and bytes (bit-exact).  Heads are sampled across the budget range.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O
import workload as WL
from hk_testlib import HostCache, check_log_scores, check_prob, np64, np_i, unpack_bits

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
            # temperature: oracle bisection on the GPU's redundancy scores and target
            c_attn, _ = O.calibrate_head(s_gpu[h], cand)
            r_attn = O.topp_head(b.c_attn[h].cpu().numpy(), cand, cfg["p"])
            T_ref = O.solve_T_head(xr_gpu[h], cand, r_attn.k, r_attn.sel_mass / 2.0 ** 40)
            assert T_gpu[h] == pytest.approx(T_ref, rel=2e-3), f"cfg{c} T head {h}"
            c1, _ = O.calibrate_head(s_gpu[h], cand)
            c2, _ = O.calibrate_head(xr_gpu[h], cand, float(T_gpu[h]))
            c_ref = O.mix([c1, c2], [0.5, 0.5])
        else:
            c_ref, _ = O.calibrate_head(s_gpu[h], cand)
        check_prob(c_gpu[h], c_ref, 2e-3, f"cfg{c} c head {h}")
        r = O.topp_head(c_gpu[h], cand, cfg["p"])
        assert int(k_all[h]) == r.k, f"cfg{c} k head {h}"
        assert np.array_equal(unpack_bits(sel_gpu[h], S), r.sel), f"cfg{c} selection head {h}"
        # rewrite: the new logical rows equal the oracle layout over the pristine pages
        res = O.compact_head(pre["table"][h], pre["mask"][h], n, r.sel, cfg["L_dense"], cfg["L_sparse"])
        new_table = np_i(w.page_table[h])
        new_mask = np_i(w.page_mask[h]).astype(np.int64) & 0xFFFF
        assert int(w.n_pages[h]) == len(res.pages)
        pos_of = {int(pid): i for i, pid in enumerate(pre["table"][h][:n])}
        for i, e in enumerate(res.pages):
            assert new_mask[i] == e.mask, f"cfg{c} mask head {h} page {i}"
            if e.kind != "new":
                assert new_table[i] == e.phys
                continue
            got = w.k_pool[int(new_table[i])][:len(e.src)].float().cpu().numpy()
            gotv = w.v_pool[int(new_table[i])][:len(e.src)].float().cpu().numpy()
            want = np.stack([rows[pos_of[ph] * 16 + t] for ph, t in e.src])
            wantv = np.stack([vrows[pos_of[ph] * 16 + t] for ph, t in e.src])
            assert np.array_equal(got, want) and np.array_equal(gotv, wantv), f"cfg{c} bytes head {h} page {i}"

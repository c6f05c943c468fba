"""Full-size workloads in the launch configuration bench.py times, checked on sampled heads.

Stages whose inputs are the seeded workload are compared with the oracle run on that
workload: scores (rtol 2e-3, log domain), redundancy scores, calibrated probabilities
from the oracle's own scores, and for config 4 the redundancy temperature and the 0.5 / 0.5
mixture against the oracle's whole chain (its own scores, redundancy, Top-p count and mass,
temperature and mixture).  Stages that consume the GPU's own outputs are also checked by
their defining properties: the temperature solves its equation on the GPU's inputs (and
equals the oracle's bisection on them), the selection satisfies the Top-p rule on the GPU's
probabilities, and the rewritten cache holds exactly the selected rows in order (bytes)
with the sparse and dense pages in place.  Eight heads are sampled across the budget range
for the oracle comparisons; the Top-p rule and the rewritten layout are checked on every
head, and no physical page may be listed twice.
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
    heads = _sample_heads(k_all, 8)
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
            # redundancy at every candidate slot
            xr_full = O.redundancy_head(rows, valid, cand_len, np_i(ref[h]))
            xr_ref = np.full(S, -np.inf)
            xr_ref[:len(xr_full)] = xr_full
            assert np.all(np.isneginf(xr_gpu[h][~cand])), f"cfg{c} x_red head {h}: non-candidates"
            err = np.abs(xr_gpu[h][cand] - xr_ref[cand])
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
            # ... and equals the oracle's own chain on the raw inputs: oracle scores and
            # redundancy, its Top-p count and mass, its temperature, its 0.5 / 0.5 mixture
            c_att, _ = O.calibrate_head(full, cand)
            r_att = O.topp_head(c_att.astype(np.float32), cand, cfg["p"])
            T_ref = O.solve_T_head(xr_ref, cand, r_att.k, r_att.sel_mass / 2.0 ** 40)
            c_red, _ = O.calibrate_head(xr_ref, cand, T_ref)
            c_mix = O.mix([c_att, c_red], [0.5, 0.5])
            check_prob(cg, c_mix, 2e-3, f"cfg{c} mixture head {h} (oracle chain)")
            assert float(T_gpu[h]) == pytest.approx(T_ref, rel=2e-3), f"cfg{c} T chain head {h}"
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
    # beyond the sampled heads: the Top-p rule on every head, each on the values its
    # selection was made from, and the rewritten layout of every head (page counts, masks,
    # the sparse and dense pages kept in place); no physical page is listed twice
    c_all = b.c.cpu().numpy()
    sel_all = np_i(b.sel_bits)
    tab_all, n_all = np_i(w.page_table), np_i(w.n_pages)
    msk_all = np_i(w.page_mask).astype(np.int64) & 0xFFFF
    for h in range(w.n_heads):
        n = int(pre["n"][h])
        nc, ns, nd = O.tier_pages(n, cfg["L_dense"], cfg["L_sparse"])
        m = pre["mask"][h][:n]
        valid = ((m[:, None] >> np.arange(16)[None, :]) & 1).reshape(-1).astype(bool)
        cand = np.zeros(S, bool)
        cand[:len(valid)] = O.candidate_mask(valid, 16 * (n - nd))
        sel = unpack_bits(sel_all[h], S)
        check_topp_rule(c_all[h], sel, int(k_all[h]), cand, cfg["p"],
                        what=f"cfg{c} head {h} (all-heads rule)")
        kept = int((sel[:16 * nc] & valid[:16 * nc]).sum())
        npc = -(-kept // 16)
        words = (sel[:16 * n].reshape(n, 16) << np.arange(16)).sum(1)
        keep = [(int(pre["table"][h][pp]), int(m[pp] & words[pp])) for pp in range(nc, nc + ns)
                if m[pp] & words[pp]]
        keep += [(int(pre["table"][h][pp]), int(m[pp])) for pp in range(nc + ns, n)]
        assert int(n_all[h]) == npc + len(keep), f"cfg{c} n_pages head {h} (all heads)"
        full = [(1 << 16) - 1] * (npc - 1) + ([(1 << (kept - 16 * (npc - 1))) - 1] if npc else [])
        assert list(msk_all[h][:npc]) == full, f"cfg{c} condensed masks head {h}"
        assert [(int(tab_all[h][npc + i]), int(msk_all[h][npc + i])) for i in range(len(keep))] == keep, \
            f"cfg{c} kept pages head {h}"
    used = np.concatenate([tab_all[h][:n_all[h]] for h in range(w.n_heads)])
    assert len(np.unique(used)) == len(used), f"cfg{c}: a physical page listed twice"


@pytest.mark.timeout(900)
def test_budget_full_size_sampled():
    """The hard-budget step (Cautious Update votes, L_lower 2048 / L_upper 4096, 4 sinks) at
    config 3's full size in bench.py's launch configuration, on sampled heads: sampled rows'
    probabilities against the oracle, each sampled row's set by the Top-p properties on the
    probabilities it was made from, votes as the column counts of all row sets, the
    selection by its ranking properties, and the rewrite by its layout."""
    import paper_2606_28831_amd as hk
    from paper_2606_28831_amd.pipeline import BudgetCompressor
    from hk_testlib import check_topp_rule
    cfg = WL.config(3)
    w = WL.make_workload(cfg, DEV)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    comp = BudgetCompressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv, alloc, cfg["p"],
                            2048, 4096, L_dense=cfg["L_dense"], n_sink=4)
    pre = {"table": np_i(w.page_table).copy(), "mask": np_i(w.page_mask).astype(np.int64) & 0xFFFF,
           "n": np_i(w.n_pages).copy()}
    comp.select(w.q_obs)
    torch.cuda.synchronize()
    b = comp.buf
    G, D, R, S = cfg["Hq"] // cfg["Hkv"], cfg["D"], comp.R, w.S_max
    scale = 1 / math.sqrt(D)
    heads = _sample_heads(np_i(b["k"]), 3)
    host = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages, heads=heads)
    src = {h: (host.head(h)[0], host.head_v(h)[0], host.head(h)[1]) for h in heads}
    sel_all, v_all, k_all = np_i(b["sel_bits"]), np_i(b["votes"]).astype(np.int64) & 0xFFFF, np_i(b["k"])
    mode, cap = np_i(b["head_mode"]), np_i(b["k_cap"])
    rng = np.random.default_rng(9)
    for h in heads:
        rows, vrows, valid = src[h]
        n = int(pre["n"][h])
        cand = np.zeros(S, bool)
        cand[:len(valid)] = O.candidate_mask(valid, 16 * n)
        s_, kvh = divmod(h, cfg["Hkv"])
        q = w.q_obs[:, s_, kvh * G:(kvh + 1) * G].float().cpu().numpy().astype(np.float64).reshape(-1, D)
        _, lse = O.score_head(q, rows, valid, 16 * n, scale)
        row_bits = np.stack([unpack_bits(r, S) for r in np_i(b["row_sel"][h])])
        assert np.array_equal(row_bits.sum(axis=0), v_all[h]), f"votes head {h}"
        a_gpu = b["a_rows"][h].cpu().numpy()
        for r in rng.choice(R, size=3, replace=False):
            a_ref = O.score_rows_head(q[r:r + 1], rows, valid, 16 * n, scale, lse[r:r + 1])[0]
            full = np.zeros(S)
            full[:len(a_ref)] = a_ref
            check_prob(a_gpu[r], full, 2e-3, f"a head {h} row {r}")
            check_topp_rule(a_gpu[r], row_bits[r], int(row_bits[r].sum()), cand, cfg["p"],
                            what=f"row {r} head {h}")
        # selection: every head is above L_upper here, so every head is rewritten under the cap
        assert mode[h] == O.REWRITE and cap[h] == 4096
        sel = unpack_bits(sel_all[h], S)
        sinks = cand & (np.arange(S) < 4)
        base = cand & ~sinks & (v_all[h] >= 1)
        assert np.array_equal(sel & sinks, sinks) and not (sel & ~(sinks | base)).any()
        assert int(k_all[h]) == int(sel.sum()) == min(int(base.sum()), 4096 - int(sinks.sum())) + int(sinks.sum())
        kept, dropped = np.nonzero(sel & base)[0], np.nonzero(base & ~sel)[0]
        if len(kept) and len(dropped):
            assert min((v_all[h][j], j) for j in kept) > max((v_all[h][j], j) for j in dropped), h
    comp.compact()
    torch.cuda.synchronize()
    assert int(b["status"].item()) == 0
    for h in heads:
        rows, vrows, valid = src[h]
        n = int(pre["n"][h])
        sel = unpack_bits(sel_all[h], S)
        want = rewritten_sources(pre["table"][h], pre["mask"][h], n, sel, n)
        assert int(w.n_pages[h]) == -(-len(want) // 16) and 16 * int(w.n_pages[h]) <= 4096
        new_table = np_i(w.page_table[h])
        pos_of = {int(pid): i for i, pid in enumerate(pre["table"][h][:n])}
        for i in range(int(w.n_pages[h])):
            chunk = want[16 * i:16 * (i + 1)]
            got = w.k_pool[int(new_table[i])][:len(chunk)].float().cpu().numpy()
            assert np.array_equal(got, np.stack([rows[pos_of[ph] * 16 + t] for ph, t in chunk])), (h, i)

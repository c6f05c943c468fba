"""GPU parity of the multi-workgroup selector (hk_topp_select_ws, hk_calibrate_topp_ws)
against the oracle's Top-p and calibration (Sec. 3.2, Problem 1 and Solution 2).

Up to 32768 slots the wide selector must also reproduce the single-workgroup selector bit
for bit; past it (65536 .. 262144 slots, 16 .. 64 chunk workgroups per head) the oracle
alone decides.  The inputs cover every branch of the threshold search: keys of one digit
that fit the finishing workgroup's list and ones that do not (uniform and tied values),
the count clamp, ties split at the threshold, NaN / out-of-range values, empty heads and
ragged candidate counts with page-mask holes.
"""
import numpy as np
import pytest
import torch

import oracle as O
from hk_testlib import (check_lse, check_prob, check_topp_rule, np64, np_i, topp_edge_inputs,
                        unpack_bits)

pytestmark = pytest.mark.gpu

DEV = "cuda"
KINDS = ["uniform", "ties", "onehot", "nan_range", "zeros", "clamp", "crowded", "spread"]


def _hk():
    import paper_2606_28831_amd as hk
    return hk


def _topp_ws(c, cand_len, p, kmin, kmax, mask=None):
    hk = _hk()
    H, S = c.shape
    sel = torch.full((H, S // 32), 0x5A5A5A5A, dtype=torch.int32, device=DEV)
    k = torch.full((H,), -7, dtype=torch.int32, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    sm = torch.full((H,), float("nan"), device=DEV)
    ws = hk.select_workspace(H, S, DEV)
    ws.fill_(0xA5)                                # the kernels clear what must start at zero
    hk.hk_topp_select_ws(H, S, torch.tensor(cand_len, device=DEV), mask,
                         torch.tensor(c, device=DEV), p, sel, k, ws, k_min=kmin, k_max=kmax,
                         sel_mass=sm, status=st)
    torch.cuda.synchronize()
    return np_i(sel), np_i(k), sm.cpu().numpy(), int(st.item())


def _check_topp(c, cands, p, kmin, kmax, sel, k, sm, what):
    H, S = c.shape
    for h in range(H):
        r = O.topp_head(c[h], cands[h], p, k_min=kmin, k_max=kmax)
        assert int(k[h]) == r.k, (what, h, int(k[h]), r.k)
        assert np.array_equal(unpack_bits(sel[h], S), r.sel), (what, h)
        assert sm[h] == np.float32(r.sel_mass / 2.0 ** 40), (what, h, sm[h], r.sel_mass)


@pytest.mark.parametrize("S", [2048, 32768])
@pytest.mark.parametrize("kind", KINDS)
def test_topp_ws_equals_single_workgroup_and_oracle(kind, S):
    hk = _hk()
    c, cand_len, kmin, kmax, p = topp_edge_inputs(kind, S)
    H = c.shape[0]
    sel, k, sm, st = _topp_ws(c, cand_len, p, kmin, kmax)
    sel1 = torch.empty(H, S // 32, dtype=torch.int32, device=DEV)
    k1 = torch.empty(H, dtype=torch.int32, device=DEV)
    sm1 = torch.empty(H, device=DEV)
    st1 = torch.zeros(1, dtype=torch.int32, device=DEV)
    hk.hk_topp_select(H, S, torch.tensor(cand_len, device=DEV), None, torch.tensor(c, device=DEV),
                      p, sel1, k1, k_min=kmin, k_max=kmax, sel_mass=sm1, status=st1)
    torch.cuda.synchronize()
    assert np.array_equal(sel, np_i(sel1)) and np.array_equal(k, np_i(k1))
    assert np.array_equal(sm.view(np.int32), sm1.cpu().numpy().view(np.int32))
    assert st == int(st1.item())
    cands = [np.arange(S) < cand_len[h] for h in range(H)]
    _check_topp(c, cands, p, kmin, kmax, sel, k, sm, kind)
    if kind == "nan_range":
        assert st & hk.FLAG_NAN and st & hk.FLAG_RANGE
    else:
        assert st == 0


@pytest.mark.parametrize("kind,S", [("spread", 65536), ("crowded", 65536), ("uniform", 65536),
                                    ("ties", 65536), ("clamp", 65536), ("onehot", 65536),
                                    ("nan_range", 131072), ("ties", 131072), ("spread", 131072),
                                    ("uniform", 262144), ("crowded", 262144)])
def test_topp_ws_long_caches(kind, S):
    """Past the single-workgroup limit: 16 to 64 chunk workgroups per head."""
    c, cand_len, kmin, kmax, p = topp_edge_inputs(kind, S, seed=S + len(kind))
    sel, k, sm, st = _topp_ws(c, cand_len, p, kmin, kmax)
    cands = [np.arange(S) < cand_len[h] for h in range(c.shape[0])]
    _check_topp(c, cands, p, kmin, kmax, sel, k, sm, kind)
    assert (st != 0) == (kind == "nan_range")


def _holes(H, S, rng, frac=0.15):
    """Page masks with random holes (whole pages and single slots), as int16 words."""
    bits = rng.random((H, S)) >= frac * 0.3
    pages = rng.random((H, S // 16)) >= frac
    bits &= np.repeat(pages, 16, axis=1)
    words = (bits.reshape(H, S // 16, 16).astype(np.int64) << np.arange(16)).sum(-1)
    return bits, words.astype(np.uint16).view(np.int16)


@pytest.mark.parametrize("S,p", [(4128, 0.9), (65536, 0.95), (131072, 0.5)])
def test_topp_ws_page_mask_and_thresholds(S, p):
    """Candidates through the page mask as well as the count; a p that splits a run of
    tied values at the threshold, so the later slots of the tie are the ones taken."""
    rng = np.random.default_rng(S)
    H = 4
    valid, words = _holes(H, S, rng)
    cand_len = np.array([S, S - 100, S // 3 + 5, 4097], np.int32)
    c = np.zeros((H, S), np.float32)
    for h in range(H):
        # few distinct values with many ties each: the threshold lands inside a tie run
        c[h] = rng.choice(np.float32([4.0, 2.0, 1.0, 0.5]), S) / S
    cands = [O.candidate_mask(valid[h], int(cand_len[h])) for h in range(H)]
    sel, k, sm, st = _topp_ws(c, cand_len, p, 1, 0, mask=torch.tensor(words, device=DEV))
    _check_topp(c, cands, p, 1, 0, sel, k, sm, f"mask S={S}")
    assert st == 0


@pytest.mark.parametrize("S", [4096 + 32, 32768, 131072])
@pytest.mark.parametrize("two_metrics", [False, True])
def test_calibrate_topp_ws_vs_oracle(S, two_metrics):
    """c_out and lse_out against the oracle's calibration (mixture for two metrics).  The c this
    call wrote is the GPU's own, so the selection made from it is checked by Top-p's defining
    properties instead of an oracle run on it."""
    hk = _hk()
    rng = np.random.default_rng(S + two_metrics)
    H = 4
    valid, words = _holes(H, S, rng)
    cand_len = np.array([S, S - 33, S // 2, 0], np.int32)
    scale = np.array([0.3, 1.5, 4.0, 1.0])[:, None]
    x1 = (rng.standard_normal((H, S)) * scale).astype(np.float32)
    x2 = rng.standard_normal((H, S)).astype(np.float32)
    T2 = np.linspace(0.2, 3.0, H).astype(np.float32)
    weights = [0.25, 0.75] if two_metrics else [1.0]
    xs = [torch.tensor(x1, device=DEV)] + ([torch.tensor(x2, device=DEV)] if two_metrics else [])
    Ts = [None, torch.tensor(T2, device=DEV)] if two_metrics else None
    n = len(xs)
    c = torch.full((H, S), 9.0, device=DEV)
    lse = torch.empty(H, n, device=DEV)
    sel = torch.empty(H, S // 32, dtype=torch.int32, device=DEV)
    k = torch.empty(H, dtype=torch.int32, device=DEV)
    sm = torch.empty(H, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    ws = hk.select_workspace(H, S, DEV)
    p = 0.9
    hk.hk_calibrate_topp_ws(H, S, torch.tensor(cand_len, device=DEV), torch.tensor(words, device=DEV),
                            xs, Ts, weights, p, sel, k, ws, c_out=c, lse_out=lse, sel_mass=sm,
                            status=st)
    torch.cuda.synchronize()
    c_np, lse_np = c.cpu().numpy(), np64(lse)
    sel_np, k_np, sm_np = np_i(sel), np_i(k), sm.cpu().numpy()
    for h in range(H):
        cand = O.candidate_mask(valid[h], int(cand_len[h]))
        ca, la = O.calibrate_head(x1[h].astype(np.float64), cand)
        refs, lses = [ca], [la]
        if two_metrics:
            cb, lb = O.calibrate_head(x2[h].astype(np.float64), cand, float(T2[h]))
            refs, lses = [ca, cb], [la, lb]
        check_prob(c_np[h], O.mix(refs, weights), 1e-5, f"c head {h}")
        check_lse(lse_np[h], lses, 1e-5, f"lse head {h}")
        m = check_topp_rule(c_np[h], unpack_bits(sel_np[h], S), k_np[h], cand, p,
                            what=f"Top-p head {h}")
        assert sm_np[h] == np.float32(m / 2.0 ** 40), (h, sm_np[h], m)
    assert int(st.item()) == 0


def test_calibrate_topp_ws_repeated_calls_reuse_the_workspace():
    """Two calls on one workspace, the second with fewer heads and a shorter cache, each
    matching a call on a fresh workspace: nothing of the first call leaks into the second."""
    hk = _hk()
    rng = np.random.default_rng(3)
    outs = []
    for H, S in ((6, 65536), (3, 8192)):
        x = torch.tensor((rng.standard_normal((H, S)) * 2).astype(np.float32), device=DEV)
        cl = torch.full((H,), S - 7, dtype=torch.int32, device=DEV)
        outs.append((H, S, x, cl))
    shared = hk.select_workspace(6, 65536, DEV)
    for H, S, x, cl in outs:
        res = []
        for ws in (shared, hk.select_workspace(H, S, DEV)):
            sel = torch.empty(H, S // 32, dtype=torch.int32, device=DEV)
            k = torch.empty(H, dtype=torch.int32, device=DEV)
            c = torch.empty(H, S, device=DEV)
            hk.hk_calibrate_topp_ws(H, S, cl, None, [x], None, [1.0], 0.9, sel, k, ws, c_out=c)
            torch.cuda.synchronize()
            res.append((sel.cpu(), k.cpu(), c.cpu()))
        for a, b in zip(*res):
            assert torch.equal(a, b)


def test_compression_step_on_long_rows():
    """The whole step on rows of 131072 slots (64 select chunks per head), where only the
    wide selector applies: Compressor's separate calls and the one-call hk_compress leave
    the same cache, counts and bitmap bit for bit; the scores and calibrated probabilities
    match the oracle's; the selection obeys the Top-p rule on the calibrated values it was
    made from, and the rewrite leaves the page list the tiers define for it."""
    import math
    import workload as WL
    from hk_testlib import HostCache, check_compaction, check_log_scores, q_rows, rewrite_layout, snapshot
    from paper_2606_28831_amd.pipeline import Compressor
    hk = _hk()
    cfg = dict(L=1, B=1, Hq=8, Hkv=2, D=128, N=131072 - 37, dtype="bf16", W=16, seed=5,
               recipe="tempered")
    G, p, scale = 4, 0.9, 1 / math.sqrt(128)
    outs = []
    for fused in (False, True):
        w = WL.make_workload(cfg, DEV, hole_prob=0.05, max_pages=8192)
        kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
        alloc = hk.Allocator(w.free_ids, w.free_top)
        H, S = w.n_heads, w.S_max
        assert S == 131072
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        before = snapshot(w)
        if fused:
            d = hk.dims(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"])
            k = torch.empty(H, dtype=torch.int32, device=DEV)
            sel = torch.empty(H, S // 32, dtype=torch.int32, device=DEV)
            hk.hk_compress(d, w.q_obs, kv, 0, 0, scale, p, alloc, k,
                           hk.workspace(hk.OP_COMPRESS, d, w.max_pages, DEV), status=st,
                           sel_bits_out=sel)
            torch.cuda.synchronize()
        else:
            host = HostCache(w.k_pool, None, w.page_table, w.page_mask, w.n_pages)
            comp = Compressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv, alloc, p)
            comp.score(w.q_obs)
            comp.select()
            torch.cuda.synchronize()
            b = comp.buf
            s_np, c_np = np64(b.s_attn), b.c.cpu().numpy()
            sel_np, k_np = np_i(b.sel_bits), np_i(b.k)
            qn = np64(w.q_obs)
            for h in range(H):
                rows, valid = host.head(h)
                cand_len = 16 * int(host.n[h])
                s_ref, _ = O.score_head(q_rows(qn, h, cfg["Hkv"], G), rows, valid, cand_len, scale)
                full = np.full(S, -np.inf)
                full[:len(s_ref)] = s_ref
                check_log_scores(s_np[h], full, 2e-3, f"long-row score head {h}")
                cand = np.zeros(S, bool)
                cand[:len(valid)] = O.candidate_mask(valid, cand_len)
                c_ref, _ = O.calibrate_head(full, cand)
                check_prob(c_np[h].astype(np.float64), c_ref, 2e-3, f"long-row c head {h}")
                check_topp_rule(c_np[h], unpack_bits(sel_np[h], S), int(k_np[h]), cand, p,
                                what=f"long-row head {h}")
            comp.compact()
            torch.cuda.synchronize()
            check_compaction(w, before, sel_np, S, lambda h, sl: rewrite_layout(
                before["table"][h], before["mask"][h], int(before["n"][h]), sl, 0))
            k, sel, st = b.k, b.sel_bits, b.status
        assert int(st.item()) == 0
        outs.append([t.cpu().clone() for t in (k, sel, w.page_table, w.page_mask, w.n_pages,
                                               w.free_ids, w.free_top)]
                    + [w.k_pool.view(torch.int16).cpu(), w.v_pool.view(torch.int16).cpu()])
        del w, kv
        torch.cuda.empty_cache()
    for a, b in zip(*outs):
        assert torch.equal(a, b)


@pytest.mark.parametrize("seed", range(12))
def test_topp_ws_random_shapes_equal_single_workgroup(seed):
    """Random row lengths (any multiple of 32 up to 32768, so chunks of every fill and a last
    chunk of any length), candidate counts, page holes, clamps and value mixes -- coarse
    values with many exact ties, one-binade values, spread values, zeros and NaN: the wide
    selector equals the single-workgroup selector bit for bit (bitmap, count, mass, flags)."""
    hk = _hk()
    rng = np.random.default_rng(1000 + seed)
    H = 5
    S = int(rng.integers(1, 1025)) * 32
    kind = seed % 4
    if kind == 0:
        c = np.round(rng.random((H, S)), 2).astype(np.float32) / S          # ties
    elif kind == 1:
        c = (1.0 + rng.random((H, S)) * 0.01).astype(np.float32) / S        # one binade
    elif kind == 2:
        c = np.exp2(-rng.random((H, S)) * 30).astype(np.float32)            # 30 binades
    else:
        c = rng.random((H, S)).astype(np.float32)
        c[:, ::7] = 0.0
        c[0, :3] = [np.nan, -1.0, 2.0]
    cand_len = rng.integers(0, S + 1, H).astype(np.int32)
    cand_len[0] = S
    valid, words = _holes(H, S, rng)
    kmin, kmax = (int(rng.integers(0, 4)), int(rng.integers(0, S // 2 + 2))) if seed % 3 == 0 else (1, 0)
    p = float(rng.choice([0.5, 0.9, 0.999, 1.0]))
    mask = torch.tensor(words, device=DEV)
    sel, k, sm, st = _topp_ws(c, cand_len, p, kmin, kmax, mask=mask)
    sel1 = torch.empty(H, S // 32, dtype=torch.int32, device=DEV)
    k1 = torch.empty(H, dtype=torch.int32, device=DEV)
    sm1 = torch.empty(H, device=DEV)
    st1 = torch.zeros(1, dtype=torch.int32, device=DEV)
    hk.hk_topp_select(H, S, torch.tensor(cand_len, device=DEV), mask, torch.tensor(c, device=DEV),
                      p, sel1, k1, k_min=kmin, k_max=kmax, sel_mass=sm1, status=st1)
    torch.cuda.synchronize()
    assert np.array_equal(sel, np_i(sel1)) and np.array_equal(k, np_i(k1)), (seed, S, kind)
    assert np.array_equal(sm.view(np.int32), sm1.cpu().numpy().view(np.int32)), (seed, S)
    assert st == int(st1.item()), (seed, st, int(st1.item()))
    if seed < 4:                                   # and the oracle, on the smaller draws
        cands = [O.candidate_mask(valid[h], int(cand_len[h])) for h in range(H)]
        _check_topp(c, cands, p, kmin, kmax, sel, k, sm, f"random {seed}")


def test_two_metric_step_on_long_rows():
    """The mixture path (attention mass + sampled redundancy, 0.5 / 0.5 after the
    redundancy temperature is solved) on 65536-slot rows, where both the selector and the
    temperature search take their long-row kernels: each head's mixture equals the oracle's
    chain on the same cache (oracle scores and redundancy, its Top-p count and mass, its
    temperature, its mixture), and the selection obeys the Top-p rule on it."""
    import math
    import workload as WL
    from hk_testlib import HostCache, check_log_scores, q_rows
    from paper_2606_28831_amd.pipeline import Compressor
    hk = _hk()
    cfg = dict(L=1, B=1, Hq=8, Hkv=2, D=128, N=65536 - 200, dtype="bf16", W=16, seed=9,
               recipe="normal", n_ref=256)
    G, p, scale = 4, 0.9, 1 / math.sqrt(128)
    w = WL.make_workload(cfg, DEV, max_pages=4096, hole_prob=0.02)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    host = HostCache(w.k_pool, None, w.page_table, w.page_mask, w.n_pages)
    comp = Compressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv,
                      hk.Allocator(w.free_ids, w.free_top), p, metric="attn+red", n_ref=256)
    H, S = w.n_heads, w.S_max
    assert S == 65536
    comp.score(w.q_obs, ref_slots=w.ref_slots)
    comp.select()
    torch.cuda.synchronize()
    b = comp.buf
    assert int(b.status.item()) == 0
    s_np, c_np, sel_np, k_np = np64(b.s_attn), b.c.cpu().numpy(), np_i(b.sel_bits), np_i(b.k)
    T_gpu, qn, ref = np64(b.T_red), np64(w.q_obs), np_i(w.ref_slots)
    for h in range(H):
        rows, valid = host.head(h)
        cand_len = 16 * int(host.n[h])
        s_ref, _ = O.score_head(q_rows(qn, h, cfg["Hkv"], G), rows, valid, cand_len, scale)
        full = np.full(S, -np.inf)
        full[:len(s_ref)] = s_ref
        check_log_scores(s_np[h], full, 2e-3, f"score head {h}")
        cand = np.zeros(S, bool)
        cand[:len(valid)] = O.candidate_mask(valid, cand_len)
        xr = np.full(S, -np.inf)
        xr_full = O.redundancy_head(rows, valid, cand_len, ref[h])
        xr[:len(xr_full)] = xr_full
        c_att, _ = O.calibrate_head(full, cand)
        r_att = O.topp_head(c_att.astype(np.float32), cand, p)
        T_ref = O.solve_T_head(xr, cand, r_att.k, r_att.sel_mass / 2.0 ** 40)
        assert float(T_gpu[h]) == pytest.approx(T_ref, rel=2e-3), (h, float(T_gpu[h]), T_ref)
        c_red, _ = O.calibrate_head(xr, cand, T_ref)
        check_prob(c_np[h].astype(np.float64), O.mix([c_att, c_red], [0.5, 0.5]), 2e-3,
                   f"mixture head {h}")
        check_topp_rule(c_np[h], unpack_bits(sel_np[h], S), int(k_np[h]), cand, p,
                        what=f"mixture head {h}")

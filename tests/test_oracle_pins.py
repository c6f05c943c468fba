"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Nothing here re-types an oracle formula: each check is a closed form, a special
case that reduces to a library routine (scipy), brute force over tiny inputs, an
invariant, or a hand-derived golden value (tests/golden/*.json, each citing the
passage it follows).  A plausible slip in the oracle (dropped term, wrong axis,
sign, index or tie rule) fails at least one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special as sps

import oracle as O

RNG = np.random.default_rng(1234)


def _golden(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- score (a1)
def _rand_head(R=6, S=40, D=8, seed=0, scale=1.0):
    r = np.random.default_rng(seed)
    return r.standard_normal((R, D)) * scale, r.standard_normal((S, D))


def test_score_golden(golden_dir):
    g = _golden(golden_dir, "score_hand.json")
    valid = np.ones(2, bool)
    s, lse = O.score_head(np.array(g["q_rows"]), np.array(g["keys"]), valid, 2, g["sm_scale"])
    np.testing.assert_allclose(s, g["s"], rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, g["row_lse"], rtol=0, atol=1e-13)


def test_score_mass_sums_to_one():
    q, k = _rand_head(R=12, S=77, D=16, seed=1, scale=2.0)
    valid = np.ones(77, bool)
    s, _ = O.score_head(q, k, valid, 77, 0.25)
    assert abs(np.sum(np.exp(s)) - 1.0) < 1e-12


def test_score_single_row_is_log_softmax():
    q, k = _rand_head(R=1, S=50, D=8, seed=2)
    valid = np.ones(50, bool)
    s, lse = O.score_head(q, k, valid, 50, 0.3)
    np.testing.assert_allclose(s, sps.log_softmax(0.3 * (q @ k.T))[0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, sps.logsumexp(0.3 * (q @ k.T), axis=1), rtol=1e-14)


def test_score_is_log_mean_of_row_softmax():
    q, k = _rand_head(R=9, S=33, D=4, seed=3, scale=3.0)
    valid = np.ones(33, bool)
    s, _ = O.score_head(q, k, valid, 33, 0.5)
    probs = np.stack([sps.softmax(0.5 * (q[r] @ k.T)) for r in range(9)])
    np.testing.assert_allclose(np.exp(s), probs.mean(axis=0), rtol=1e-12)


def test_score_row_permutation_and_duplication_invariant():
    q, k = _rand_head(R=5, S=20, D=6, seed=4)
    valid = np.ones(20, bool)
    s, _ = O.score_head(q, k, valid, 20, 0.7)
    s2, _ = O.score_head(q[::-1], k, valid, 20, 0.7)
    s3, _ = O.score_head(np.concatenate([q, q]), k, valid, 20, 0.7)
    np.testing.assert_allclose(s2, s, atol=1e-13)
    np.testing.assert_allclose(s3, s, atol=1e-13)


def test_score_key_permutation_equivariant():
    q, k = _rand_head(R=4, S=30, D=5, seed=5)
    valid = np.ones(30, bool)
    perm = RNG.permutation(30)
    s, _ = O.score_head(q, k, valid, 30, 1.0)
    sp, _ = O.score_head(q, k[perm], valid, 30, 1.0)
    np.testing.assert_allclose(sp, s[perm], atol=1e-13)


def test_score_masked_slots_equal_removed_slots():
    q, k = _rand_head(R=4, S=32, D=5, seed=6)
    valid = RNG.random(32) < 0.6
    s, lse = O.score_head(q, k, valid, 32, 0.9)
    s_red, lse_red = O.score_head(q, k[valid], np.ones(valid.sum(), bool), valid.sum(), 0.9)
    np.testing.assert_allclose(s[valid], s_red, atol=1e-13)
    assert np.all(np.isneginf(s[~valid]))
    np.testing.assert_allclose(lse, lse_red, atol=1e-13)


def test_score_cand_len_keeps_full_normaliser():
    q, k = _rand_head(R=3, S=48, D=4, seed=7)
    valid = np.ones(48, bool)
    s_all, lse_all = O.score_head(q, k, valid, 48, 1.0)
    s_c, lse_c = O.score_head(q, k, valid, 32, 1.0)
    np.testing.assert_allclose(s_c[:32], s_all[:32], atol=1e-13)
    assert np.all(np.isneginf(s_c[32:]))
    np.testing.assert_allclose(lse_c, lse_all, atol=1e-13)
    # supplying the true normaliser gives the same scores
    s_in, _ = O.score_head(q, k, valid, 32, 1.0, row_lse_in=sps.logsumexp(q @ k.T, axis=1))
    np.testing.assert_allclose(s_in, s_c, atol=1e-12)


def test_read_head_page_shuffle():
    D, n_pages = 3, 5
    logical = RNG.standard_normal((n_pages * 16, D))
    ids = RNG.permutation(11)[:n_pages]
    pool = np.zeros((11, 16, D))
    for pp, pid in enumerate(ids):
        pool[pid] = logical[pp * 16:(pp + 1) * 16]
    masks = [0xFFFF, 0x00F0, 0xFFFF, 0x8001, 0x0001]
    rows, valid = O.read_head(pool, ids, masks, n_pages)
    np.testing.assert_array_equal(rows, logical)
    assert valid.sum() == 16 + 4 + 16 + 2 + 1
    assert valid[16 + 4] and not valid[16 + 3] and valid[3 * 16 + 15] and valid[4 * 16]


# ---------------------------------------------------------------- redundancy
def test_redundancy_closed_forms():
    keys = np.array([[1.0, 0.0], [2.0, 0.0], [0.0, 3.0], [-1.0, 0.0],
                     [math.cos(0.3), math.sin(0.3)], [0.0, 0.0]])
    valid = np.ones(6, bool)
    # slot 1 duplicates slot 0 up to scale -> cos = 1 -> -1
    x = O.redundancy_head(keys, valid, 6, [0])
    assert x[1] == pytest.approx(-1.0)
    assert x[2] == pytest.approx(0.0, abs=1e-15)     # orthogonal
    assert x[3] == pytest.approx(1.0)                # antiparallel: -(-1)
    assert x[4] == pytest.approx(-math.cos(0.3))     # 2-D angle
    assert x[5] == pytest.approx(0.0)                # zero-norm key
    assert x[0] == pytest.approx(1.0)                # only reference is itself: empty set
    # self excluded, the other reference counts
    x2 = O.redundancy_head(keys, valid, 6, [0, 2])
    assert x2[0] == pytest.approx(0.0, abs=1e-15)
    # max over references
    x3 = O.redundancy_head(keys, valid, 6, [2, 4])
    assert x3[0] == pytest.approx(-math.cos(0.3))
    # candidates only
    x4 = O.redundancy_head(keys, valid, 3, [0])
    assert np.all(np.isneginf(x4[3:]))


def test_redundancy_scale_invariant():
    k = RNG.standard_normal((20, 7))
    valid = np.ones(20, bool)
    refs = [1, 4, 9, 13]
    a = O.redundancy_head(k, valid, 20, refs)
    b = O.redundancy_head(k * np.linspace(0.5, 3, 20)[:, None], valid, 20, refs)
    np.testing.assert_allclose(a, b, atol=1e-13)


def test_redundancy_matches_scipy_cosine():
    """Against scipy's cosine distance over every (candidate, reference) pair, the reference
    equal to the candidate skipped; candidates are valid slots below cand_len."""
    from scipy.spatial.distance import cdist
    k = RNG.standard_normal((60, 9))
    valid = RNG.random(60) < 0.85
    refs = sorted(RNG.choice(60, size=12, replace=False).tolist())
    x = O.redundancy_head(k, valid, 50, refs)
    cosm = 1.0 - cdist(k, k[refs], metric="cosine")
    for j in range(60):
        if not (valid[j] and j < 50):
            assert np.isneginf(x[j])
            continue
        others = [c for c, i in enumerate(refs) if i != j]
        assert x[j] == pytest.approx(-max(cosm[j, others]), abs=1e-12)


# ---------------------------------------------------------------- calibrate (a2)
def test_calibrate_sums_to_one_and_matches_scipy():
    x = RNG.standard_normal(100) * 4
    cand = RNG.random(100) < 0.8
    for T in (0.05, 0.5, 1.0, 7.0):
        c, lse = O.calibrate_head(x, cand, T)
        assert abs(c.sum() - 1.0) < 1e-12
        assert np.all(c[~cand] == 0)
        np.testing.assert_allclose(c[cand], sps.softmax(x[cand] / T), rtol=1e-12)
        assert lse == pytest.approx(sps.logsumexp(x[cand] / T), rel=1e-14)


def test_calibrate_order_invariance():
    """App. D.2 theorem: for every T > 0 the ranking of S(x/T) is that of x."""
    x = RNG.standard_normal(64)
    cand = np.ones(64, bool)
    ref = np.argsort(-x, kind="stable")
    for T in (1e-2, 0.3, 1.0, 3.0, 50.0):
        c, _ = O.calibrate_head(x, cand, T)
        assert list(np.argsort(-c, kind="stable")) == list(ref)


def test_calibrate_uniform_and_empty():
    c, lse = O.calibrate_head(np.full(8, 3.0), np.ones(8, bool), 2.0)
    np.testing.assert_allclose(c, 1 / 8)
    assert lse == pytest.approx(1.5 + math.log(8))
    c, lse = O.calibrate_head(np.full(4, -np.inf), np.ones(4, bool))
    assert np.all(c == 0) and lse == -math.inf


def test_mixture_is_distribution():
    x1, x2 = RNG.standard_normal(30), RNG.standard_normal(30)
    cand = np.ones(30, bool)
    c = O.mix([O.calibrate_head(x1, cand)[0], O.calibrate_head(x2, cand, 0.3)[0]], [0.5, 0.5])
    assert abs(c.sum() - 1) < 1e-12


# ---------------------------------------------------------------- pooling (Solution 1, SnapKV form)
def test_pool_radius_zero_is_identity():
    x = RNG.standard_normal(50)
    cand = RNG.random(50) < 0.7
    out = O.pool_max_head(x, cand, 0)
    assert np.array_equal(out[cand], x[cand]) and np.all(np.isneginf(out[~cand]))


@pytest.mark.parametrize("radius", [1, 3, 8])
def test_pool_matches_scipy_maximum_filter(radius):
    import scipy.ndimage as ndi
    x = RNG.standard_normal(300) * 3
    cand = RNG.random(300) < 0.6
    masked = np.where(cand, x, -np.inf)
    ref = ndi.maximum_filter1d(masked, size=2 * radius + 1, mode="constant", cval=-np.inf)
    ref = np.where(cand, ref, -np.inf)
    assert np.array_equal(O.pool_max_head(x, cand, radius), ref)


def test_pool_invariants():
    x = RNG.standard_normal(200)
    cand = RNG.random(200) < 0.5
    out = O.pool_max_head(x, cand, 3)
    assert np.all(out[cand] >= x[cand])                       # dominates its input
    c = np.where(cand, 2.5, -np.inf)
    assert np.array_equal(O.pool_max_head(c, cand, 4)[cand], np.full(cand.sum(), 2.5))
    # a single peak spreads to exactly the candidates within the radius
    y = np.full(40, -1.0)
    y[20] = 5.0
    allc = np.ones(40, bool)
    out = O.pool_max_head(y, allc, 2)
    assert set(np.nonzero(out == 5.0)[0]) == {18, 19, 20, 21, 22}
    # monotone transforms commute with the pooling (so pooling log scores is pooling mass)
    z = RNG.random(60) + 0.01
    cz = RNG.random(60) < 0.8
    assert np.allclose(O.pool_max_head(np.log(z), cz, 2)[cz], np.log(O.pool_max_head(z, cz, 2)[cz]))


# ---------------------------------------------------------------- Top-p (a3)
def test_topp_golden(golden_dir):
    g = _golden(golden_dir, "topp_hand.json")
    for case in g["cases"]:
        c = np.array(case["c"], dtype=np.float32)
        r = O.topp_head(c, np.ones(len(c), bool), case["p"])
        assert r.k == case["k"], case["name"]
        assert sorted(np.nonzero(r.sel)[0].tolist()) == case["selected"], case["name"]


def _brute_force_k(weights, target):
    n = len(weights)
    if target == 0:
        return 0, 0
    for k in range(1, n + 1):
        best = max(sum(weights[i] for i in sub) for sub in itertools.combinations(range(n), k))
        if best >= target:
            return k, best
    raise AssertionError("unreachable")


@pytest.mark.parametrize("trial", range(60))
def test_topp_brute_force_small(trial):
    r = np.random.default_rng(100 + trial)
    # every size up to 12, with the largest sizes (4095 subsets) taken in a third of the trials
    n = 12 if trial % 6 == 1 else 11 if trial % 6 == 2 else int(r.integers(1, 13))
    raw = r.exponential(size=n) ** r.uniform(0.5, 4)
    if trial % 5 == 0:
        raw[r.integers(0, n)] = raw.max()          # planted tie
    c = (raw / raw.sum()).astype(np.float32)
    p = float(r.choice([0.3, 0.5, 0.7, 0.9, 0.95, 0.999, 1.0, r.uniform(0.01, 1)]))
    res = O.topp_head(c, np.ones(n, bool), p)
    w = [math.floor(float(v) * 2 ** 40) for v in c]
    total = sum(w)
    target = math.ceil(Fraction(round(p * 10 ** 6), 10 ** 6) * total)
    k_bf, best = _brute_force_k(w, target)
    assert res.k == max(k_bf, 1)
    chosen = np.nonzero(res.sel)[0]
    assert sum(w[i] for i in chosen) == (best if k_bf >= 1 else sorted(w)[-1])
    # the exact real-valued rule agrees unless the real prefix mass sits within
    # n*2^-40 of p*Total (fixed-point reading of Problem 1)
    order = O.order_desc(c, range(n))
    ptot = Fraction(round(p * 10 ** 6), 10 ** 6) * sum(Fraction(float(v)) for v in c)
    cum, k_real = Fraction(0), n
    for i, j in enumerate(order):
        cum += Fraction(float(c[j]))
        if cum >= ptot:
            k_real = i + 1
            break
    if k_real != res.k:
        assert abs(float(cum - ptot)) <= n * 2.0 ** -40


@pytest.mark.parametrize("N", [1, 2, 7, 16, 100, 1000, 2048, 4097])
@pytest.mark.parametrize("p", [0.1, 0.5, 0.9, 0.95, 0.999999])
def test_topp_uniform_is_ceil_pN(N, p):
    c = np.full(N, np.float32(1.0 / N), dtype=np.float32)
    r = O.topp_head(c, np.ones(N, bool), p)
    assert r.k == math.ceil(round(p * 1e6) * N / 1e6)
    # ties resolve to the most recent slots
    assert np.all(r.sel[N - r.k:]) and not np.any(r.sel[:N - r.k])


def test_topp_invariants_random():
    for seed in range(20):
        r = np.random.default_rng(seed)
        n = int(r.integers(50, 500))
        c = r.dirichlet(np.full(n, r.uniform(0.05, 2))).astype(np.float32)
        cand = r.random(n) < 0.9
        p = float(r.uniform(0.05, 0.999))
        res = O.topp_head(c, cand, p)
        assert not np.any(res.sel & ~cand)
        w = np.array([math.floor(float(v) * 2 ** 40) for v in c], dtype=object)
        mass = sum(w[res.sel])
        assert mass >= res.target
        weakest = min(w[res.sel])
        assert mass - weakest < res.target or res.k == 1
        # every unselected candidate weighs no more than the weakest selected
        if (cand & ~res.sel).any():
            assert max(w[cand & ~res.sel]) <= weakest


def test_topp_clamps_and_empty():
    c = np.array([0.7, 0.1, 0.1, 0.1], np.float32)
    assert O.topp_head(c, np.ones(4, bool), 0.99, k_max=2).k == 2
    assert O.topp_head(c, np.ones(4, bool), 0.0).k == 1       # k_min
    assert O.topp_head(c, np.ones(4, bool), 0.0, k_min=0).k == 0
    assert O.topp_head(c, np.zeros(4, bool), 0.9).k == 0      # no candidate
    cn = np.array([np.nan, 0.5, 0.5], np.float32)
    r = O.topp_head(cn, np.ones(3, bool), 1.0)
    assert r.k == 2 and not r.sel[0]
    # values above 1 clamp to 1 and then tie: the more recent slot ranks first
    cc = np.array([3.0, 2.0, 0.0, 0.0], np.float32)
    r = O.topp_head(cc, np.ones(4, bool), 0.5)
    assert r.k == 1 and r.sel[1] and not r.sel[0]


# ---------------------------------------------------------------- T solve (a2')
def test_solve_T_closed_form(golden_dir):
    g = _golden(golden_dir, "solveT_twolevel.json")
    for case in g["cases"]:
        n, k = case["n"], case["k"]
        x = np.full(n, case["b"])
        pos = RNG.permutation(n)[:k]
        x[pos] = case["a"]
        T = O.solve_T_head(x, np.ones(n, bool), k, case["m"])
        assert T == pytest.approx(case["T"], rel=1e-6)
        # and the solved T reproduces the mass
        c, _ = O.calibrate_head(x, np.ones(n, bool), T)
        assert O.topk_mass(c, np.ones(n, bool), k) == pytest.approx(case["m"], rel=1e-6)


def test_solve_T_monotone_and_clamped():
    x = RNG.standard_normal(200)
    cand = np.ones(200, bool)
    k = 20
    Ts = np.exp(np.linspace(math.log(1e-3), math.log(1e3), 60))
    masses = [O.topk_mass(O.calibrate_head(x, cand, T)[0], cand, k) for T in Ts]
    assert all(a >= b - 1e-11 for a, b in zip(masses, masses[1:]))  # fp64 exp of |x/T| ~ 1e3
    # a target above every reachable mass drives T to the sharp end, one below
    # every reachable mass (the uniform limit k/n) drives it to the flat end
    assert O.solve_T_head(x, cand, k, 1.5) == pytest.approx(1e-4, rel=1e-9)
    assert O.solve_T_head(x, cand, k, 0.0) == pytest.approx(1e4, rel=1e-9)


# ---------------------------------------------------------------- compact (a4)
def test_compact_golden(golden_dir):
    g = _golden(golden_dir, "compact_hand.json")
    sel = np.zeros(g["n_pages"] * 16, bool)
    sel[g["selected_slots"]] = True
    res = O.compact_head(g["table"], g["masks"], g["n_pages"], sel, g["L_dense"], g["L_sparse"])
    exp = g["expect"]
    assert res.freed == exp["freed"] and res.n_new == exp["n_new"]
    assert len(res.pages) == len(exp["pages"])
    for got, want in zip(res.pages, exp["pages"]):
        assert got.kind == want["kind"] and got.mask == want["mask"]
        if "phys" in want:
            assert got.phys == want["phys"]
        if "src" in want:
            assert [list(x) for x in got.src] == want["src"]


def test_tier_pages_closed_form():
    assert O.tier_pages(10, 40, 64) == (3, 4, 3)
    assert O.tier_pages(10, 0, 0) == (10, 0, 0)
    assert O.tier_pages(2, 512, 2048) == (0, 0, 2)
    assert O.tier_pages(40, 512, 2048) == (0, 8, 32)
    assert O.tier_pages(1024, 512, 2048) == (864, 128, 32)


@pytest.mark.parametrize("seed", range(8))
def test_compact_matches_take(seed):
    r = np.random.default_rng(seed)
    D, n_pages, pool_n = 4, int(r.integers(1, 30)), 64
    ids = r.permutation(pool_n)[:n_pages]
    masks = r.integers(1, 1 << 16, n_pages)
    masks[-1] = (1 << int(r.integers(1, 17))) - 1
    pool = r.standard_normal((pool_n, 16, D))
    rows, valid = O.read_head(pool, ids, masks, n_pages)
    sel = r.random(n_pages * 16) < r.uniform(0.05, 0.95)
    Ld, Ls = int(r.integers(0, 5)) * 16 + int(r.integers(0, 2)) * 5, int(r.integers(0, 6)) * 16
    res = O.compact_head(ids, masks, n_pages, sel, Ld, Ls)
    nc, ns, nd = O.tier_pages(n_pages, Ld, Ls)
    want = np.nonzero(valid[:nc * 16] & sel[:nc * 16])[0]
    got = [pool[ph, t] for e in res.pages if e.kind == "new" for (ph, t) in e.src]
    np.testing.assert_array_equal(np.array(got).reshape(-1, D), rows[want].reshape(-1, D))
    news = [e for e in res.pages if e.kind == "new"]
    assert all(e.mask == 0xFFFF for e in news[:-1])
    assert res.n_new == -(-len(want) // 16)
    kept = [e.phys for e in res.pages if e.kind != "new"]
    assert set(kept).isdisjoint(res.freed)
    assert sorted(kept + res.freed) == sorted(ids.tolist())
    total_valid = sum(bin(e.mask).count("1") for e in res.pages)
    sparse_sel = int(np.sum(valid[nc * 16:(nc + ns) * 16] & sel[nc * 16:(nc + ns) * 16]))
    dense_valid = int(np.sum(valid[(nc + ns) * 16:]))
    assert total_valid == len(want) + sparse_sel + dense_valid
    kinds = [e.kind for e in res.pages]
    assert kinds == sorted(kinds, key=["new", "sparse", "dense"].index)


# ---------------------------------------------------------------- decode (a5)
def test_decode_golden(golden_dir):
    g = _golden(golden_dir, "decode_hand.json")
    o, lse = O.decode_head(np.array(g["q"]), np.array(g["keys"]), np.array(g["vals"]),
                           np.ones(2, bool), g["sm_scale"])
    np.testing.assert_allclose(o, g["o"], atol=1e-13)
    np.testing.assert_allclose(lse, g["lse"], atol=1e-13)


def test_decode_single_slot_and_empty():
    q = RNG.standard_normal((3, 8))
    k = RNG.standard_normal((5, 8))
    v = RNG.standard_normal((5, 8))
    valid = np.zeros(5, bool)
    valid[2] = True
    o, lse = O.decode_head(q, k, v, valid, 0.4)
    np.testing.assert_array_equal(o, np.tile(v[2], (3, 1)))
    np.testing.assert_allclose(lse, 0.4 * q @ k[2], rtol=1e-15)
    o, lse = O.decode_head(q, k, v, np.zeros(5, bool), 0.4)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_decode_matches_scipy_softmax():
    q = RNG.standard_normal((4, 16))
    k = RNG.standard_normal((40, 16))
    v = RNG.standard_normal((40, 16))
    valid = RNG.random(40) < 0.7
    o, lse = O.decode_head(q, k, v, valid, 0.25)
    pr = sps.softmax(0.25 * q @ k[valid].T, axis=1)
    np.testing.assert_allclose(o, pr @ v[valid], rtol=1e-12)
    np.testing.assert_allclose(lse, sps.logsumexp(0.25 * q @ k[valid].T, axis=1), rtol=1e-13)


def test_merge_over_partitions_equals_whole():
    q = RNG.standard_normal((2, 8))
    k = RNG.standard_normal((30, 8)) * 2
    v = RNG.standard_normal((30, 8))
    valid = np.ones(30, bool)
    o_all, lse_all = O.decode_head(q, k, v, valid, 1.0)
    for cuts in ([10], [3, 17, 29], [1, 2, 3, 4]):
        parts = np.split(np.arange(30), cuts)
        o, lse = O.decode_head(q, k[parts[0]], v[parts[0]], np.ones(len(parts[0]), bool), 1.0)
        for idx in parts[1:]:
            o2, lse2 = O.decode_head(q, k[idx], v[idx], np.ones(len(idx), bool), 1.0)
            o, lse = O.merge_states(o, lse, o2, lse2)
        np.testing.assert_allclose(o, o_all, rtol=1e-12)
        np.testing.assert_allclose(lse, lse_all, rtol=1e-13)
    # empty state is the identity of the merge
    o, lse = O.merge_states(o_all, lse_all, np.zeros_like(o_all), np.full(2, -np.inf))
    np.testing.assert_allclose(o, o_all, rtol=1e-15)


# ---------------------------------------------------------------- append (a6)
def test_append_position():
    assert O.append_position([], 0) == (0, 0, True)
    assert O.append_position([0xFFFF], 1) == (1, 0, True)
    assert O.append_position([0xFFFF, 0x001F], 2) == (1, 5, False)
    assert O.append_position([0xFFFF, 0x8000], 2) == (2, 0, True)
    assert O.append_position([0x0101], 1) == (0, 9, False)


# ---------------------------------------------------------------- whole chain
def test_chain_uniform_logits_select_ceil_pN():
    """Zero keys give uniform attention, so the chain keeps exactly ceil(p N) slots."""
    N, R, D = 200, 8, 4
    q = RNG.standard_normal((R, D))
    k = np.zeros((N, D))
    valid = np.ones(N, bool)
    s, _ = O.score_head(q, k, valid, N, 0.5)
    c, _ = O.calibrate_head(s, valid)
    for p in (0.5, 0.9, 0.95):
        assert O.topp_head(c.astype(np.float32), valid, p).k == math.ceil(p * N)


# ---------------------------------------------------------------- hard budget (Step 4)
def test_score_rows_match_scipy_softmax_and_mean():
    q, k = _rand_head(R=5, S=37, D=8, seed=21, scale=1.5)
    valid = RNG.random(37) > 0.2
    z = 0.7 * (q @ k.T)
    lse = np.array([sps.logsumexp(z[r, valid]) for r in range(5)])
    a = O.score_rows_head(q, k, valid, 37, 0.7, lse)
    for r in range(5):
        ref = np.zeros(37)
        ref[valid] = sps.softmax(z[r, valid])
        np.testing.assert_allclose(a[r], ref, rtol=1e-12, atol=0)
    # with a dense tail, the rows are the same probabilities, zero past cand_len
    a2 = O.score_rows_head(q, k, valid, 20, 0.7, lse)
    np.testing.assert_array_equal(a2[:, 20:], 0.0)
    np.testing.assert_allclose(a2[:, :20], a[:, :20], rtol=1e-15)
    s, _ = O.score_head(q, k, valid, 37, 0.7)
    np.testing.assert_allclose(np.log(a.mean(axis=0)[valid]), s[valid], rtol=1e-12)


def test_vote_golden(golden_dir):
    g = _golden(golden_dir, "vote_hand.json")
    cand = np.array(g["valid"])
    votes, row_k, row_sel = O.vote_head(np.array(g["a_rows"]), cand, g["p"])
    assert votes.tolist() == g["votes"]
    assert row_k.tolist() == g["row_k"]
    assert row_sel.sum(axis=1).tolist() == g["row_k"]


def test_vote_invariants():
    r = np.random.default_rng(5)
    S = 50
    cand = r.random(S) > 0.15
    a = r.dirichlet(np.full(S, 0.3), size=6)
    for p in (0.3, 0.9, 1.0):
        votes, row_k, row_sel = O.vote_head(a, cand, p)
        # one row is the Top-p rule itself
        one = O.topp_head(a[2], cand, p)
        v1, k1, _ = O.vote_head(a[2:3], cand, p)
        assert np.array_equal(v1 == 1, one.sel) and k1[0] == one.k
        # the rows vote independently: any row order gives the same votes
        vp, _, _ = O.vote_head(a[::-1], cand, p)
        assert np.array_equal(vp, votes)
        # votes count the rows' selections, never outside the candidates
        assert np.array_equal(votes, row_sel.sum(axis=0))
        assert votes[~cand].max(initial=0) == 0 and votes.max() <= 6
    # identical rows vote together
    same = np.repeat(a[:1], 4, axis=0)
    vs, _, _ = O.vote_head(same, cand, 0.8)
    assert set(np.unique(vs)) <= {0, 4}


def test_budget_plan_cases():
    full = [0xFFFF] * 10
    # 10 pages = 160 slots of memory > L_upper 128: rewrite; 2 dense pages leave 96 slots
    assert O.budget_plan_head(10, full, 32, 64, 128) == (O.REWRITE, 96)
    # exactly L_upper is not above it; 100 valid > L_lower: sparse loading
    holes = [0xFFFF] * 6 + [0x0FFF, 0x0FFF]
    assert O.budget_plan_head(8, holes, 32, 64, 128) == (O.SPARSE, -1)
    # 60 valid slots in 8 pages: keep
    few = [0x00FF] * 7 + [0x000F]
    assert O.budget_plan_head(8, few, 32, 64, 128) == (O.KEEP, -1)
    # L_upper not a multiple of 16 rounds down; the dense tier may use the whole budget
    assert O.budget_plan_head(3, full, 32, 0, 40) == (O.REWRITE, 0)
    assert O.budget_plan_head(5, full, 0, 0, 70) == (O.REWRITE, 64)


def test_budget_select_golden(golden_dir):
    g = _golden(golden_dir, "vote_hand.json")["budget"]
    cand = np.ones(len(g["votes"]), bool)
    sel, k = O.budget_select_head(cand, votes=np.array(g["votes"]), c=np.array(g["c"]),
                                  mode=O.REWRITE, k_cap=g["k_cap"], n_sink=g["n_sink"])
    assert np.nonzero(sel)[0].tolist() == g["sel"] and k == len(g["sel"])


@pytest.mark.parametrize("trial", range(30))
def test_budget_select_ranking_brute(trial):
    r = np.random.default_rng(100 + trial)
    S = int(r.integers(1, 14))
    cand = r.random(S) > 0.2
    votes = r.integers(0, 4, S)
    c = np.round(r.random(S), 1)           # coarse values: plenty of ties
    n_sink = int(r.integers(0, 3))
    k_cap = int(r.integers(-1, S + 2))
    sel, k = O.budget_select_head(cand, votes=votes, c=c, mode=O.REWRITE, k_cap=k_cap,
                                  n_sink=n_sink)
    sinks = cand & (np.arange(S) < n_sink)
    base = cand & ~sinks & (votes >= 1)
    assert np.array_equal(sel & sinks, sinks) and not (sel & ~cand).any()
    kept, dropped = np.nonzero(sel & base)[0], np.nonzero(base & ~sel)[0]
    want = base.sum() if k_cap < 0 else min(base.sum(), max(0, k_cap - sinks.sum()))
    assert len(kept) == want and k == want + sinks.sum()
    # every kept base slot outranks every dropped one (votes, then c, then slot index)
    for i in kept:
        for j in dropped:
            assert (votes[i], c[i], i) > (votes[j], c[j], j)


def test_budget_select_reduces_to_topp_cap():
    r = np.random.default_rng(77)
    S = 60
    cand = r.random(S) > 0.1
    c = r.dirichlet(np.full(S, 0.5)).astype(np.float32)
    c[[3, 9, 20]] = c[7]                   # ties
    top = O.topp_head(c, cand, 0.9)
    prev = None
    for cap in range(0, top.k + 3):
        sel, k = O.budget_select_head(cand, c=c, sel_in=top.sel, mode=O.REWRITE, k_cap=cap)
        ref = O.topp_head(c, cand, 0.9, k_min=0, k_max=cap) if cap > 0 else None
        if ref is not None:
            assert np.array_equal(sel, ref.sel if cap < top.k else top.sel)
        else:
            assert k == 0
        if prev is not None:
            assert not (prev & ~sel).any()  # caps nest
        prev = sel
    # no cap keeps the Top-p set; KEEP keeps every candidate
    assert np.array_equal(O.budget_select_head(cand, c=c, sel_in=top.sel)[0], top.sel)
    assert np.array_equal(O.budget_select_head(cand, c=c, mode=O.KEEP)[0], cand)


@pytest.mark.parametrize("seed", range(40))
def test_budget_chain_respects_L_upper(seed):
    """plan -> select -> compact: a rewritten head never holds more than L_upper slots,
    sparse loading moves no page, and a kept head is unchanged."""
    r = np.random.default_rng(seed)
    n = int(r.integers(1, 40))
    masks = [int(m) for m in r.integers(1, 1 << 16, n)]
    masks[-1] |= 1
    table = list(r.permutation(200)[:n])
    n_valid = sum(bin(m).count("1") for m in masks)
    L_dense = int(r.integers(0, 80))
    want = seed % 3                        # thresholds drawn on the wanted side
    if want == O.REWRITE:
        L_upper = int(r.integers(0, 16 * n))
        L_lower = int(r.integers(0, L_upper + 1))
    else:
        L_upper = 16 * n + int(r.integers(0, 100))
        L_lower = int(r.integers(0, n_valid)) if want == O.SPARSE else n_valid + int(r.integers(0, 50))
    mode, k_cap = O.budget_plan_head(n, masks, L_dense, L_lower, L_upper)
    assert mode == want
    valid = ((np.array(masks)[:, None] >> np.arange(16)) & 1).reshape(-1).astype(bool)
    nd = O.tier_pages(n, L_dense, 0)[2]
    cand = O.candidate_mask(valid, 16 * (n - nd))
    votes = r.integers(0, 3, 16 * n)
    n_sink = int(r.integers(0, 20))
    sel, k = O.budget_select_head(cand, votes=votes, c=r.random(16 * n), mode=mode,
                                  k_cap=k_cap, n_sink=n_sink)
    res = O.compact_mode_head(table, masks, n, sel, L_dense, mode)
    n_sinks = int((cand & (np.arange(16 * n) < n_sink)).sum())
    if mode == O.REWRITE:
        if n_sinks <= k_cap and 16 * nd <= L_upper:
            assert 16 * len(res.pages) <= L_upper
        assert sum(bin(p.mask).count("1") for p in res.pages if p.kind == "new") == \
            int((sel & cand).sum())
    elif mode == O.SPARSE:
        kept = [p.phys for p in res.pages]
        assert kept == [t for t in table if t in kept] and res.n_new == 0
    else:
        assert [p.phys for p in res.pages] == table and res.freed == []


# ---------------------------------------------------------------- temperature by gradient descent
def test_solve_T_gd_two_level_closed_form(golden_dir):
    """Alg. 1 reaches the two-level closed form of the temperature."""
    for n, k, a, b, mass in [(100, 10, 1.0, 0.0, 0.5), (400, 7, 2.0, -1.0, 0.3), (50, 25, 0.5, 0.0, 0.8)]:
        x = np.full(n, b)
        x[:k] = a
        cand = np.ones(n, bool)
        T, loss = O.solve_T_gd_head(x, cand, k, mass, iters=400)
        closed = (a - b) / math.log(mass * (n - k) / (k * (1 - mass)))
        assert T == pytest.approx(closed, rel=1e-3) and loss < 1e-10


def test_solve_T_gd_gradient_matches_finite_differences():
    r = np.random.default_rng(3)
    x = r.standard_normal(60) * 2
    top = np.zeros(60, bool)
    top[np.argsort(-x)[:9]] = True
    for theta in (-1.0, 0.0, 0.7):
        def mass(th):
            return sps.softmax(x * math.exp(-th))[top].sum()
        M, dM = O.topk_mass_and_grad(x, top, theta)
        assert M == pytest.approx(mass(theta), rel=1e-12)
        h = 1e-5     # central difference: error O(h^2) plus rounding O(1e-16 / h)
        assert dM == pytest.approx((mass(theta + h) - mass(theta - h)) / (2 * h), rel=1e-4)


def test_solve_T_gd_edges():
    x = np.array([3.0, 1.0, 0.0, -2.0])
    cand = np.ones(4, bool)
    assert O.solve_T_gd_head(x, cand, 2, 0.7, T_init=2.5, iters=0)[0] == 2.5
    T, loss = O.solve_T_gd_head(x, cand, 2, 0.7, iters=300)
    _, loss0 = O.solve_T_gd_head(x, cand, 2, 0.7, iters=1)
    assert loss <= loss0
    # agrees with the bisection of App. D.1 on the same problem
    assert T == pytest.approx(O.solve_T_head(x, cand, 2, 0.7), rel=1e-3)
    # an early stop leaves the loss below the tolerance
    T2, l2 = O.solve_T_gd_head(x, cand, 2, 0.7, iters=300, tol=1e-8)
    assert l2 < 1e-8
    # no candidates: no mass and no gradient, so Adam never moves and the loss is target^2
    none = np.zeros(4, bool)
    assert O.topk_mass_and_grad(np.zeros(0), np.zeros(0, bool), 0.3) == (0.0, 0.0)
    T3, l3 = O.solve_T_gd_head(x, none, 2, 0.7, T_init=1.7, iters=50)
    assert T3 == pytest.approx(1.7, rel=1e-15) and l3 == pytest.approx(0.49, rel=1e-15)


def test_solve_T_gd_first_adam_step():
    """Adam's bias-corrected first step moves theta = log T by exactly lr against the
    gradient's sign (m_hat / sqrt(v_hat) = g / |g|), whatever the gradient's size."""
    x = np.array([3.0, 1.0, 0.0, -2.0])
    cand = np.ones(4, bool)
    top = np.array([True, True, False, False])
    for target, lr in ((0.99, 0.05), (0.5, 0.2)):
        M, dM = O.topk_mass_and_grad(x, top, 0.0)
        g = 2 * (M - target) * dM
        T, _ = O.solve_T_gd_head(x, cand, 2, target, T_init=1.0, lr=lr, iters=1)
        assert math.log(T) == pytest.approx(-lr * math.copysign(1.0, g), rel=1e-6)


def test_topp_p_is_quantised_to_1e_6():
    """p counts in steps of 1e-6 (round half to even): ten equal values need exactly three
    slots for p = 0.3 and for any p that rounds to 0.300000, and a fourth as soon as p
    rounds to 0.300001 (its target then exceeds three equal weights)."""
    c = np.full(10, 0.1, np.float32)
    cand = np.ones(10, bool)
    assert O.topp_head(c, cand, 0.3).k == 3
    assert O.topp_head(c, cand, 0.3000004).k == 3
    assert O.topp_head(c, cand, 0.2999996).k == 3
    assert O.topp_head(c, cand, 0.3000006).k == 4
    # the target is ceil(p_q * Total / 10^6) in exact integers
    r = O.topp_head(c, cand, 0.3000006)
    w = int(math.floor(float(np.float32(0.1)) * 2 ** 40))
    assert r.total == 10 * w and r.target == -(-(300001 * 10 * w) // 10 ** 6)

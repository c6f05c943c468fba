"""CPU checks of the test library's own restatements (the rewrite's page list and the
budget-selection rule), which the chained GPU tests use in place of the oracle where the
input is the GPU's own selection: on seeded inputs they agree with the oracle, and a set the
oracle did not choose fails the budget rule."""
import numpy as np
import pytest

import oracle as O
from hk_testlib import check_budget_selection, rewrite_layout

assert (O.KEEP, O.SPARSE, O.REWRITE) == (0, 1, 2)


def _pages(r):
    return [(e.kind, e.mask, e.phys if e.kind != "new" else -1,
             [tuple(map(int, x)) for x in e.src]) for e in r.pages]


@pytest.mark.parametrize("seed", range(12))
def test_rewrite_layout_matches_the_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 40))
    table = rng.permutation(200)[:n]
    mask = rng.integers(0, 1 << 16, n)
    mask[rng.random(n) < 0.2] = 0xFFFF
    mask[rng.random(n) < 0.1] = 0
    sel = rng.random(16 * n + 16) < rng.uniform(0.05, 0.95)
    L_dense = int(rng.choice([0, 1, 16, 48, 700]))
    L_sparse = int(rng.choice([0, 16, 96, 4000]))
    got = rewrite_layout(table, mask, n, sel, L_dense, O.REWRITE, L_sparse)
    assert _pages(got) == _pages(O.compact_head(table, mask, n, sel, L_dense, L_sparse))
    for mode in (O.KEEP, O.SPARSE, O.REWRITE):
        got = rewrite_layout(table, mask, n, sel, L_dense, mode)
        assert _pages(got) == _pages(O.compact_mode_head(table, mask, n, sel, L_dense, mode))


@pytest.mark.parametrize("seed", range(20))
def test_budget_rule_accepts_the_oracle_and_rejects_other_sets(seed):
    rng = np.random.default_rng(100 + seed)
    S = int(rng.choice([32, 64, 320]))
    cand = rng.random(S) < 0.8
    cand[int(rng.integers(0, S)):] &= rng.random() < 0.5
    votes = rng.integers(0, 4, S)
    mode = int(rng.integers(0, 3))
    cap = int(rng.integers(-1, S // 2))
    n_sink = int(rng.choice([0, 4]))
    ref, k = O.budget_select_head(cand, votes=votes, mode=mode, k_cap=cap, n_sink=n_sink)
    check_budget_selection(ref, k, cand, votes, mode, cap, n_sink)
    # flip one slot: a set the rule does not define fails it (or its count does)
    j = int(rng.integers(0, S))
    bad = ref.copy()
    bad[j] = not bad[j]
    with pytest.raises(AssertionError):
        check_budget_selection(bad, int(bad.sum()), cand, votes, mode, cap, n_sink)


def test_workload_head_lengths():
    """The generator's length mix: head h keeps ceil(len/16) pages with its last one filled
    to the length, released pages rejoin the free list in address order, and every pool
    page is either live once or free once; the draws are those of the unshortened cache."""
    import workload as WL
    cfg = dict(L=1, B=2, Hq=4, Hkv=2, D=16, N=100, dtype="f32", W=4, seed=3, recipe="normal")
    lens = [100, 0, 17, 64]
    full = WL.make_workload(cfg)
    w = WL.make_workload(cfg, head_lens=lens)
    n, table, mask = w.n_pages.numpy(), w.page_table.numpy(), w.page_mask.numpy().astype(np.int64) & 0xFFFF
    assert n.tolist() == [7, 0, 2, 4]
    for h, ln in enumerate(lens):
        bits = ((mask[h, :n[h], None] >> np.arange(16)) & 1).reshape(-1)
        assert bits.sum() == ln and (bits[:ln] == 1).all()
        assert (table[h, n[h]:] == -1).all() and (mask[h, n[h]:] == 0).all()
        assert np.array_equal(table[h, :n[h]], full.page_table.numpy()[h, :n[h]])
    top = int(w.free_top.item())
    free = w.free_ids.numpy()[:top]
    assert np.array_equal(free, np.sort(free))
    live = [int(p) for h in range(4) for p in table[h, :n[h]]]
    assert len(set(live)) == len(live) and not set(live) & set(free.tolist())
    assert len(live) + top == w.k_pool.shape[0]
    assert all(np.array_equal(w.k_pool[p].numpy(), full.k_pool[p].numpy()) for p in live)

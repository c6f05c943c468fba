"""Shared test helpers: host copies of device inputs for the oracle, bit unpacking,
and the parity comparisons with their tolerances (test infrastructure only)."""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle as O

RTOL = {"bf16": 2e-3, "f32": 1e-5}


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def np_i(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


class HostCache:
    """Host snapshot of a paged cache (tables, masks, counts, pools) for the oracle."""

    def __init__(self, k_pool, v_pool, page_table, page_mask, n_pages, heads=None):
        self.table = np_i(page_table).astype(np.int64)
        self.mask = np_i(page_mask).astype(np.int64) & 0xFFFF
        self.n = np_i(n_pages).astype(np.int64)
        if heads is None:
            self.k = k_pool.detach().float().cpu().numpy()
            self.v = v_pool.detach().float().cpu().numpy() if v_pool is not None else None
            self.ids = None
        else:
            ids = sorted({int(i) for h in heads for i in self.table[h, :self.n[h]]})
            self.ids = {pid: r for r, pid in enumerate(ids)}
            idx = torch.tensor(ids, dtype=torch.long, device=k_pool.device)
            self.k = k_pool.index_select(0, idx).float().cpu().numpy() if ids else None
            self.v = v_pool.index_select(0, idx).float().cpu().numpy() if ids and v_pool is not None else None

    def _local(self, h):
        row = self.table[h, :self.n[h]]
        if self.ids is None:
            return row
        return np.array([self.ids[int(i)] for i in row], dtype=np.int64)

    def head(self, h):
        rows, valid = O.read_head(self.k, self._local(h), self.mask[h], int(self.n[h]))
        return rows.astype(np.float64), valid

    def head_v(self, h):
        rows, valid = O.read_head(self.v, self._local(h), self.mask[h], int(self.n[h]))
        return rows.astype(np.float64), valid


def q_rows(q_obs_np, h, Hkv, G):
    """The R = W*G window rows of head h (sequence h // Hkv, KV head h % Hkv)."""
    s, kv = divmod(h, Hkv)
    W, D = q_obs_np.shape[0], q_obs_np.shape[-1]
    return q_obs_np[:, s, kv * G:(kv + 1) * G, :].reshape(W * G, D)


def unpack_bits(words_row: np.ndarray, S: int) -> np.ndarray:
    w = words_row.astype(np.int64) & 0xFFFFFFFF
    bits = (w[:, None] >> np.arange(32)[None, :]) & 1
    return bits.reshape(-1)[:S].astype(bool)


def check_log_scores(gpu, ref, rtol, what="s"):
    """Log-domain scores: |d| <= rtol where the reference mass is >= 1e-30; below that the
    GPU value must be <= -60 or -inf; -inf reference slots must be -inf."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    ninf = np.isneginf(ref)
    assert np.all(np.isneginf(gpu[ninf])), f"{what}: expected -inf at non-candidates"
    big = ~ninf & (ref >= math.log(1e-30))
    small = ~ninf & ~big
    if big.any():
        err = np.abs(gpu[big] - ref[big])
        assert err.max() <= rtol, f"{what}: max log error {err.max():.3g} > {rtol}"
    if small.any():
        assert np.all((gpu[small] <= -60) | np.isneginf(gpu[small])), f"{what}: tiny masses"


def check_prob(gpu, ref, rtol, what="c"):
    """|d| <= rtol*|ref| + atol with atol = rtol * max|ref| (per row)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    atol = rtol * (np.max(np.abs(ref)) if ref.size else 0.0)
    err = np.abs(gpu - ref)
    bound = rtol * np.abs(ref) + atol
    assert np.all(err <= bound), f"{what}: max excess {np.max(err - bound):.3g}"


def check_lse(gpu, ref, rtol, what="lse"):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    inf = np.isinf(ref)
    assert np.all(gpu[inf] == ref[inf]), f"{what}: infinities differ"
    err = np.abs(gpu[~inf] - ref[~inf])
    bound = rtol * np.maximum(1.0, np.abs(ref[~inf]))
    assert np.all(err <= bound), f"{what}: max excess {np.max(err - bound) if err.size else 0:.3g}"


def snapshot(w):
    """Host copy of a workload's cache state (tables, masks, counts, free list, pools)."""
    return dict(table=np_i(w.page_table).copy(), mask=np_i(w.page_mask).astype(np.int64) & 0xFFFF,
                n=np_i(w.n_pages).copy(), free=np_i(w.free_ids).copy(), top=int(w.free_top.item()),
                k=w.k_pool.detach().clone(), v=w.v_pool.detach().clone())


def check_compaction(w, before, sel_np, S, ref_fn):
    """The cache after a compaction call against ref_fn(h, sel) -> oracle CompactResult of
    each head: layout, masks, kept page ids, byte-exact rewritten rows, and a free list that
    together with the live pages accounts for every page exactly once."""
    table, mask, n_new = np_i(w.page_table), np_i(w.page_mask).astype(np.int64) & 0xFFFF, np_i(w.n_pages)
    top = int(w.free_top.item())
    free = set(np_i(w.free_ids)[:top].tolist())
    live = set()
    new_ids = []
    for h in range(table.shape[0]):
        sel = unpack_bits(sel_np[h], S)
        r = ref_fn(h, sel)
        assert n_new[h] == len(r.pages), f"n_pages head {h}"
        for pos, e in enumerate(r.pages):
            pid = int(table[h, pos])
            assert mask[h, pos] == e.mask, f"mask head {h} pos {pos}"
            assert pid not in live
            live.add(pid)
            if e.kind == "new":
                new_ids.append(pid)
                src = torch.tensor([ph * 16 + t for ph, t in e.src], device=w.k_pool.device)
                got_k = w.k_pool.view(-1, w.k_pool.shape[-1])[pid * 16: pid * 16 + len(e.src)]
                got_v = w.v_pool.view(-1, w.v_pool.shape[-1])[pid * 16: pid * 16 + len(e.src)]
                want_k = before["k"].view(-1, w.k_pool.shape[-1]).index_select(0, src)
                want_v = before["v"].view(-1, w.v_pool.shape[-1]).index_select(0, src)
                assert torch.equal(got_k.view(torch.int16) if got_k.dtype == torch.bfloat16 else got_k.view(torch.int32),
                                   want_k.view(torch.int16) if want_k.dtype == torch.bfloat16 else want_k.view(torch.int32)), \
                    f"K bytes head {h} pos {pos}"
                assert torch.equal(got_v.view(torch.int16) if got_v.dtype == torch.bfloat16 else got_v.view(torch.int32),
                                   want_v.view(torch.int16) if want_v.dtype == torch.bfloat16 else want_v.view(torch.int32)), \
                    f"V bytes head {h} pos {pos}"
            else:
                assert pid == e.phys, f"kept page head {h} pos {pos}"
        assert np.all(table[h, len(r.pages):] == -1)
        assert np.all(mask[h, len(r.pages):] == 0)
    assert live.isdisjoint(free)
    assert len(live) + len(free) == len(before["free"]), "pages lost or duplicated"
    assert set(new_ids) <= set(before["free"][:before["top"]].tolist())


def check_topp_rule(c, sel, k, cand, p, k_min=1, k_max=0, what="Top-p"):
    """Property check of a Top-p selection against the fp32 values it was made from (for
    chained stages, whose input is the GPU's own output and so not an oracle input): the
    set lies in the candidates, has k members within the clamps, ranks above every other
    candidate in (value, slot) order, reaches p of the fixed-point mass floor(c 2^40)
    (unless clamped at the top), and would not without its weakest member (unless clamped
    at the bottom)."""
    c = np.asarray(c, np.float32).astype(np.float64)
    vals = np.clip(np.where(np.isnan(c), 0.0, c), 0.0, 1.0)
    sel = np.asarray(sel, bool)
    cand = np.asarray(cand, bool)
    assert not (sel & ~cand).any(), f"{what}: selection outside the candidates"
    idx = np.nonzero(cand)[0]
    n, kk = len(idx), int(sel.sum())
    assert kk == int(k), f"{what}: k {k} but {kk} selected"
    lo, hi = min(max(k_min, 0), n), (n if k_max <= 0 else min(k_max, n))
    assert lo <= kk <= hi, f"{what}: k {kk} outside [{lo}, {hi}]"
    w = {int(j): int(math.floor(vals[j] * 2.0 ** 40)) for j in idx}
    total = sum(w.values())
    pq = int(round(float(p) * 10 ** 6))
    chosen = [int(j) for j in idx if sel[j]]
    rest = [int(j) for j in idx if not sel[j]]
    if chosen and rest:
        assert min((vals[j], j) for j in chosen) > max((vals[j], j) for j in rest), \
            f"{what}: a dropped candidate outranks a kept one"
    m = sum(w[j] for j in chosen)
    assert kk == hi or 10 ** 6 * m >= pq * total, f"{what}: mass below p"
    if chosen and kk > lo:
        weakest = min(chosen, key=lambda j: (vals[j], j))
        assert 10 ** 6 * (m - w[weakest]) < pq * total, f"{what}: not the smallest such set"


def rewritten_sources(table_row, mask_row, n_pages, sel, n_condensed):
    """(physical page, slot) of every selected valid slot of the condensed band, in
    ascending logical order: what a rewrite must copy, in that order."""
    out = []
    for pp in range(n_condensed):
        m = int(mask_row[pp])
        for t in range(16):
            if (m >> t) & 1 and sel[pp * 16 + t]:
                out.append((int(table_row[pp]), t))
    return out

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
    """The cache after a compaction call against ref_fn(h, sel) -> the expected page list of
    each head (the oracle's compaction for a seeded selection, rewrite_layout for the GPU's
    own): layout, masks, kept page ids, byte-exact rewritten rows, and a free list that
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
    at the bottom).  Returns the selected fixed-point mass."""
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
    return m


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


MODE_KEEP, MODE_SPARSE, MODE_REWRITE = 0, 1, 2       # a head's hard-budget state


class _Page:
    """One entry of an expected page list: kind "new" (a fresh page holding the rows src),
    "sparse" (the physical page phys kept in place) or "dense" (phys untouched)."""

    def __init__(self, kind, mask, phys=-1, src=()):
        self.kind, self.mask, self.phys, self.src = kind, mask, phys, list(src)


class _Layout:
    def __init__(self, pages):
        self.pages = pages


def rewrite_layout(table_row, mask_row, n_pages, sel, L_dense, mode=MODE_REWRITE, L_sparse=0):
    """The page list a Cascade-Cache rewrite must leave (Sec. 3.1 tiers; Sec. 3.3.1 states),
    restated from the rewrite's defining properties for tests whose selection is the GPU's
    own, so that no oracle routine is run on it:
      dense tier  the newest ceil(L_dense/16) pages, untouched and last;
      sparse band the L_sparse/16 pages before them (every non-dense page in state SPARSE,
                  none in state REWRITE), each kept in place with its mask cut by the
                  selection, dropped once empty;
      condensed   every older page: its selected valid slots in logical order, sixteen to a
                  fresh page with a full-prefix mask, first in the list.
    A head in state KEEP keeps every page as it is."""
    n = int(n_pages)
    if mode == MODE_KEEP:
        return _Layout([_Page("dense", int(mask_row[pp]), int(table_row[pp])) for pp in range(n)])
    nd = min(n, -(-int(L_dense) // 16))
    ns = n - nd if mode == MODE_SPARSE else min(n - nd, int(L_sparse) // 16)
    nc = n - nd - ns
    src = rewritten_sources(table_row, mask_row, n, sel, nc)
    pages = [_Page("new", (1 << len(src[i:i + 16])) - 1, src=src[i:i + 16])
             for i in range(0, len(src), 16)]
    for pp in range(nc, nc + ns):
        kept = sum(1 << t for t in range(16) if sel[pp * 16 + t]) & int(mask_row[pp])
        if kept:
            pages.append(_Page("sparse", kept, int(table_row[pp])))
    pages += [_Page("dense", int(mask_row[pp]), int(table_row[pp])) for pp in range(nc + ns, n)]
    return _Layout(pages)


def check_budget_selection(got, k, cand, votes, mode, cap, n_sink, what="budget"):
    """Property check of a budget selection made from the GPU's own votes (Sec. 3.1 Step 4
    under the hard budget): a KEEP head selects every candidate; otherwise the sinks (the
    first n_sink candidates' slots) are all kept, nothing outside the sinks and the voted
    candidates is taken, the voted candidates taken number min(voted, cap - sinks) (all of
    them when there is no cap) and outrank every voted candidate left out in (votes, slot)
    order, and k counts the set."""
    got, cand = np.asarray(got, bool), np.asarray(cand, bool)
    S = len(cand)
    assert not (got & ~cand).any() and int(k) == int(got.sum()), f"{what}: set or count"
    if mode == MODE_KEEP:
        assert np.array_equal(got, cand), f"{what}: KEEP head"
        return
    sinks = cand & (np.arange(S) < n_sink)
    base = cand & ~sinks & (np.asarray(votes) >= 1)
    assert np.array_equal(got & sinks, sinks) and not (got & ~sinks & ~base).any(), what
    want = base.sum() if cap < 0 else min(base.sum(), max(0, int(cap) - int(sinks.sum())))
    assert (got & base).sum() == want, f"{what}: {(got & base).sum()} voted kept, want {want}"
    kept, dropped = np.nonzero(got & base)[0], np.nonzero(base & ~got)[0]
    if len(kept) and len(dropped):
        assert min((votes[j], j) for j in kept) > max((votes[j], j) for j in dropped), \
            f"{what}: a dropped candidate outranks a kept one"


class DecodeReplay:
    """Host model of a decode loop's cache (append, decode attention, periodic compression)
    for a set of heads, built on the oracle: per head its pages in logical order with their
    16-slot masks and K/V rows.  Each step appends a row where the oracle's append_position
    puts it and returns the oracle's decode attention over the valid slots; each compression
    checks the GPU's scores and selection against the model and then rewrites the model with
    the GPU's selection, once that selection has passed the Top-p rule: near the threshold
    two fp32 computations of c may rank slots differently, so the set itself is not unique
    across implementations and the model follows the GPU's valid one.  Heads are (layer, sequence, KV head) rows of the
    loop's cache, h // Hkv the sequence s.  Step inputs are host arrays [n, H*, D] whose row
    sidx[s] holds sequence s (sidx=None: row s)."""

    def __init__(self, w, heads, Hkv, G, D, scale, max_pages):
        self.heads, self.Hkv, self.G, self.D, self.scale = list(heads), Hkv, G, D, scale
        host = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages, heads=self.heads)
        self.K, self.V, self.mask, self.n = {}, {}, {}, {}
        for h in self.heads:
            n = int(host.n[h])
            K, _ = host.head(h)
            V, _ = host.head_v(h)
            self.K[h] = np.zeros((max_pages, 16, D))
            self.V[h] = np.zeros((max_pages, 16, D))
            self.K[h][:n], self.V[h][:n] = K.reshape(n, 16, D), V.reshape(n, 16, D)
            self.mask[h] = [int(m) for m in host.mask[h][:n]]
            self.n[h] = n
        self._pack()

    def _pack(self):
        # the valid rows in logical order (an append always lands after every valid slot,
        # and a rewrite keeps the order), which decode attention reads
        self.RK, self.RV, self.nr = {}, {}, {}
        for h in self.heads:
            K, valid = self.head(h)
            V, _ = self.head_v(h)
            cap = 16 * self.K[h].shape[0]
            self.RK[h], self.RV[h] = np.zeros((cap, self.D)), np.zeros((cap, self.D))
            nv = int(valid.sum())
            self.RK[h][:nv], self.RV[h][:nv] = K[valid], V[valid]
            self.nr[h] = nv

    def head(self, h):
        """(K rows of every slot [16 n, D], validity [16 n]) of head h."""
        n = self.n[h]
        valid = ((np.array(self.mask[h], np.int64)[:, None] >> np.arange(16)) & 1).reshape(-1).astype(bool)
        return self.K[h][:n].reshape(-1, self.D), valid

    def head_v(self, h):
        return self.V[h][:self.n[h]].reshape(-1, self.D), self.head(h)[1]

    def step(self, q_t, k_t, v_t, sidx=None, decode=True):
        """Append one step's rows and (decode=True) return the oracle's decode output and LSE
        of every modelled head for that step's queries: {h: (o [G, D], lse [G])}."""
        out = {}
        for h in self.heads:
            s, kvh = divmod(h, self.Hkv)
            r = s if sidx is None else sidx[s]
            pos, slot, new = O.append_position(self.mask[h], self.n[h])
            if new:
                self.mask[h].append(0)
                self.n[h] += 1
            self.K[h][pos, slot], self.V[h][pos, slot] = k_t[r, kvh], v_t[r, kvh]
            self.mask[h][pos] |= 1 << slot
            nr = self.nr[h]
            self.RK[h][nr], self.RV[h][nr] = k_t[r, kvh], v_t[r, kvh]
            self.nr[h] = nr + 1
            if decode:
                out[h] = O.decode_head(np.asarray(q_t[r, kvh * self.G:(kvh + 1) * self.G], np.float64),
                                       self.RK[h][:nr + 1], self.RV[h][:nr + 1], np.ones(nr + 1, bool),
                                       self.scale)
        return out

    def check_cache(self, w, what):
        """The GPU cache equals the model: page counts and masks exactly, K and V of every
        valid slot byte for byte."""
        now = HostCache(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages, heads=self.heads)
        for h in self.heads:
            n = self.n[h]
            assert int(now.n[h]) == n, f"{what}: head {h} has {int(now.n[h])} pages, model {n}"
            assert [int(m) for m in now.mask[h][:n]] == self.mask[h], f"{what}: masks of head {h}"
            K, valid = now.head(h)
            V, _ = now.head_v(h)
            Km, vm = self.head(h)
            Vm, _ = self.head_v(h)
            assert np.array_equal(K[valid], Km[vm]) and np.array_equal(V[valid], Vm[vm]), \
                f"{what}: K/V rows of head {h} differ from the model"

    def compress(self, q_win, lse_win, s_gpu, c_gpu, sel_gpu, k_gpu, L_dense, p, S, what, sidx=None):
        """One compression of every modelled head (the model holds the cache the compression
        saw): the GPU scores (single pass over the decode LSEs) against the oracle's score fed
        the oracle's own window LSEs, and the GPU's selection by the Top-p rule on its own
        probabilities; the model is then rewritten to the page list the rewrite defines for
        that selection (rewrite_layout: no oracle routine is run on the GPU's selection).  q_win [W, n, Hq, D] host; lse_win {h: [W, G]} oracle LSEs; s_gpu, c_gpu,
        sel_gpu: {h: the head's row}; k_gpu [n_heads]."""
        for h in self.heads:
            s, kvh = divmod(h, self.Hkv)
            r = s if sidx is None else sidx[s]
            n = self.n[h]
            Kfull, valid = self.head(h)
            nd = O.tier_pages(n, L_dense, 0)[2]
            cand_len = 16 * (n - nd)
            q_rows_h = np.asarray(q_win[:, r, kvh * self.G:(kvh + 1) * self.G], np.float64).reshape(-1, self.D)
            s_ref, _ = O.score_head(q_rows_h, Kfull, valid, cand_len, self.scale,
                                    row_lse_in=np.asarray(lse_win[h]).reshape(-1))
            full = np.full(S, -np.inf)
            full[:len(s_ref)] = s_ref
            check_log_scores(s_gpu[h], full, 2e-3, f"{what}: score head {h}")
            cand = np.zeros(S, bool)
            cand[:len(valid)] = O.candidate_mask(valid, cand_len)
            sel = unpack_bits(sel_gpu[h], S)
            check_topp_rule(c_gpu[h], sel, int(k_gpu[h]), cand, p, what=f"{what}: head {h}")
            res = rewrite_layout(np.arange(n), self.mask[h], n, sel, L_dense)
            K0, V0 = self.K[h][:n].copy(), self.V[h][:n].copy()
            for i, e in enumerate(res.pages):
                if e.kind == "new":
                    for t, (ph, st) in enumerate(e.src):
                        self.K[h][i, t], self.V[h][i, t] = K0[ph, st], V0[ph, st]
                else:
                    self.K[h][i], self.V[h][i] = K0[e.phys], V0[e.phys]
            self.mask[h] = [e.mask for e in res.pages]
            self.n[h] = len(res.pages)
        self._pack()


def topp_edge_inputs(kind: str, S: int, seed: int = 7):
    """Seeded Top-p inputs of one kind over six heads of S slots whose candidate counts
    cover full, about half with a ragged tail, one, none, 33 and the last full word:
    returns (c [6][S] fp32, cand_len [6] int32, k_min, k_max, p)."""
    H = 6
    rng = np.random.default_rng(seed)
    c = np.zeros((H, S), np.float32)
    cand_len = np.array([S, S // 2 - 24, 1, 0, 33, (S - 1) // 32 * 32], np.int32)
    kmin, kmax, p = 1, 0, 0.9
    for h in range(H):
        n = cand_len[h]
        if kind == "crowded":
            # one binade, distinct low mantissa bits: the search's low-bit phase sees them all
            c[h, :n] = ((1.0 + rng.integers(0, 1 << 12, n) * 2.0 ** -12) / (2 * max(n, 1))).astype(np.float32)
        elif kind == "spread":
            # log-uniform over ~30 binades
            c[h, :n] = np.exp2(-rng.random(n) * 30.0).astype(np.float32) / max(n, 1)
        elif kind == "uniform":
            c[h, :n] = np.float32(1.0 / max(n, 1))
        elif kind == "ties":
            c[h, :n] = rng.choice(np.float32([0.5, 0.25, 0.125]), n) / max(n, 1)
        elif kind == "onehot":
            if n:
                c[h, rng.integers(0, n)] = 1.0
        elif kind == "nan_range":
            c[h, :n] = rng.random(n).astype(np.float32) / max(n, 1)
            if n > 3:
                c[h, 1] = np.nan
                c[h, 2] = 3.0
                c[h, 3] = -0.5
        elif kind == "zeros":
            pass
        elif kind == "clamp":
            c[h, :n] = rng.dirichlet(np.ones(max(n, 1)))[:n].astype(np.float32)
            kmin, kmax, p = 5, 40, 0.99
        else:
            raise ValueError(kind)
    return c, cand_len, kmin, kmax, p

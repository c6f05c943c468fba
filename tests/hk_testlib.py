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

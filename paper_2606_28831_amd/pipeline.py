"""Chaining of the C entry points into one compression step and one decode step.

Marshalling only: buffers are allocated once (static shapes) and every call goes to
libhardkv.  The compression step is Steps 2-3 of the continuous compression pipeline
(Sec. 3.1): score -> calibrate -> Top-p -> rewrite; the budgeted step adds Step 4
(hard budget with Cautious Update voting and attention sinks).
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch

from . import (Allocator, PagedKV, OP_APPEND, OP_COMPACT, OP_DECODE, OP_SCORE, dims, hk_append_kv,
               hk_budget_plan, hk_budget_select, hk_calibrate, hk_calibrate_solve_T,
               hk_calibrate_solve_T_gd, hk_calibrate_topp_ws, hk_compact, hk_compact_modes, hk_decode_attn, hk_pool_max,
               hk_score, hk_score_rows, hk_vote_topp, select_workspace, workspace)


@dataclass
class CompressBuffers:
    s_attn: torch.Tensor
    s_pool: torch.Tensor | None
    x_red: torch.Tensor | None
    c: torch.Tensor
    c_attn: torch.Tensor | None
    cand_len: torch.Tensor
    row_lse: torch.Tensor
    sel_bits: torch.Tensor
    k: torch.Tensor
    sel_mass: torch.Tensor
    k_attn: torch.Tensor | None
    mass_attn: torch.Tensor | None
    T_red: torch.Tensor | None
    status: torch.Tensor
    ws_score: torch.Tensor
    ws_compact: torch.Tensor
    ws_select: torch.Tensor


class Compressor:
    """One compression step over every head of a paged cache.

    metric "attn": attention mass over the window, calibrated with T = 1.
    metric "attn+red": attention mass and key redundancy, each calibrated (the
    redundancy temperature solved once per head, on the first call), mixed 0.5/0.5.
    Calibration and Top-p run as one launch; keep_c=False leaves the calibrated
    probabilities on chip (buf.c / buf.c_attn are then not written).
    pool_radius: if set, the attention-mass scores are max-pooled along the sequence
    (Solution 1, SnapKV form) before calibration, into buf.s_pool.
    t_solver: "bisect" (App. D.1) or "gd" (Alg. 1, Adam on log T) for the redundancy
    temperature.
    """

    def __init__(self, NS, Hq, Hkv, D, W, kv: PagedKV, alloc: Allocator, p: float,
                 L_dense: int = 0, L_sparse: int = 0, metric: str = "attn", n_ref: int = 0,
                 k_max: int = 0, keep_c: bool = True, pool_radius: int | None = None,
                 t_solver: str = "bisect"):
        if t_solver not in ("bisect", "gd"):
            raise ValueError("t_solver must be 'bisect' or 'gd'")
        self.t_solver = t_solver
        self.d = dims(NS, Hq, Hkv, D, W)
        self.kv, self.alloc, self.p = kv, alloc, p
        self.L_dense, self.L_sparse = L_dense, L_sparse
        self.metric, self.n_ref, self.k_max, self.keep_c = metric, n_ref, k_max, keep_c
        self.pool_radius = pool_radius
        self.sm_scale = 1.0 / math.sqrt(D)
        dev = kv.k_pool.device
        H = NS * Hkv
        S = kv.max_pages * 16
        self.n_heads, self.S_max = H, S
        f32, i32 = torch.float32, torch.int32
        red = metric == "attn+red"
        self.buf = CompressBuffers(
            s_attn=torch.empty(H, S, dtype=f32, device=dev),
            s_pool=torch.empty(H, S, dtype=f32, device=dev) if pool_radius is not None else None,
            x_red=torch.empty(H, S, dtype=f32, device=dev) if red else None,
            c=torch.empty(H, S, dtype=f32, device=dev),
            c_attn=torch.empty(H, S, dtype=f32, device=dev) if red else None,
            cand_len=torch.empty(H, dtype=i32, device=dev),
            row_lse=torch.empty(W, NS, Hq, dtype=f32, device=dev),
            sel_bits=torch.empty(H, S // 32, dtype=i32, device=dev),
            k=torch.empty(H, dtype=i32, device=dev),
            sel_mass=torch.empty(H, dtype=f32, device=dev),
            k_attn=torch.empty(H, dtype=i32, device=dev) if red else None,
            mass_attn=torch.empty(H, dtype=f32, device=dev) if red else None,
            T_red=None,
            status=torch.zeros(1, dtype=i32, device=dev),
            ws_score=workspace(OP_SCORE, self.d, kv.max_pages, dev),
            ws_compact=workspace(OP_COMPACT, self.d, kv.max_pages, dev),
            ws_select=select_workspace(H, S, dev),
        )

    def score(self, q_obs, ref_slots=None, row_lse_in=None, stream=None):
        b = self.buf
        hk_score(self.d, q_obs, self.kv, self.L_dense, self.sm_scale, b.s_attn, b.cand_len,
                 row_lse_in=row_lse_in, row_lse_out=b.row_lse if row_lse_in is None else None,
                 ref_slots=ref_slots, n_ref=self.n_ref if ref_slots is not None else 0,
                 x_red=b.x_red if ref_slots is not None else None, ws=b.ws_score, stream=stream)

    def select(self, stream=None):
        b, H, S, pm = self.buf, self.n_heads, self.S_max, self.kv.page_mask
        s_attn = b.s_attn
        if self.pool_radius is not None:
            hk_pool_max(H, S, b.cand_len, pm, b.s_attn, self.pool_radius, b.s_pool, stream=stream)
            s_attn = b.s_pool
        if self.metric == "attn":
            xs, Ts, ws = [s_attn], None, [1.0]
        else:
            if b.T_red is None:
                # temperature of the redundancy metric, solved at the first compression only
                hk_calibrate_topp_ws(H, S, b.cand_len, pm, [s_attn], None, [1.0], self.p,
                                     b.sel_bits, b.k_attn, b.ws_select,
                                     c_out=b.c_attn if self.keep_c else None,
                                     sel_mass=b.mass_attn, status=b.status, stream=stream)
                b.T_red = torch.empty(H, dtype=torch.float32, device=b.c.device)
                solve = hk_calibrate_solve_T_gd if self.t_solver == "gd" else hk_calibrate_solve_T
                solve(H, S, b.cand_len, pm, b.x_red, b.k_attn, b.mass_attn, b.T_red, stream=stream)
            xs, Ts, ws = [s_attn, b.x_red], [None, b.T_red], [0.5, 0.5]
        hk_calibrate_topp_ws(H, S, b.cand_len, pm, xs, Ts, ws, self.p, b.sel_bits, b.k,
                             b.ws_select, c_out=b.c if self.keep_c else None, k_max=self.k_max,
                             sel_mass=b.sel_mass, status=b.status, stream=stream)

    def compact(self, stream=None):
        b = self.buf
        hk_compact(self.d, self.kv, b.sel_bits, self.L_dense, self.L_sparse, self.alloc, b.status,
                   b.ws_compact, stream=stream)

    def step(self, q_obs, ref_slots=None, row_lse_in=None, stream=None):
        self.score(q_obs, ref_slots=ref_slots, row_lse_in=row_lse_in, stream=stream)
        self.select(stream=stream)
        self.compact(stream=stream)


class BudgetCompressor:
    """One compression step under the hard budget (Sec. 3.1 Step 4 and the budget
    thresholds of Sec. 3.3.1) with Cautious Update voting (Sec. 3.1):

      budget state (keep / sparse loading / rewrite, and the cap L_upper leaves)
      -> row LSEs of the window -> every row's own probabilities -> per-row Top-p votes
      -> selection ranked by votes under the cap, sinks kept -> mode-driven rewrite.

    rank_by_c: break ties in the votes by the window's calibrated mean attention (adds the
    attention-mass pass and the calibration); otherwise by recency.  The per-row
    probabilities take n_heads * G * W * S_max * 4 bytes (buf["a_rows"]).
    """

    def __init__(self, NS, Hq, Hkv, D, W, kv: PagedKV, alloc: Allocator, p: float,
                 L_lower: int, L_upper: int, L_dense: int = 0, n_sink: int = 0,
                 rank_by_c: bool = False):
        self.d = dims(NS, Hq, Hkv, D, W)
        self.kv, self.alloc, self.p = kv, alloc, p
        self.L_lower, self.L_upper, self.L_dense, self.n_sink = L_lower, L_upper, L_dense, n_sink
        self.rank_by_c = rank_by_c
        self.sm_scale = 1.0 / math.sqrt(D)
        dev = kv.k_pool.device
        H, S, R = NS * Hkv, kv.max_pages * 16, Hq // Hkv * W
        self.n_heads, self.S_max, self.R = H, S, R
        f32, i32 = torch.float32, torch.int32
        self.buf = dict(
            head_mode=torch.empty(H, dtype=i32, device=dev),
            k_cap=torch.empty(H, dtype=i32, device=dev),
            cand_len=torch.empty(H, dtype=i32, device=dev),
            row_lse=torch.empty(W, NS, Hq, dtype=f32, device=dev),
            s_attn=torch.empty(H, S, dtype=f32, device=dev) if rank_by_c else None,
            c=torch.empty(H, S, dtype=f32, device=dev) if rank_by_c else None,
            a_rows=torch.empty(H, R, S, dtype=f32, device=dev),
            votes=torch.empty(H, S, dtype=torch.int16, device=dev),
            row_sel=torch.empty(H, R, S // 32, dtype=i32, device=dev),
            sel_bits=torch.empty(H, S // 32, dtype=i32, device=dev),
            k=torch.empty(H, dtype=i32, device=dev),
            status=torch.zeros(1, dtype=i32, device=dev),
            ws_score=workspace(OP_SCORE, self.d, kv.max_pages, dev),
            ws_compact=workspace(OP_COMPACT, self.d, kv.max_pages, dev),
        )

    def select(self, q_obs, stream=None):
        b, H, S, pm = self.buf, self.n_heads, self.S_max, self.kv.page_mask
        hk_budget_plan(self.d, self.kv, self.L_dense, self.L_lower, self.L_upper, b["head_mode"],
                       b["k_cap"], stream=stream)
        hk_score(self.d, q_obs, self.kv, self.L_dense, self.sm_scale, b["s_attn"], b["cand_len"],
                 row_lse_out=b["row_lse"], ws=b["ws_score"], stream=stream)
        hk_score_rows(self.d, q_obs, self.kv, self.L_dense, self.sm_scale, b["row_lse"],
                      b["a_rows"], stream=stream)
        hk_vote_topp(H, self.R, S, b["cand_len"], pm, b["a_rows"], self.p, b["votes"],
                     b["row_sel"], status=b["status"], stream=stream)
        if self.rank_by_c:
            hk_calibrate(H, S, b["cand_len"], pm, [b["s_attn"]], None, [1.0], b["c"], stream=stream)
        hk_budget_select(H, S, b["cand_len"], pm, b["sel_bits"], b["k"], votes=b["votes"],
                         c=b["c"], head_mode=b["head_mode"], k_cap=b["k_cap"],
                         n_sink=self.n_sink, stream=stream)

    def compact(self, stream=None):
        b = self.buf
        hk_compact_modes(self.d, self.kv, b["sel_bits"], self.L_dense, b["head_mode"], self.alloc,
                         b["status"], b["ws_compact"], stream=stream)

    def step(self, q_obs, stream=None):
        self.select(q_obs, stream=stream)
        self.compact(stream=stream)


class Decoder:
    """One decode step of one layer: append the step's K/V, then attend."""

    def __init__(self, NS, Hq, Hkv, D, kv: PagedKV, alloc: Allocator):
        self.d = dims(NS, Hq, Hkv, D, 0)
        self.kv, self.alloc = kv, alloc
        self.sm_scale = 1.0 / math.sqrt(D)
        dev = kv.k_pool.device
        self.ws = workspace(OP_DECODE, self.d, kv.max_pages, dev)
        self.ws_app = workspace(OP_APPEND, self.d, kv.max_pages, dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)

    def append(self, k_new, v_new, stream=None):
        hk_append_kv(self.d, self.kv, k_new, v_new, self.alloc, self.status, self.ws_app,
                     stream=stream)

    def attend(self, q, o, lse, stream=None):
        hk_decode_attn(self.d, q, self.kv, self.sm_scale, o, lse, self.ws, stream=stream)


class DecodeLoop:
    """End-to-end decode loop over L independent attention layers sharing one page pool
    and one allocator (config-5 style).

    step():     append this step's K/V for every layer (Step 1, dense tier), then one paged
                decode-attention launch per layer, writing o and the row LSE.
    compress(): Steps 2-3 over every layer at once, with the window queries and the decode
                step's own LSEs (single-pass score).
    Heads are ordered (layer, sequence, KV head); sequence index = layer * B + b.
    """

    def __init__(self, L, B, Hq, Hkv, D, W, kv: PagedKV, alloc: Allocator, p: float,
                 L_dense: int, L_sparse: int = 0, keep_c: bool = True):
        self.L, self.B, self.Hq, self.Hkv, self.D, self.W = L, B, Hq, Hkv, D, W
        self.kv, self.alloc = kv, alloc
        self.NS = L * B
        dev = kv.k_pool.device
        self.d_all = dims(self.NS, Hq, Hkv, D, W)
        self.d_layer = dims(B, Hq, Hkv, D, W)
        self.layers = [kv.rows(l * B * Hkv, B * Hkv) for l in range(L)]
        self.sm_scale = 1.0 / math.sqrt(D)
        self.ws_dec = workspace(OP_DECODE, self.d_layer, kv.max_pages, dev)
        self.ws_app = workspace(OP_APPEND, self.d_all, kv.max_pages, dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.o = torch.empty(self.NS, Hq, D, dtype=torch.float32, device=dev)
        self.comp = Compressor(self.NS, Hq, Hkv, D, W, kv, alloc, p, L_dense=L_dense,
                               L_sparse=L_sparse, metric="attn", keep_c=keep_c)

    def step(self, q_t, k_t, v_t, lse_t, stream=None):
        hk_append_kv(self.d_all, self.kv, k_t, v_t, self.alloc, self.status, self.ws_app,
                     stream=stream)
        B = self.B
        for l, kv_l in enumerate(self.layers):
            hk_decode_attn(self.d_layer, q_t[l * B:(l + 1) * B], kv_l, self.sm_scale,
                           self.o[l * B:(l + 1) * B], lse_t[l * B:(l + 1) * B], self.ws_dec,
                           stream=stream)

    def compress(self, q_win, lse_win, stream=None):
        self.comp.step(q_win, row_lse_in=lse_win, stream=stream)

    def segment(self, q_seg, k_seg, v_seg, lse_seg, stream=None):
        """len(q_seg) decode steps, then one compression over the last W steps' queries
        and their decode LSEs (Sec. 3.1 Steps 1-3)."""
        T = q_seg.shape[0]
        for t in range(T):
            self.step(q_seg[t], k_seg[t], v_seg[t], lse_seg[t], stream=stream)
        self.compress(q_seg[T - self.W:], lse_seg[T - self.W:], stream=stream)

    def capture_segment(self, q_seg, k_seg, v_seg, lse_seg):
        """Record one segment into a HIP graph (torch.cuda.CUDAGraph).  The graph keeps the
        buffers' addresses: refill q_seg / k_seg / v_seg in place and replay it.  Every step
        of a segment is a kernel launch on the capture stream with device-side metadata
        updates (no host synchronisation, no allocation, no memset), so one graph serves
        every segment.  Nothing runs at capture time."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.segment(q_seg, k_seg, v_seg, lse_seg)
        return g

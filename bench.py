#!/usr/bin/env python3
"""Benchmark of the Hard-KV decoding-time compression step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config {1,2,3,4,5}]

A step (configs 1-4) is one pass of the whole hot path over every head of the
workload: score -> calibrate -> Top-p -> Cascade-Cache rewrite.  The rewrite
mutates the cache, so before each step the small metadata (tables, masks, page
counts, free list) is restored to its pristine copy -- the K/V pages themselves
are never overwritten by a rewrite (it writes only freshly popped pages), so the
pristine cache is whole again.  The restore (a few MB of device copies) stays
inside the timed region, which makes the reported rate slightly conservative.

Config 5 runs the end-to-end decode loop (append + paged decode attention per
layer per step, compression every 128 steps) and reports decode tokens/s.

Prints ONE JSON line (rank 0).  value = compressed KV tokens/s = candidate
(head, slot) pairs processed per second.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
EVENT_EVERY = 4          # steps of the timed region whose dominant-kernel launches carry events
BF16_PEAK_TFLOPS = 2500.0
METRIC = "compressed KV tokens/s (score+Top-p+compact) & % HBM peak; decode tok/s"


def _events(n):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def _esize(cfg):
    return 2 if cfg["dtype"] == "bf16" else 4


def _cand_tokens(w, L_dense):
    """Candidate (head, slot) pairs of the pristine cache: valid slots older than the dense tier."""
    m = w.page_mask.to(torch.int32) & 0xFFFF
    bits = ((m[:, :, None] >> torch.arange(16, device=m.device, dtype=torch.int32)) & 1)
    n = w.n_pages.long()
    nd = torch.clamp(n, max=-(-L_dense // 16))
    pos = torch.arange(w.max_pages, device=m.device)[None, :]
    cand_pages = pos < (n - nd)[:, None]
    return int((bits.sum(-1) * cand_pages).sum().item())


def _condensed_kept(w, sel_bits, L_dense, L_sparse):
    """Selected slots inside the condensed tier (the rows the rewrite copies), per the
    pristine page counts: dense = newest ceil(L_dense/16) pages, sparse = the
    floor(L_sparse/16) pages before them, condensed = the rest."""
    n = w.n_pages.long()
    nd = torch.clamp(n, max=-(-L_dense // 16))
    ns = torch.minimum(n - nd, torch.full_like(n, L_sparse // 16))
    nc = n - nd - ns
    words = sel_bits.to(torch.int64) & 0xFFFFFFFF
    bits = (words[:, :, None] >> torch.arange(32, device=words.device)) & 1
    bits = bits.reshape(words.shape[0], -1)
    pos = torch.arange(bits.shape[1], device=bits.device)[None, :]
    return int((bits * (pos < 16 * nc[:, None])).sum().item())


# source file of each timed kernel (a stored counter reading is only valid for that source)
ROOFLINE_KERNELS = ("score_pass1", "score_pass2", "compact_gather", "decode_split")
BUDGET_ROOFLINE_KERNELS = ("score_pass1", "score_rows", "vote", "compact_gather")
KERNEL_SOURCE = {"score_pass1": "hk_score.hip", "score_pass2": "hk_score.hip",
                 "compact_gather": "hk_compact.hip", "decode_split": "hk_decode.hip",
                 "score_rows": "hk_score.hip", "vote": "hk_budget.hip"}

# hard-budget workload (Step 4): Cautious Update votes, L_lower = L_upper / 2 with the
# paper's 4096-token budget, four attention sinks
BUDGET = {"L_lower": 2048, "L_upper": 4096, "n_sink": 4}


def _source_sha(kernel):
    """sha256 over the kernel's source file and the shared device helpers it includes."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_28831_amd", "csrc")
    for f in (KERNEL_SOURCE[kernel], "hk_internal.h"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()


def _traffic(kernel, workload):
    """HBM bytes per launch from the stored rocprofv3 counter summary of this kernel and
    workload (FETCH_SIZE and WRITE_SIZE, scaled by the plain-copy calibration), or None when
    there is none or the kernel's source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    src = os.path.join(ROOT, "paper_2606_28831_amd", "csrc", KERNEL_SOURCE.get(kernel, ""))
    if not os.path.isfile(path) or not os.path.isfile(src):
        return None, "no stored counter summary"
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != _source_sha(kernel):
        return None, "kernel source changed since the counters were taken"
    try:
        return float(kv["hbm_bytes_per_launch"]), os.path.relpath(path, ROOT)
    except (KeyError, ValueError):
        return None, "malformed counter summary"


def _mfma_counters(kernel, workload):
    """The stored MFMA counter summary of this kernel and workload (flop counted, clock,
    busy share), or None when there is none or the kernel's source has changed since."""
    path = os.path.join(ROOT, "profiles", f"mfma_{kernel}_{workload}.txt")
    if not os.path.isfile(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != _source_sha(kernel):
        return None
    try:
        return {"flop_counted": float(kv["mfma_flop_per_dispatch"]), "clock_ghz": float(kv["clock_ghz"]),
                "busy_frac_of_simd_cycles": float(kv["mfma_busy_frac_of_simd_cycles"]),
                "source": os.path.relpath(path, ROOT)}
    except (KeyError, ValueError):
        return None


def _roofline(ktime, per_launch, workload):
    """Roofline entry for the kernel with the largest share of the timed region."""
    timed = {k: v for k, v in ktime.items() if k in per_launch}
    if not timed:
        return None
    name = max(timed, key=lambda k: timed[k]["ms_per_step"])
    nbytes, flops = per_launch[name]
    dur_s = timed[name]["avg_ms"] / 1e3
    achieved = nbytes / dur_s / 1e9
    traffic, note = _traffic(name, workload)
    out = {"kernel": name, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
           "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
           "traffic_source": note, "bytes_per_launch": nbytes, "avg_launch_ms": timed[name]["avg_ms"],
           "launches_per_step": timed[name]["launches_per_step"]}
    if flops:
        out["mfma_tflops"] = flops / dur_s / 1e12
        out["mfma_frac_bf16"] = out["mfma_tflops"] / BF16_PEAK_TFLOPS
    return out


def run_compression(args):
    import paper_2606_28831_amd as hk
    import workload as WL
    from paper_2606_28831_amd.pipeline import Compressor

    c = args.config
    cfg = WL.config(c)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    w = WL.make_workload(cfg, dev)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    metric = "attn+red" if cfg.get("n_ref") else "attn"
    comp = Compressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv, alloc, cfg["p"],
                      L_dense=cfg["L_dense"], L_sparse=cfg["L_sparse"], metric=metric,
                      n_ref=cfg.get("n_ref", 0), keep_c=False)
    pristine = WL.clone_state(w)
    ref = w.ref_slots
    tokens = _cand_tokens(w, cfg["L_dense"])
    positions = w.NS * cfg["N"]

    def restore():
        WL.restore_state(w, pristine)

    # one cold step (first-call costs), then one untimed step with every kernel timed: finds
    # the kernel with the largest share of a step.  The warmup steps come after both, right
    # before the timed region: the timer reads leave the GPU idle for a moment, and a timed
    # region that began there would start below the clock the steps run at.
    restore()
    comp.step(w.q_obs, ref_slots=ref)
    torch.cuda.synchronize()
    for name in hk.TIMED_KERNELS:
        hk.hk_timing_read(name)
    hk.hk_timing_enable()
    restore()
    comp.step(w.q_obs, ref_slots=ref)
    torch.cuda.synchronize()
    hk.hk_timing_enable([])
    kwarm = {}
    for name in hk.TIMED_KERNELS:
        tot, n = hk.hk_timing_read(name)
        if n:
            kwarm[name] = tot
    dominant = max((k for k in kwarm if k in ROOFLINE_KERNELS), key=lambda k: kwarm[k])
    for _ in range(args.warmup):
        restore()
        comp.step(w.q_obs, ref_slots=ref)

    # ---------------- timed region: exactly K steps.  The library records HIP events around
    # each launch of the dominant kernel, on its launch stream, in every EVENT_EVERY-th
    # step (each event record costs the stream time of its own; sampled steps keep that
    # out of most of the region while the kernel is still timed inside it).
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sampled = 0
    for i in range(args.steps):
        on = i % EVENT_EVERY == 0
        hk.hk_timing_enable([dominant] if on else [])
        sampled += on
        restore()
        comp.step(w.q_obs, ref_slots=ref)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    hk.hk_timing_enable([])
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    status = int(comp.buf.status.item())
    tot, n = hk.hk_timing_read(dominant)
    ktime = {dominant: {"avg_ms": tot / n, "launches_per_step": n / sampled,
                        "ms_per_step": tot / sampled}}
    kernels_discovery = dict(kwarm)

    # the same K steps with kernel timing off (event records cost a little launch time)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        restore()
        comp.step(w.q_obs, ref_slots=ref)
    torch.cuda.synchronize()
    ms_per_step_plain = (time.perf_counter() - t2) * 1e3 / args.steps

    # ---------------- per-stage timing (HIP events on the launch stream), outside the timed loop
    reps = max(3, min(args.steps, 10))
    ev = _events(8 * reps)
    lse_given = comp.buf.row_lse.clone()
    for r in range(reps):
        restore()
        e = ev[8 * r:8 * r + 8]
        e[0].record()
        comp.score(w.q_obs, ref_slots=ref)
        e[1].record()
        comp.select()
        e[2].record()
        comp.compact()
        e[3].record()
        restore()
        e[4].record()
        comp.score(w.q_obs, ref_slots=ref, row_lse_in=lse_given)     # pass 2 alone: one kernel
        e[5].record()
    torch.cuda.synchronize()

    def avg(a, b):
        return sum(ev[8 * r + a].elapsed_time(ev[8 * r + b]) for r in range(reps)) / reps

    st = {"score": avg(0, 1), "select": avg(1, 2), "compact": avg(2, 3), "score_pass2": avg(4, 5)}
    st["score_pass1_merge"] = st["score"] - st["score_pass2"]
    step_ms_events = st["score"] + st["select"] + st["compact"]
    steps_ev = sorted(ev[8 * r].elapsed_time(ev[8 * r + 3]) for r in range(reps))

    def pct(q):
        return steps_ev[min(len(steps_ev) - 1, int(round(q * (len(steps_ev) - 1))))]
    step_pcts = {"p10": pct(0.1), "p50": pct(0.5), "p90": pct(0.9), "reps": reps}

    # ---------------- budget statistics of the last step
    restore()
    comp.step(w.q_obs, ref_slots=ref)
    torch.cuda.synchronize()
    k = comp.buf.k.float()
    cl = comp.buf.cand_len.float()
    nc_valid = tokens / max(1, w.n_heads)
    frac = (k / torch.clamp(cl, min=1)).cpu()
    kept_mean = float(k.mean())

    # ---------------- algorithmic bytes (K read once, scores written+read, selection bits,
    # condensed K and V read + written); per-kernel bytes and flops per launch
    D, e = cfg["D"], _esize(cfg)
    S = w.S_max
    G = cfg["Hq"] // cfg["Hkv"]
    R = G * cfg["W"]
    H = w.n_heads
    n_metric = 2 if metric == "attn+red" else 1
    restore()
    valid_tokens = _cand_tokens(w, 0)
    k_cond_total = _condensed_kept(w, comp.buf.sel_bits, cfg["L_dense"], cfg["L_sparse"])
    bytes_k = tokens * D * e
    bytes_scores = H * S * 4 * 2 * n_metric
    bytes_sel = H * S / 8 * 2
    bytes_rewrite = 4 * k_cond_total * D * e
    bytes_q = cfg["W"] * w.NS * cfg["Hq"] * D * e
    alg_bytes = bytes_k + bytes_scores + bytes_sel + bytes_rewrite + bytes_q
    step_s = ms_per_step / 1e3
    n_ref = cfg.get("n_ref", 0) if metric == "attn+red" else 0
    per_launch = {
        # every valid key against the window (row LSE), the window queries
        "score_pass1": (valid_tokens * D * e + bytes_q, 2.0 * R * valid_tokens * D),
        # candidate keys, window queries and reference keys; score rows written (one per metric)
        "score_pass2": (tokens * D * e + bytes_q + H * n_ref * D * e + H * S * 4 * n_metric,
                        2.0 * (R + n_ref) * tokens * D),
        # condensed rows: K and V, each read once and written once
        "compact_gather": (bytes_rewrite, 0.0),
    }
    roof_kernel = _roofline(ktime, per_launch, cfg["name"])
    roof_kernel["events_every_n_steps"] = EVENT_EVERY
    roof_kernel["share_of_step"] = ktime[dominant]["ms_per_step"] / ms_per_step

    out = {
        "metric": METRIC,
        "value": tokens / step_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": cfg["name"], "sequences": w.NS, "q_heads": cfg["Hq"],
                   "kv_heads": cfg["Hkv"], "head_dim": D, "cache_len": cfg["N"],
                   "window": cfg["W"], "top_p": cfg["p"], "page": 16,
                   "L_dense": cfg["L_dense"], "L_sparse": cfg["L_sparse"], "metric": metric},
        "hbm_frac_step": alg_bytes / step_s / 1e9 / HBM_PEAK_GBS,
        "alg_bytes_per_step": alg_bytes,
        "positions_per_s": positions / step_s,
        "stage_ms": st,
        "step_ms_events": step_ms_events,
        "step_ms_events_percentiles": step_pcts,
        # score GEMM throughput per pass (two passes unless the row LSEs are given)
        "score_mfma": {"pass1_tflops": per_launch["score_pass1"][1] / (st["score_pass1_merge"] * 1e-3) / 1e12,
                       "pass2_tflops": per_launch["score_pass2"][1] / (st["score_pass2"] * 1e-3) / 1e12,
                       "pass2_frac_bf16_peak": per_launch["score_pass2"][1] / (st["score_pass2"] * 1e-3)
                       / 1e12 / BF16_PEAK_TFLOPS, "flops_per_pass": per_launch["score_pass2"][1],
                       "counters": {k: _mfma_counters(k, cfg["name"]) for k in ("score_pass1", "score_pass2")}},
        "ms_per_step_no_kernel_events": ms_per_step_plain,
        "kernel_ms_discovery_step": kernels_discovery,
        "budget": {"mean_kept": kept_mean, "min_frac": float(frac.min()),
                   "mean_frac": float(frac.mean()), "max_frac": float(frac.max()),
                   "SU": float(frac.mean() / max(1e-9, float(frac.max())))},
        "status_flags": status,
        "gen_s": t_gen,
        "roofline": roof_kernel,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, cfg, comp, args)
    return out


# ---------------------------------------------------------------- CPU baseline (the oracle)
# A pool of worker processes, one per host core of this process's affinity mask, forked at
# start-up before anything touches the GPU; each worker runs the oracle on one head at a time
# with a single BLAS thread.
_POOL = None
_POOL_WORKERS = 0


def _pool_init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def start_cpu_pool():
    """Fork the oracle's worker pool (call before any GPU work)."""
    global _POOL, _POOL_WORKERS
    import multiprocessing as mp
    _POOL_WORKERS = max(1, len(os.sched_getaffinity(0)))
    _POOL = mp.get_context("fork").Pool(_POOL_WORKERS, initializer=_pool_init)


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return None


def _oracle_chain_head(task):
    """The whole step for one head with the oracle: score -> calibrate (-> redundancy,
    temperature, mixture) -> Top-p -> rewrite, including the rewrite's row copies."""
    import numpy as np

    import oracle as O
    kh, vh, q, mask_h, n_h, refs, cfg, scale = task
    t0 = time.perf_counter()
    D = kh.shape[-1]
    local = np.arange(n_h)
    rows, valid = O.read_head(kh, local, mask_h, n_h)
    nc, ns, nd = O.tier_pages(n_h, cfg["L_dense"], cfg["L_sparse"])
    cand_len = 16 * (n_h - nd)
    s, _ = O.score_head(q, rows, valid, cand_len, scale)
    cand = O.candidate_mask(valid, cand_len)
    c, _ = O.calibrate_head(s, cand)
    if refs is not None:
        xr = O.redundancy_head(rows, valid, cand_len, refs)
        r0 = O.topp_head(c.astype(np.float32), cand, cfg["p"])
        T = O.solve_T_head(xr, cand, r0.k, r0.sel_mass / 2.0 ** 40)
        c = O.mix([c, O.calibrate_head(xr, cand, T)[0]], [0.5, 0.5])
    r = O.topp_head(c.astype(np.float32), cand, cfg["p"])
    res = O.compact_head(local, mask_h, n_h, r.sel, cfg["L_dense"], cfg["L_sparse"])
    for ent in res.pages:
        if ent.kind == "new":
            src = [ph * 16 + t for ph, t in ent.src]
            _ = kh.reshape(-1, D)[src].copy(), vh.reshape(-1, D)[src].copy()
    return int(cand.sum()), time.perf_counter() - t0


def cpu_baseline(w, cfg, comp, args):
    """The oracle, as it stands, on a bounded sample of heads of the same workload, run by the
    worker pool (one head per task); value = candidate slots of the sample / pool wall time."""
    import numpy as np
    G = cfg["Hq"] // cfg["Hkv"]
    D = cfg["D"]
    scale = 1 / math.sqrt(D)
    pristine_table = w.page_table.cpu().numpy()
    masks = w.page_mask.cpu().numpy().astype(np.int64) & 0xFFFF
    n = w.n_pages.cpu().numpy()
    heads = list(range(0, w.n_heads, max(1, w.n_heads // args.cpu_heads)))
    small = {k: cfg[k] for k in ("L_dense", "L_sparse", "p")}
    tasks = []
    for h in heads:
        ids = torch.tensor(pristine_table[h, :n[h]], dtype=torch.long, device=w.k_pool.device)
        kh = w.k_pool.index_select(0, ids).float().cpu().numpy()
        vh = w.v_pool.index_select(0, ids).float().cpu().numpy()
        s_, kv = divmod(h, cfg["Hkv"])
        q = w.q_obs[:, s_, kv * G:(kv + 1) * G].float().cpu().numpy().reshape(-1, D)
        refs = w.ref_slots[h].cpu().numpy() if w.ref_slots is not None else None
        tasks.append((kh, vh, q, masks[h], int(n[h]), refs, small, scale))
    t0 = time.perf_counter()
    results = _POOL.map(_oracle_chain_head, tasks, chunksize=1)
    wall = time.perf_counter() - t0
    done_tokens = sum(r[0] for r in results)
    busy = sum(r[1] for r in results)
    return {"value": done_tokens / wall, "unit": "tokens/s", "cores": _POOL_WORKERS,
            "kind": "oracle",
            "sample": f"{len(heads)} of {w.n_heads} heads ({done_tokens} candidate slots), full "
                      f"chain score->calibrate->Top-p->rewrite, one head per task on "
                      f"{_POOL_WORKERS} worker processes (1 BLAS thread each), {wall:.1f} s wall, "
                      f"{busy:.1f} s of worker time",
            "host_cpus": len(os.sched_getaffinity(0)), "blas_threads_per_worker": 1,
            "serial_tokens_per_s": done_tokens / busy}


def run_budget(args):
    """The compression step under the hard budget (Step 4) with Cautious Update voting, on
    the workload of --config: budget state -> row LSEs -> per-row probabilities -> votes ->
    vote-ranked selection with sinks -> mode-driven rewrite."""
    import paper_2606_28831_amd as hk
    import workload as WL
    from paper_2606_28831_amd.pipeline import BudgetCompressor

    cfg = WL.config(args.config)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    w = WL.make_workload(cfg, dev)
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    comp = BudgetCompressor(w.NS, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["W"], kv, alloc, cfg["p"],
                            BUDGET["L_lower"], BUDGET["L_upper"], L_dense=cfg["L_dense"],
                            n_sink=BUDGET["n_sink"])
    pristine = WL.clone_state(w)
    tokens = _cand_tokens(w, cfg["L_dense"])
    workload = f"{cfg['name']}_budget{BUDGET['L_upper']}"

    def restore():
        WL.restore_state(w, pristine)

    # cold step, kernel discovery, then the warmup steps right before the timed region (as
    # in run_compression)
    restore()
    comp.step(w.q_obs)
    torch.cuda.synchronize()
    for name in hk.TIMED_KERNELS:
        hk.hk_timing_read(name)
    hk.hk_timing_enable()
    restore()
    comp.step(w.q_obs)
    torch.cuda.synchronize()
    hk.hk_timing_enable([])
    kwarm = {}
    for name in hk.TIMED_KERNELS:
        tot, n = hk.hk_timing_read(name)
        if n:
            kwarm[name] = tot
    dominant = max((k for k in kwarm if k in BUDGET_ROOFLINE_KERNELS), key=lambda k: kwarm[k])
    for _ in range(args.warmup):
        restore()
        comp.step(w.q_obs)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sampled = 0
    for i in range(args.steps):
        on = i % EVENT_EVERY == 0
        hk.hk_timing_enable([dominant] if on else [])
        sampled += on
        restore()
        comp.step(w.q_obs)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    hk.hk_timing_enable([])
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    tot, n = hk.hk_timing_read(dominant)
    ktime = {dominant: {"avg_ms": tot / n, "launches_per_step": n / sampled,
                        "ms_per_step": tot / sampled}}
    b = comp.buf
    status = int(b["status"].item())
    k = b["k"].float()
    modes = torch.bincount(b["head_mode"].long(), minlength=3).tolist()
    votes = (b["votes"].to(torch.int32) & 0xFFFF).float()
    voted = float((votes >= 1).sum()) / w.n_heads

    D, e = cfg["D"], _esize(cfg)
    S, H = w.S_max, w.n_heads
    R = cfg["Hq"] // cfg["Hkv"] * cfg["W"]
    bytes_q = cfg["W"] * w.NS * cfg["Hq"] * D * e
    valid_tokens = _cand_tokens(w, 0)
    restore()
    comp.select(w.q_obs)
    torch.cuda.synchronize()
    k_cond = _condensed_kept(w, b["sel_bits"], cfg["L_dense"], 0)
    a_bytes = H * R * S * 4
    per_launch = {
        "score_pass1": (valid_tokens * D * e + bytes_q, 2.0 * R * valid_tokens * D),
        # candidate keys and the window read, every row's probabilities written
        "score_rows": (tokens * D * e + bytes_q + a_bytes, 2.0 * R * tokens * D),
        # every row's probabilities read, every row's selection bitmap written
        "vote": (a_bytes + H * R * S / 8, 0.0),
        "compact_gather": (4 * k_cond * D * e, 0.0),
    }
    roof = _roofline(ktime, per_launch, workload)
    roof["events_every_n_steps"] = EVENT_EVERY
    roof["share_of_step"] = ktime[dominant]["ms_per_step"] / ms_per_step
    out = {
        "metric": "compressed KV tokens/s under the hard budget (Cautious Update votes)",
        "value": tokens / (ms_per_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": workload, "base": cfg["name"], "sequences": w.NS,
                   "q_heads": cfg["Hq"], "kv_heads": cfg["Hkv"], "head_dim": D,
                   "cache_len": cfg["N"], "window": cfg["W"], "rows": R, "top_p": cfg["p"],
                   "L_dense": cfg["L_dense"], **BUDGET},
        "kernel_ms_discovery_step": kwarm,
        "budget": {"head_modes_keep_sparse_rewrite": modes, "mean_kept": float(k.mean()),
                   "mean_voted": voted, "mean_votes_of_voted": float(votes.sum()) / max(1.0, voted * H)},
        "row_probabilities_bytes": a_bytes,
        "status_flags": status,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_budget(w, cfg, args)
    return out


def cpu_baseline_budget(w, cfg, args):
    """The oracle's hard-budget chain, as it stands, on a bounded sample: the window rows of
    one head, as many as fit the time budget (every row's vote is one Top-p over the head)."""
    import numpy as np

    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    G, D = cfg["Hq"] // cfg["Hkv"], cfg["D"]
    R = G * cfg["W"]
    scale = 1 / math.sqrt(D)
    h = 0
    n = int(w.n_pages[h].item())
    ids = w.page_table[h, :n].long()
    kh = w.k_pool.index_select(0, ids).float().cpu().numpy()
    masks = w.page_mask[h].cpu().numpy().astype(np.int64) & 0xFFFF
    q = w.q_obs[:, 0, 0:G].float().cpu().numpy().reshape(-1, D)
    t0 = time.perf_counter()
    rows, valid = O.read_head(kh, np.arange(n), masks, n)
    nd = O.tier_pages(n, cfg["L_dense"], 0)[2]
    cand_len = 16 * (n - nd)
    cand = O.candidate_mask(valid, cand_len)
    _, lse = O.score_head(q, rows, valid, cand_len, scale)
    mode, cap = O.budget_plan_head(n, masks, cfg["L_dense"], BUDGET["L_lower"], BUDGET["L_upper"])
    done = 0
    votes = np.zeros(len(valid), dtype=np.int64)
    for r in range(R):
        a = O.score_rows_head(q[r:r + 1], rows, valid, cand_len, scale, lse[r:r + 1])
        votes += O.topp_head(a[0].astype(np.float32), cand, cfg["p"]).sel
        done += 1
        if time.perf_counter() - t0 >= args.cpu_seconds:
            break
    if done == R:
        O.budget_select_head(cand, votes=votes, mode=mode, k_cap=cap, n_sink=BUDGET["n_sink"])
    spent = time.perf_counter() - t0
    # candidate slots of one head, scaled by the share of its rows done
    slots = float(cand.sum()) * done / R
    return {"value": slots / spent, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"head 0: {done} of its {R} window rows (per-row probabilities and Top-p "
                      f"vote over {int(cand.sum())} candidates), {spent:.1f} s in one process "
                      f"(cores = its BLAS threads); value = candidate slots x rows done / rows "
                      f"per head / seconds",
            "host_cpus": len(os.sched_getaffinity(0))}


def run_decode(args):
    """Config 5: end-to-end decode loop.  One timed "step" = one segment of
    `compress_every` decode steps (append + per-layer paged decode attention) followed by
    one compression of every layer; the segment's random q/k/v are drawn into HBM before
    its timed region starts."""
    import paper_2606_28831_amd as hk
    import workload as WL
    from paper_2606_28831_amd.pipeline import DecodeLoop

    cfg = WL.config(5)
    L, B, Hq, Hkv, D, W = (cfg[k] for k in ("L", "B", "Hq", "Hkv", "D", "W"))
    T = cfg["compress_every"]
    n_seg = args.decode_segments if args.decode_segments else cfg["decode_steps"] // T
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    max_pages = (cfg["N"] + cfg["decode_steps"]) // 16
    H = L * B * Hkv
    t_gen = time.perf_counter()
    w = WL.make_workload(cfg, dev, max_pages=max_pages, pool_pages=H * max_pages + H * 256)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
    alloc = hk.Allocator(w.free_ids, w.free_top)
    loop = DecodeLoop(L, B, Hq, Hkv, D, W, kv, alloc, cfg["p"], cfg["L_dense"], keep_c=False)
    NS = L * B
    dt = WL.TORCH_DTYPE[cfg["dtype"]]
    seg_ms, seg_tokens_kv, kept = [], [], []
    graph = None
    if args.graph:
        # one HIP graph for a whole segment over persistent input buffers, refilled in
        # place before each replay (the graph keeps their addresses)
        bufs = (torch.empty(T, NS, Hq, D, device=dev, dtype=dt), torch.empty(T, NS, Hkv, D, device=dev, dtype=dt),
                torch.empty(T, NS, Hkv, D, device=dev, dtype=dt), torch.empty(T, NS, Hq, device=dev))
        t_cap = time.perf_counter()
        graph = loop.capture_segment(*bufs)
        torch.cuda.synchronize()
        t_cap = time.perf_counter() - t_cap
    for name in hk.TIMED_KERNELS:
        hk.hk_timing_read(name)
    hk.hk_timing_enable(["decode_split"])    # the dominant kernel of the loop
    for seg in range(n_seg):
        g = torch.Generator(device=dev).manual_seed(cfg["seed"] * 7919 + seg + 1)
        q_seg = torch.randn(T, NS, Hq, D, generator=g, device=dev).to(dt)
        k_seg = torch.randn(T, NS, Hkv, D, generator=g, device=dev).to(dt)
        v_seg = torch.randn(T, NS, Hkv, D, generator=g, device=dev).to(dt)
        lse_seg = torch.empty(T, NS, Hq, device=dev)
        m = w.page_mask.to(torch.int32) & 0xFFFF
        valid = int(sum(bin(i).count("1") * c for i, c in zip(*torch.unique(m, return_counts=True))))
        seg_tokens_kv.append(valid)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if graph is not None:
            for dst, src in zip(bufs, (q_seg, k_seg, v_seg)):
                dst.copy_(src)
            torch.cuda.synchronize()
            e0.record()
            graph.replay()
            e1.record()
        else:
            e0.record()
            loop.segment(q_seg, k_seg, v_seg, lse_seg)
            e1.record()
        torch.cuda.synchronize()
        seg_ms.append(e0.elapsed_time(e1))
        kept.append(float(loop.comp.buf.k.float().mean()))
        del q_seg, k_seg, v_seg, lse_seg
    hk.hk_timing_enable([])
    tot, n = hk.hk_timing_read("decode_split")
    # graph replays launch nothing from the host, so no per-kernel events are recorded
    ktime = {"decode_split": {"avg_ms": tot / n, "launches_per_step": n / n_seg,
                              "ms_per_step": tot / n_seg}} if n else {}
    status = int(loop.status.item()) | int(loop.comp.buf.status.item())
    total_s = sum(seg_ms) / 1e3
    tokens = B * T * n_seg
    e = 2 if cfg["dtype"] == "bf16" else 4
    # decode attention bytes: every valid K and V row read once per step per layer (the
    # append adds one row per head per step), the step's queries read, outputs written
    dec_bytes = sum(2 * D * e * (T * v + H * T * (T + 1) // 2) for v in seg_tokens_kv)
    dec_bytes += n_seg * T * NS * Hq * (D * e + D * 4 + 4)
    per_launch = {"decode_split": (dec_bytes / max(1, n_seg * T * L), 0.0)}
    roof = _roofline(ktime, per_launch, cfg["name"])
    if roof is not None:
        roof["share_of_step"] = ktime["decode_split"]["ms_per_step"] / (sum(seg_ms) / n_seg)
    return {
        "metric": METRIC, "value": tokens / total_s, "unit": "decode tokens/s",
        "n_gpus": 1, "steps": n_seg, "warmup": 0, "ms_per_step": sum(seg_ms) / n_seg,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": cfg["name"], "layers": L, "batch": B, "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": D, "prompt": cfg["N"], "decode_steps": T * n_seg,
                   "compress_every": T, "window": W, "top_p": cfg["p"], "L_dense": cfg["L_dense"],
                   "hip_graph": bool(args.graph)},
        "graph_capture_s": t_cap if args.graph else None,
        "decode_attn_hbm_frac_lower_bound": dec_bytes / total_s / 1e9 / HBM_PEAK_GBS,
        "kernels": ktime, "roofline": roof,
        "segment_ms": seg_ms, "valid_kv_slots_per_segment": seg_tokens_kv, "mean_kept_per_head": kept,
        "status_flags": status, "gen_s": t_gen,
    }


def decode_summary(d):
    """The config-5 decode figures carried by the default bench line: decode tokens/s over the
    stated segments and the dominant decode kernel against the HBM roofline."""
    r = d.get("roofline") or {}
    return {"workload": d["config"]["workload"], "segments": d["steps"],
            "decode_steps": d["config"]["decode_steps"], "value": d["value"],
            "unit": "decode tokens/s", "ms_per_segment": d["ms_per_step"],
            "decode_attn_hbm_frac_lower_bound": d["decode_attn_hbm_frac_lower_bound"],
            "roofline": {"kernel": r.get("kernel"), "bound": "hbm", "achieved": r.get("achieved"),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": r.get("frac"),
                         "traffic": r.get("traffic"), "traffic_source": r.get("traffic_source"),
                         "bytes_per_launch": r.get("bytes_per_launch"),
                         "avg_launch_ms": r.get("avg_launch_ms"),
                         "launches_per_segment": r.get("launches_per_step"),
                         "share_of_segment": r.get("share_of_step")},
            "status_flags": d["status_flags"]}


def run_crossover(args):
    """Sparse loading vs rewrite (Sec. 3.3.1 HA-Sparse vs HA-Max), re-created synthetically:
    per cache length and batch, the preparation time of each form (hk_compact with every
    page in the sparse band, i.e. masks only, or every page condensed, i.e. rewritten),
    the decode-attention time per step over the result, the memory each holds, and the
    decode step after which the rewrite has paid back its preparation (time) and its
    transient memory (memory-time integral).  Selections are drawn per head, scattered
    uniformly over the valid slots, with keep fractions uniform in [0, 25%] (mean 12.5%,
    the paper's setting); the kernels are the tested ones, only the tier split differs."""
    import paper_2606_28831_amd as hk
    import workload as WL
    dev = torch.device("cuda", 0)
    Hq, Hkv, D = 32, 8, 128
    G = Hq // Hkv
    page_bytes = 16 * D * 2 * 2                         # K and V of one 16-slot page, bf16
    rows = []
    for B in (1, 32):
        for N in (2048, 4096, 8192, 12288, 16384, 20480):
            cfg = dict(L=1, B=B, Hq=Hq, Hkv=Hkv, D=D, N=N, dtype="bf16", W=8, seed=7 + N + B,
                       recipe="normal")
            w = WL.make_workload(cfg, dev, pool_slack=1.3)
            H, S = w.n_heads, w.S_max
            g = torch.Generator(device=dev).manual_seed(N * 131 + B)
            frac = torch.rand(H, generator=g, device=dev) * 0.25
            r = torch.rand(H, S, generator=g, device=dev)
            sel = (r < frac[:, None]) & (torch.arange(S, device=dev)[None, :] < N)
            bits = (sel.view(H, S // 32, 32).to(torch.int64) << torch.arange(32, device=dev)).sum(-1)
            sel_bits = bits.to(torch.int64).bitwise_and(0xFFFFFFFF).to(torch.int32)
            kv = hk.PagedKV(w.k_pool, w.v_pool, w.page_table, w.page_mask, w.n_pages)
            alloc = hk.Allocator(w.free_ids, w.free_top)
            d = hk.dims(B, Hq, Hkv, D, 0)
            st = torch.zeros(1, dtype=torch.int32, device=dev)
            wsc = hk.workspace(hk.OP_COMPACT, d, w.max_pages, dev)
            wsd = hk.workspace(hk.OP_DECODE, d, w.max_pages, dev)
            q = torch.randn(B, Hq, D, generator=g, device=dev).to(torch.bfloat16)
            o = torch.empty(B, Hq, D, device=dev)
            lse = torch.empty(B, Hq, device=dev)
            pristine = WL.clone_state(w)
            pages_before = int(w.n_pages.sum())
            out = {"batch": B, "tokens": N, "kept_mean": float(frac.mean()), "pages_before": pages_before}
            for mode, L_sparse in (("sparse", N + 16), ("rewrite", 0)):
                prep = []
                for _ in range(5):
                    WL.restore_state(w, pristine)
                    torch.cuda.synchronize()
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    hk.hk_compact(d, kv, sel_bits, 0, L_sparse, alloc, st, wsc)
                    e1.record()
                    torch.cuda.synchronize()
                    prep.append(e0.elapsed_time(e1))
                for _ in range(3):
                    hk.hk_decode_attn(d, q, kv, 1 / math.sqrt(D), o, lse, wsd)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(20):
                    hk.hk_decode_attn(d, q, kv, 1 / math.sqrt(D), o, lse, wsd)
                e1.record()
                torch.cuda.synchronize()
                pages_after = int(w.n_pages.sum())
                out[mode] = {"prep_ms": sorted(prep)[len(prep) // 2], "decode_ms": e0.elapsed_time(e1) / 20,
                             "pages_held": pages_after, "bytes_held": pages_after * page_bytes,
                             "new_pages": pages_after if mode == "rewrite" else 0}
            assert int(st.item()) == 0
            sp, rw = out["sparse"], out["rewrite"]
            dd = sp["decode_ms"] - rw["decode_ms"]
            out["time_breakeven_steps"] = ((rw["prep_ms"] - sp["prep_ms"]) / dd) if dd > 0 else None
            # memory-time integral (bytes x ms) from the compression on, as a function of the
            # decode steps t that follow: A + B t.  The rewrite holds old and new pages while it
            # runs, then only the new ones; sparse loading holds the old pages throughout.  The
            # pay-back is the (fractional) t where the two lines cross.
            a_sp, b_sp = sp["bytes_held"] * sp["prep_ms"], sp["bytes_held"] * sp["decode_ms"]
            a_rw = (pages_before + rw["new_pages"]) * page_bytes * rw["prep_ms"]
            b_rw = rw["bytes_held"] * rw["decode_ms"]
            if a_rw <= a_sp:
                out["mti_breakeven_steps"] = 0.0
            elif b_sp > b_rw:
                out["mti_breakeven_steps"] = (a_rw - a_sp) / (b_sp - b_rw)
            else:
                out["mti_breakeven_steps"] = None
            out["decode_speedup"] = sp["decode_ms"] / rw["decode_ms"]
            rows.append(out)
            print(json.dumps({k: out[k] for k in ("batch", "tokens", "decode_speedup", "time_breakeven_steps",
                                                  "mti_breakeven_steps")}), file=sys.stderr, flush=True)
            del w, kv, alloc, wsc, wsd
            torch.cuda.empty_cache()
    return {"experiment": "sparse loading vs rewrite (HA-Sparse vs HA-Max)", "data": "synthetic",
            "heads_per_sequence": Hkv, "q_heads": Hq, "head_dim": D, "dtype": "bf16", "rows": rows}


def copy_calibration():
    """A plain 1 GiB device-to-device copy, three times: the reference the FETCH_SIZE and
    WRITE_SIZE counters are scaled by (each copy reads and writes exactly 1 GiB)."""
    a = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    return {"copy_calibration_bytes": a.numel() * 4, "copies": 3}


def run_peaks():
    """Measured rates behind the score passes' rooflines: the hardware exponential
    (v_exp_f32) and the bf16 MFMA (32x32x16), each from a throughput kernel of the library
    (hk_probe) timed with events on the launch stream, best of five launches; and the time
    of the passes' MFMA + VALU mix alone, interleaved in one wave, and split over waves."""
    import paper_2606_28831_amd as hk
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 4 * n_cu                            # 16 waves per CU: every SIMD busy
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

    def best_ms(kind, iters):
        hk.hk_probe(kind, blocks, iters, out)     # warm
        best = float("inf")
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            hk.hk_probe(kind, blocks, iters, out)
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        if not torch.isfinite(out).all():
            raise SystemExit("rate probe produced a non-finite value")
        return best

    it_exp, it_mfma, it_mix = 4096, 2048, 1024
    ms_exp = best_ms(hk.PROBE_EXP, it_exp)
    ms_mfma = best_ms(hk.PROBE_MFMA, it_mfma)
    n_exp = 8 * it_exp * 256 * blocks
    n_mfma = 16 * it_mfma * blocks
    # MFMA and VALU work of the score passes' mix, alone, interleaved in one wave, and in
    # different waves of one SIMD (equal total work in the last two)
    mix = {name: best_ms(kind, it_mix) for name, kind in
           (("mfma_only_ms", hk.PROBE_MFMA4), ("valu_only_ms", hk.PROBE_VALU),
            ("same_wave_ms", hk.PROBE_MIX), ("split_waves_ms", hk.PROBE_SPLIT))}
    return {"probe": "rates", "compute_units": n_cu, "workgroups": blocks,
            "exp_per_s": n_exp / (ms_exp / 1e3), "exp_ms": ms_exp,
            "mfma_bf16_tflops": n_mfma * 32768 / (ms_mfma / 1e3) / 1e12, "mfma_ms": ms_mfma,
            "mfma_bf16_peak_tflops": 2500.0, "mix_steps_per_wave": 4 * it_mix, **mix}


def _pmc_mean(run_dir, counter, match):
    """Mean per-dispatch value (KiB) of one counter over the dispatches of kernels whose
    name contains `match`, from a rocprofv3 --pmc output directory."""
    import csv
    import glob
    vals = []
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        for row in csv.DictReader(open(f)):
            if row["Counter_Name"] == counter and match in row["Kernel_Name"]:
                vals.append(float(row["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} dispatches of '{match}' under {run_dir}")
    return sum(vals) / len(vals), len(vals)


KERNEL_SYMBOL = {"score_pass1": "score_pass1_coop_kernel", "score_pass2": "score_pass2_coop_kernel",
                 "compact_gather": "compact_gather_kernel", "decode_split": "decode_split_kernel",
                 "score_rows": "score_rows_kernel", "vote": "vote_topp_kernel"}


def summarize_pmc(a):
    """Write profiles/traffic_<kernel>_<workload>.txt from four rocprofv3 --pmc runs: the
    benchmark with FETCH_SIZE, with WRITE_SIZE, and the copy calibration with each."""
    fetch_dir, write_dir, cal_fetch_dir, cal_write_dir = a.summarize_pmc
    sym = KERNEL_SYMBOL[a.kernel]
    cal_bytes = float(1 << 30)
    cf, _ = _pmc_mean(cal_fetch_dir, "FETCH_SIZE", "copyBuffer")
    cw, _ = _pmc_mean(cal_write_dir, "WRITE_SIZE", "copyBuffer")
    f_scale, w_scale = cal_bytes / (cf * 1024), cal_bytes / (cw * 1024)
    kf, nf = _pmc_mean(fetch_dir, "FETCH_SIZE", sym)
    kw, nw = _pmc_mean(write_dir, "WRITE_SIZE", sym)
    hbm = kf * 1024 * f_scale + kw * 1024 * w_scale
    sha = _source_sha(a.kernel)
    path = os.path.join(ROOT, "profiles", f"traffic_{a.kernel}_{a.workload}.txt")
    with open(path, "w") as f:
        f.write(f"# HBM traffic of {sym} on workload {a.workload}, per dispatch\n")
        f.write(f"# made by: {a.command}\n")
        f.write("# FETCH_SIZE and WRITE_SIZE are KiB per dispatch; each is scaled by what the same\n")
        f.write("# counter reads for a plain 1 GiB device copy (__amd_rocclr_copyBuffer).\n")
        f.write(f"kernel: {sym}\n")
        f.write(f"workload: {a.workload}\n")
        f.write(f"dispatches_fetch: {nf}\n")
        f.write(f"dispatches_write: {nw}\n")
        f.write(f"fetch_size_kib_per_dispatch: {kf:.1f}\n")
        f.write(f"write_size_kib_per_dispatch: {kw:.1f}\n")
        f.write(f"copy_fetch_kib_per_GiB: {cf:.1f}\n")
        f.write(f"copy_write_kib_per_GiB: {cw:.1f}\n")
        f.write(f"fetch_scale: {f_scale:.4f}\n")
        f.write(f"write_scale: {w_scale:.4f}\n")
        f.write(f"hbm_read_bytes_per_launch: {kf * 1024 * f_scale:.0f}\n")
        f.write(f"hbm_write_bytes_per_launch: {kw * 1024 * w_scale:.0f}\n")
        f.write(f"hbm_bytes_per_launch: {hbm:.0f}\n")
        f.write(f"source: paper_2606_28831_amd/csrc/{KERNEL_SOURCE[a.kernel]} + hk_internal.h\n")
        f.write(f"source_sha256: {sha}\n")
    return {"traffic_summary": path, "hbm_bytes_per_launch": hbm}


# the score passes' MFMA: v_mfma_f32_32x32x16_bf16, 32 cycles of one SIMD each
MFMA_CYCLES_PER_OP = 32
MFMA_FLOP_PER_OP = 32 * 32 * 16 * 2
N_SIMD = 256 * 4
N_XCD = 8


def _pmc_dispatches(run_dir, match):
    """Per-dispatch counter values {counter: value, "ns": duration} of the kernels whose name
    contains `match`, from a rocprofv3 --pmc output directory."""
    import csv
    import glob
    per = {}
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        for row in csv.DictReader(open(f)):
            if match not in row["Kernel_Name"]:
                continue
            d = per.setdefault((f, row["Dispatch_Id"]), {})
            d[row["Counter_Name"]] = float(row["Counter_Value"])
            if row.get("Start_Timestamp") and row.get("End_Timestamp"):
                d["ns"] = float(row["End_Timestamp"]) - float(row["Start_Timestamp"])
    if not per:
        raise SystemExit(f"no dispatches of '{match}' under {run_dir}")
    return list(per.values())


def summarize_mfma(a):
    """Write profiles/mfma_<kernel>_<workload>.txt from one rocprofv3 --pmc run with
    SQ_VALU_MFMA_BUSY_CYCLES (summed over every SIMD: 32 per 32x32x16 MFMA) and
    GRBM_GUI_ACTIVE (GPU cycles, summed over the 8 XCDs): the MFMA work the counters saw,
    the clock the kernel ran at, and the MFMA pipes' busy share of the SIMD cycles."""
    sym = KERNEL_SYMBOL[a.kernel]
    rows = _pmc_dispatches(a.summarize_mfma, sym)
    def mean(k):
        v = [r[k] for r in rows if k in r]
        if not v:
            raise SystemExit(f"no {k} for '{sym}' under {a.summarize_mfma}")
        return sum(v) / len(v), len(v)
    busy, n = mean("SQ_VALU_MFMA_BUSY_CYCLES")
    grbm, _ = mean("GRBM_GUI_ACTIVE")
    ns, _ = mean("ns")
    ops = busy / MFMA_CYCLES_PER_OP
    flop = ops * MFMA_FLOP_PER_OP
    gpu_cycles = grbm / N_XCD
    out = {"kernel": sym, "workload": a.workload, "dispatches": n,
           "mfma_busy_cycles_per_dispatch": busy, "mfma_ops_per_dispatch": ops,
           "mfma_flop_per_dispatch": flop, "duration_us": ns / 1e3,
           "gpu_cycles_per_dispatch": gpu_cycles, "clock_ghz": gpu_cycles / ns,
           "mfma_busy_frac_of_simd_cycles": busy / (gpu_cycles * N_SIMD),
           "mfma_tflops": flop / ns / 1e3, "mfma_frac_bf16_peak": flop / ns / 1e3 / BF16_PEAK_TFLOPS}
    path = os.path.join(ROOT, "profiles", f"mfma_{a.kernel}_{a.workload}.txt")
    with open(path, "w") as f:
        f.write(f"# MFMA work and utilisation of {sym} on workload {a.workload}, per dispatch\n")
        f.write(f"# made by: {a.command}\n")
        f.write("# SQ_VALU_MFMA_BUSY_CYCLES is summed over every SIMD (32 per 32x32x16 bf16 MFMA);\n")
        f.write("# GRBM_GUI_ACTIVE over the 8 XCDs; durations are the dispatches' own timestamps.\n")
        for k, v in out.items():
            f.write(f"{k}: {v:.6g}\n" if isinstance(v, float) else f"{k}: {v}\n")
        f.write(f"source: paper_2606_28831_amd/csrc/{KERNEL_SOURCE[a.kernel]} + hk_internal.h\n")
        f.write(f"source_sha256: {_source_sha(a.kernel)}\n")
    out["mfma_summary"] = path
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=40,
                    help="untimed steps right before the timed region (the clock takes about "
                         "50 ms of back-to-back steps to settle)")
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--crossover", action="store_true",
                    help="sparse loading vs rewrite over cache length (not the bench line)")
    ap.add_argument("--budget", action="store_true",
                    help="the step under the hard budget with Cautious Update votes "
                         "(Step 4; not the bench line)")
    ap.add_argument("--graph", action="store_true",
                    help="config 5: replay each decode segment from one captured HIP graph")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="time budget of the serial hard-budget oracle baseline")
    ap.add_argument("--cpu-heads", type=int, default=128,
                    help="heads of the workload the oracle baseline runs (evenly spaced)")
    ap.add_argument("--decode-segments", type=int, default=None,
                    help="config-5 segments of 128 decode steps (default: all 32)")
    ap.add_argument("--no-decode", action="store_true",
                    help="leave the config-5 decode run out of the default bench line")
    ap.add_argument("--peaks", action="store_true",
                    help="only measure the exponential and bf16 MFMA rates (hk_probe)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the 1 GiB plain copy the byte counters are scaled by")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR",
                                                          "CAL_WRITE_DIR"),
                    help="write a profiles/traffic_*.txt summary from rocprofv3 --pmc outputs")
    ap.add_argument("--summarize-mfma", metavar="RUN_DIR", default=None,
                    help="write a profiles/mfma_*.txt summary from a rocprofv3 --pmc run with "
                         "SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE")
    ap.add_argument("--kernel", default="compact_gather", choices=sorted(KERNEL_SYMBOL))
    ap.add_argument("--workload", default=None)
    ap.add_argument("--command", default="", help="the profiling command, recorded in the summary")
    args = ap.parse_args()
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(args)), flush=True)
        return
    if args.summarize_mfma:
        print(json.dumps(summarize_mfma(args)), flush=True)
        return
    args.steps_given = args.steps is not None
    if args.steps is None:
        args.steps = 20
    if args.config == 5 and args.steps_given and args.decode_segments is None:
        args.decode_segments = args.steps
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the compression step is independent per (sequence, KV "
              "head) and is benchmarked on a single MI355X; --gpus above 1 is not supported.",
              file=sys.stderr)
        sys.exit(2)
    plain = not (args.copy_calibration or args.peaks or args.crossover or args.budget)
    if plain and args.config != 5 and not args.no_cpu_baseline:
        start_cpu_pool()          # forked now, before anything touches the GPU
    try:
        _main(args)
    finally:
        if _POOL is not None:
            _POOL.terminate()
            _POOL.join()


def _main(args):
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        print(json.dumps(copy_calibration()), flush=True)
        return
    if args.peaks:
        print(json.dumps(run_peaks()), flush=True)
        return
    if args.crossover:
        print(json.dumps(run_crossover(args)), flush=True)
        return
    if args.budget:
        if args.config == 5:
            print("--budget runs on the compression workloads (configs 1-4)", file=sys.stderr)
            sys.exit(2)
        if not args.steps_given:
            args.steps = 10
        print(json.dumps(run_budget(args)), flush=True)
        return
    if args.config == 5:
        print(json.dumps(run_decode(args)), flush=True)
        return
    out = run_compression(args)
    if args.config == 3 and not args.no_decode:
        # the metric's second half, decode tokens/s, on config 5 (its own workload)
        torch.cuda.empty_cache()
        out["decode"] = decode_summary(run_decode(args))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

"""Seeded synthetic workloads for the Hard-KV compression step.

This module only draws inputs (window queries, paged K/V caches, page tables,
reference-slot samples, free lists).  It holds none of the method's arithmetic:
both the HIP path and the CPU oracle consume what it produces.

Tensors are torch tensors on the requested device; generation is seeded with
torch's counter-based generator on that device, so a GPU run and the host copy
handed to the oracle hold the same bits.

Layouts (shared by every entry point):
  q_obs      [W, NS, Hq, D]     window queries, window-major (NS = sequences = L*B)
  k_pool     [num_pages, 16, D] physical pages (v_pool likewise)
  page_table [NS*Hkv, max_pages] int32, -1 past n_pages
  page_mask  [NS*Hkv, max_pages] int16 bit t = slot t valid
  n_pages    [NS*Hkv] int32
  free_ids   [num_pages] int32 stack of free page ids, free_top [1] int32
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

PAGE = 16

# The five benchmark workloads (sizes from the method's deployment regime: long
# reasoning decodes of 8k-32k tokens, GQA groups of 4-7, 16-token pages).  W = 32 where the
# window is not fixed otherwise.
CONFIGS = {
    1: dict(name="cfg1_l1_b1_h8x2_d64_n2048_f32", L=1, B=1, Hq=8, Hkv=2, D=64, N=2048,
            dtype="f32", W=16, p=0.9, L_dense=0, L_sparse=0, seed=0, recipe="normal"),
    2: dict(name="cfg2_l1_b8_h32x8_d128_n16384_bf16_planted", L=1, B=8, Hq=32, Hkv=8, D=128,
            N=16384, dtype="bf16", W=32, p=0.95, L_dense=0, L_sparse=0, seed=1, recipe="planted"),
    3: dict(name="cfg3_l1_b32_h28x4_d128_n32768_bf16_tempered", L=1, B=32, Hq=28, Hkv=4, D=128,
            N=32768, dtype="bf16", W=32, p=0.9, L_dense=0, L_sparse=0, seed=2, recipe="tempered"),
    4: dict(name="cfg4_l32_b16_h32x8_d128_n16384_bf16_mixed_tiers", L=32, B=16, Hq=32, Hkv=8,
            D=128, N=16384, dtype="bf16", W=32, p=0.9, L_dense=512, L_sparse=2048, seed=3,
            recipe="normal", n_ref=256),
    5: dict(name="cfg5_l32_b64_h32x8_d128_prompt8192_decode4096_bf16", L=32, B=64, Hq=32, Hkv=8,
            D=128, N=8192, decode_steps=4096, compress_every=128, dtype="bf16", W=32, p=0.9,
            L_dense=512, L_sparse=0, seed=4, recipe="normal"),
}

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass
class Workload:
    cfg: dict
    q_obs: torch.Tensor
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    page_table: torch.Tensor
    page_mask: torch.Tensor
    n_pages: torch.Tensor
    free_ids: torch.Tensor
    free_top: torch.Tensor
    max_pages: int
    tau: torch.Tensor | None = None
    ref_slots: torch.Tensor | None = None
    extra: dict = field(default_factory=dict)
    meta: torch.Tensor | None = None   # one buffer behind the five mutable metadata tensors

    @property
    def NS(self):
        return self.cfg["L"] * self.cfg["B"]

    @property
    def n_heads(self):
        return self.NS * self.cfg["Hkv"]

    @property
    def S_max(self):
        return self.max_pages * PAGE


def config(c: int, **overrides) -> dict:
    d = dict(CONFIGS[c])
    d.update(overrides)
    return d


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def make_workload(cfg: dict, device="cpu", pool_slack: float = 2.0, max_pages: int | None = None,
                  hole_prob: float = 0.0, tail_len: int | None = None,
                  pool_pages: int | None = None, head_lens=None) -> Workload:
    """Draw one workload.

    cfg keys: L, B, Hq, Hkv, D, N, dtype, W, seed, recipe ("normal" | "planted" | "tempered"),
    optional n_ref.  N need not be a multiple of 16 (the last page is partial).
    hole_prob > 0 clears random slot bits (masked slots inside pages); tail_len
    overrides the last page's filled length.  The pool holds pool_slack times
    the pages in use (room for the out-of-place rewrite) unless pool_pages is given.
    head_lens (one length <= N per head) shortens heads after the draw: head h keeps its
    first ceil(len/16) pages, the last one filled to its length, and the rest of its pages
    go back to the free list (a length mix over heads; every draw stays as without it).
    """
    dev = torch.device(device)
    g = _gen(dev, cfg["seed"])
    L, B, Hq, Hkv, D, N, W = (cfg[k] for k in ("L", "B", "Hq", "Hkv", "D", "N", "W"))
    NS, H = L * B, L * B * Hkv
    G = Hq // Hkv
    dt = TORCH_DTYPE[cfg["dtype"]]
    n_used = -(-N // PAGE)
    mp = max(n_used, max_pages or 0)
    mp += mp % 2                    # even table width: S_max is a multiple of 32
    used = H * n_used
    num_pages = int(pool_pages) if pool_pages else max(int(math.ceil(used * pool_slack)), used + 1)

    # window queries, fp32 draw, optional per-(sequence, KV head) temperature
    q = torch.randn(W, NS, Hq, D, generator=g, device=dev, dtype=torch.float32)
    tau = None
    if cfg.get("recipe") == "tempered":
        u = torch.rand(NS, Hkv, generator=g, device=dev, dtype=torch.float64) * 2.0 - 1.0
        tau = torch.pow(10.0, u).to(torch.float32)          # log-uniform in [0.1, 10]
        q = q / tau.repeat_interleave(G, dim=1)[None, :, :, None]
    q_obs = q.to(dt).contiguous()

    # page assignment: a seeded permutation of the pool, head-major
    perm = torch.randperm(num_pages, generator=g, device=dev).to(torch.int32)
    table = torch.full((H, mp), -1, dtype=torch.int32, device=dev)
    table[:, :n_used] = perm[:used].view(H, n_used)
    free_ids = torch.zeros(num_pages, dtype=torch.int32, device=dev)
    n_free = num_pages - used
    # a fresh pool's free pages are kept in address order, so a run of pops returns a
    # run of consecutive page ids (live pages stay scattered)
    free_ids[:n_free] = torch.sort(perm[used:]).values
    free_top = torch.tensor([n_free], dtype=torch.int32, device=dev)

    masks = torch.zeros((H, mp), dtype=torch.int32, device=dev)
    masks[:, :n_used] = 0xFFFF
    last = N - (n_used - 1) * PAGE if tail_len is None else tail_len
    masks[:, n_used - 1] = (1 << last) - 1
    if hole_prob > 0:
        bits = (torch.rand(H, n_used, PAGE, generator=g, device=dev) >= hole_prob).to(torch.int32)
        word = (bits << torch.arange(PAGE, device=dev, dtype=torch.int32)).sum(-1)
        masks[:, :n_used] &= word
    page_mask = masks.to(torch.int16)
    n_pages = torch.full((H,), n_used, dtype=torch.int32, device=dev)

    # K/V pools: every page holds N(0,1) draws; live pages are (re)written per head
    k_pool = torch.zeros(num_pages, PAGE, D, dtype=dt, device=dev)
    v_pool = torch.zeros(num_pages, PAGE, D, dtype=dt, device=dev)
    chunk = max(1, (1 << 28) // max(1, n_used * PAGE * D * 4))
    plant = cfg.get("recipe") == "planted"
    n_plant = int(round(0.02 * N))
    for h0 in range(0, H, chunk):
        h1 = min(H, h0 + chunk)
        kl = torch.randn(h1 - h0, n_used * PAGE, D, generator=g, device=dev, dtype=torch.float32)
        vl = torch.randn(h1 - h0, n_used * PAGE, D, generator=g, device=dev, dtype=torch.float32)
        if plant:
            for h in range(h0, h1):
                s, kv = divmod(h, Hkv)
                qm = q[:, s, kv * G:(kv + 1) * G, :].reshape(-1, D).mean(0)
                u = qm / qm.norm()
                idx = torch.randperm(N, generator=g, device=dev)[:n_plant]
                kl[h - h0, idx] += 4.0 * math.sqrt(D) * u
        ids = table[h0:h1, :n_used].reshape(-1).long()
        k_pool[ids] = kl.to(dt).view(-1, PAGE, D)
        v_pool[ids] = vl.to(dt).view(-1, PAGE, D)

    if head_lens is not None:
        lens = [int(x) for x in head_lens]
        assert len(lens) == H and all(0 <= x <= N for x in lens), "one length <= N per head"
        released = []
        for h, ln in enumerate(lens):
            nh = -(-ln // PAGE)
            released.append(table[h, nh:n_used].clone())
            table[h, nh:] = -1
            masks[h, nh:] = 0
            if nh:
                masks[h, nh - 1] &= (1 << (ln - (nh - 1) * PAGE)) - 1
            n_pages[h] = nh
        page_mask = masks.to(torch.int16)
        back = torch.sort(torch.cat([free_ids[:n_free]] + released)).values
        n_free = back.numel()
        free_ids[:n_free] = back
        free_top.fill_(n_free)

    ref = None
    n_ref = cfg.get("n_ref", 0)
    if n_ref:
        # uniform without replacement over the valid slots of each head
        keys = torch.rand(H, n_used * PAGE, generator=g, device=dev)
        bits = ((page_mask[:, :n_used].to(torch.int32)[:, :, None] >>
                 torch.arange(PAGE, device=dev, dtype=torch.int32)) & 1).reshape(H, -1)
        keys = torch.where(bits.bool(), keys, torch.full_like(keys, -1.0))
        ref = torch.topk(keys, min(n_ref, n_used * PAGE), dim=1).indices.to(torch.int32)
        ref = torch.sort(ref, dim=1).values.contiguous()

    meta, (table, page_mask, n_pages, free_ids, free_top) = _pack(
        dev, [table, page_mask, n_pages, free_ids, free_top])
    return Workload(cfg=dict(cfg), q_obs=q_obs, k_pool=k_pool, v_pool=v_pool, page_table=table,
                    page_mask=page_mask, n_pages=n_pages, free_ids=free_ids, free_top=free_top,
                    max_pages=mp, tau=tau, ref_slots=ref, meta=meta)


def _pack(dev, tensors):
    """The tensors copied into views of one byte buffer, each at a 256-byte offset, so the
    whole mutable state is saved and restored by one copy.  Returns (buffer, views)."""
    offs, total = [], 0
    for t in tensors:
        offs.append(total)
        total += -(-t.numel() * t.element_size() // 256) * 256
    buf = torch.zeros(total, dtype=torch.uint8, device=dev)
    views = []
    for t, o in zip(tensors, offs):
        v = buf[o:o + t.numel() * t.element_size()].view(t.dtype).view(t.shape)
        v.copy_(t)
        views.append(v)
    return buf, views


_STATE = ("page_table", "page_mask", "n_pages", "free_ids", "free_top")


def clone_state(w: Workload) -> dict:
    """Copy of the mutable cache metadata (tables, masks, counts, allocator)."""
    if w.meta is not None:
        return {"meta": w.meta.clone()}
    return {k: getattr(w, k).clone() for k in _STATE}


def restore_state(w: Workload, st: dict) -> None:
    """Back to a clone_state copy: one device copy when the state shares one buffer."""
    for k, v in st.items():
        getattr(w, k).copy_(v)


def decode_step_inputs(cfg: dict, step: int, layer: int, device, NS_layer: int):
    """Fresh N(0,1) q, k, v for one decode step of one layer (seed, layer, step keyed)."""
    g = _gen(torch.device(device), (cfg["seed"] * 1_000_003 + layer) * 1_000_003 + step + 1)
    Hq, Hkv, D = cfg["Hq"], cfg["Hkv"], cfg["D"]
    dt = TORCH_DTYPE[cfg["dtype"]]
    q = torch.randn(NS_layer, Hq, D, generator=g, device=device).to(dt)
    k = torch.randn(NS_layer, Hkv, D, generator=g, device=device).to(dt)
    v = torch.randn(NS_layer, Hkv, D, generator=g, device=device).to(dt)
    return q, k, v


def synthetic_log_scores(w: Workload, seed: int, scale: float = 2.0, L_dense: int = 0):
    """Seeded stand-in log-scores [n_heads, S_max] fp32 (host numpy) for the stages that
    consume scores: N(0, scale^2) draws at every candidate slot (valid slots older than the
    dense tier), -inf elsewhere; a score-like input drawn without the method's arithmetic.
    Returns (scores, cand_len) with cand_len [n_heads] int32."""
    import numpy as np
    rng = np.random.default_rng(seed)
    n = w.n_pages.cpu().numpy().astype(np.int64)
    masks = w.page_mask.cpu().numpy().astype(np.int64) & 0xFFFF
    nd = np.minimum(n, -(-L_dense // PAGE))
    cand_len = (PAGE * (n - nd)).astype(np.int32)
    S = w.S_max
    bits = ((masks[:, :, None] >> np.arange(PAGE)) & 1).reshape(w.n_heads, -1).astype(bool)
    cand = bits & (np.arange(S)[None, :] < cand_len[:, None])
    s = (rng.standard_normal((w.n_heads, S)) * scale).astype(np.float32)
    s[~cand] = -np.inf
    return s, cand_len

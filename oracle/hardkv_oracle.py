"""CPU oracle for the Hard-KV decoding-time compression step.

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the
HIP path is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  The product path
(``paper_2606_28831_amd``) never imports, links or runs anything here, and this
module imports nothing from the product path.

Arithmetic is float64 (NumPy) except where the method is defined on integers
(the Top-p mass, page bookkeeping), which use exact Python integers.  Every
function works on ONE head at a time, written out from the definitions it
cites, with no blocking, fusion or reordering beyond what the definition states.

Notation (paper):
  z        raw attention logits, sm_scale * q . k   (App. F, standard attention)
  S        Softmax of logits; M_k(S) = sum of the Top-k entries (Sec. 3.2, Problem 1)
  T        temperature; Solution 2 form S_hat = Softmax(g(z) / T)  (Sec. 3.2)
  p        Top-p threshold; head-adaptive budget (Sec. 3.2, Problem 1)
  tiers    Dense / Sparse / Condensed Cascade Cache (Sec. 3.1)
  (o, SE)  attention state and merge operator (App. F)

Readings where the paper is silent:
  * window aggregation: mean over the G*W window rows of each row's softmax
    probabilities, in log domain;
  * candidates: valid slots before the dense tier; dense tier force-kept;
  * Top-p on fixed-point mass floor(c * 2^40), p quantised to 1e-6, ties in c
    go to the larger (more recent) slot index;
  * temperature solve: bisection in log T, fixed iteration count;
  * redundancy: -max cosine similarity against a supplied set of reference slots;
  * tiers are age bands of whole 16-slot pages;
  * Cautious Update: each window row votes with its own Top-p set of the
    candidates; under the hard budget the base set is ranked by (votes, c,
    slot index); attention sinks are the first n_sink logical slots;
  * hard-budget state: rewrite when 16 * n_pages > L_upper, sparse loading when
    the valid count exceeds L_lower, otherwise keep.

Parity status of each function is given in its docstring ("pinned by ...").
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE = 16            # slots per physical page
MASS_BITS = 40       # fixed-point fraction bits of the Top-p mass
P_QUANT = 10 ** 6    # p is quantised to multiples of 1e-6


# ---------------------------------------------------------------------------
# small helpers
# ---------------------------------------------------------------------------
def logsumexp(v) -> float:
    """log(sum(exp(v))) in float64 with max subtraction; empty or all -inf -> -inf."""
    v = np.asarray(v, dtype=np.float64)
    if v.size == 0:
        return -math.inf
    m = np.max(v)
    if m == -math.inf:
        return -math.inf
    return float(m + math.log(np.sum(np.exp(v - m))))


def read_head(pool: np.ndarray, table_row, mask_row, n_pages: int):
    """Logical view of one head's paged cache.

    Logical slot j lives at page position j // 16 of the head's table row,
    slot j % 16 of that physical page; it is valid when bit (j % 16) of the
    page's 16-bit mask is set.  Returns (rows [n_pages*16, D], valid [n_pages*16]).
    Head-flattened block table: Sec. 3.3.2 (P2) and App. B.1.
    """
    ids = np.asarray(table_row[:n_pages], dtype=np.int64)
    rows = pool[ids].reshape(n_pages * PAGE, pool.shape[-1])
    masks = np.asarray(mask_row[:n_pages], dtype=np.int64)
    valid = ((masks[:, None] >> np.arange(PAGE)[None, :]) & 1).astype(bool).reshape(-1)
    return rows, valid


def tier_pages(n_pages: int, L_dense: int, L_sparse: int):
    """Age bands of a head's page list (Sec. 3.1 Cascade Cache; tier sizes in pages).

    Returns (n_condensed, n_sparse, n_dense) with
      dense  = the newest ceil(L_dense/16) pages,
      sparse = the floor(L_sparse/16) pages before them,
      condensed = every older page.
    """
    nd = min(n_pages, -(-L_dense // PAGE))
    ns = min(n_pages - nd, L_sparse // PAGE)
    return n_pages - nd - ns, ns, nd


def candidate_mask(valid: np.ndarray, cand_len: int) -> np.ndarray:
    """Candidates: valid slots with logical index below cand_len (everything older
    than the dense tier; the dense tier is kept unconditionally, Sec. 3.1 Tier 1)."""
    j = np.arange(valid.shape[0])
    return valid & (j < cand_len)


# ---------------------------------------------------------------------------
# a1: importance scoring over the observation window
# ---------------------------------------------------------------------------
def score_head(q_rows, keys, valid, cand_len: int, sm_scale: float, row_lse_in=None):
    """Attention-mass importance of every candidate slot of one KV head.

    q_rows  [R, D]  the R = G*W window queries of the head's query group
    keys    [S, D]  logical keys of the head, valid [S]
    Returns (s [S], row_lse [R]):
      z[r, j]   = sm_scale * <q_r, k_j>                       (App. F)
      LSE_r     = log sum_{j valid} exp z[r, j]   (or row_lse_in if given)
      s_j       = log( (1/R) * sum_r exp(z[r, j] - LSE_r) )  for candidates j
      s_j       = -inf for non-candidates.
    This is the Reduce step of the three-step framework (App. E) applied to the
    raw attention distribution S that Problem 1 (Sec. 3.2) calibrates toward.
    Pinned by: sum_j exp(s_j) = 1 when every valid slot is a candidate; R = 1
    reduces to scipy's log_softmax; per-row scipy softmax averaged; row and
    page permutation invariances; masked slots equal to removed slots.
    """
    q = np.asarray(q_rows, dtype=np.float64)
    k = np.asarray(keys, dtype=np.float64)
    R, S = q.shape[0], k.shape[0]
    z = sm_scale * (q @ k.T)
    if row_lse_in is None:
        row_lse = np.array([logsumexp(z[r, valid]) for r in range(R)], dtype=np.float64)
    else:
        row_lse = np.asarray(row_lse_in, dtype=np.float64).copy()
    cand = candidate_mask(valid, cand_len)
    s = np.full(S, -math.inf, dtype=np.float64)
    for j in np.nonzero(cand)[0]:
        mass = np.mean(np.exp(z[:, j] - row_lse))
        s[j] = math.log(mass) if mass > 0.0 else -math.inf
    return s, row_lse


def redundancy_head(keys, valid, cand_len: int, ref_slots):
    """Key-redundancy importance (R-KV style pairwise key similarity turned into a
    logit-level transform, Sec. 4 baseline adaptations; Solution 2 form).

      x_red_j = -max_{i in ref, i != j} cos(k_i, k_j)   for candidates j
    A zero-norm key has cosine 0 with everything.  If every reference slot equals
    j (empty set) the maximum is taken as -1.  Non-candidates get -inf.
    Pinned by: exact duplicates give -1, orthogonal keys give 0, antiparallel
    give +1, scaling invariance, and a closed-form 2-D case.
    """
    k = np.asarray(keys, dtype=np.float64)
    S = k.shape[0]
    norms = np.sqrt(np.sum(k * k, axis=1))
    cand = candidate_mask(valid, cand_len)
    out = np.full(S, -math.inf, dtype=np.float64)
    refs = np.array([int(i) for i in ref_slots], dtype=np.int64)
    for j in np.nonzero(cand)[0]:
        others = refs[refs != j]                 # the reference set without j itself
        best = -1.0
        if len(others):
            denom = norms[others] * norms[j]
            dots = k[others] @ k[j]
            # a zero-norm key has cosine 0 with every other key
            cosv = np.where(denom == 0.0, 0.0, dots / np.where(denom == 0.0, 1.0, denom))
            best = max(best, float(np.max(cosv)))
        out[j] = -best
    return out


# ---------------------------------------------------------------------------
# a2: Logits Calibration (Sec. 3.2, Solution 2) and the temperature solve
# ---------------------------------------------------------------------------
def calibrate_head(x, cand, T: float = 1.0):
    """c = Softmax(x / T) over the candidate slots, 0 elsewhere; returns (c, lse)
    with lse = log sum_{cand} exp(x / T).  All -inf -> c = 0, lse = -inf.
    Solution 2: S_hat = S(g(z) / T)  (Sec. 3.2).
    Pinned by: sum c = 1, order invariance for every T > 0 (App. D.2 theorem),
    uniform x -> 1/n, scipy logsumexp.
    """
    x = np.asarray(x, dtype=np.float64)
    c = np.zeros(x.shape[0], dtype=np.float64)
    idx = np.nonzero(cand)[0]
    xs = x[idx] / float(T)
    lse = logsumexp(xs)
    if lse == -math.inf:
        return c, -math.inf
    c[idx] = np.exp(xs - lse)
    return c, lse


def pool_max_head(x, cand, radius: int):
    """Order-preserving pooling g of Solution 1 (Sec. 3.2, S_hat = S(g(z / T))), in its
    SnapKV form (Sec. 4 baselines): each candidate's score becomes the maximum of the
    candidate scores within `radius` logical slots on either side (itself included);
    non-candidates stay -inf and are never a neighbour.  The width 2*radius + 1 is not
    stated in the paper; the radius is an argument (3 by default in the pipeline).  Max
    commutes with the monotone log, so
    pooling log scores equals pooling the probabilities they are the logs of.
    Pinned by: radius 0 is the identity; scipy's maximum_filter1d over the candidate-
    masked row; a constant row stays constant; the result dominates the input.
    """
    x = np.asarray(x, dtype=np.float64)
    cand = np.asarray(cand, dtype=bool)
    S = x.shape[0]
    out = np.full(S, -math.inf, dtype=np.float64)
    for j in range(S):
        if not cand[j]:
            continue
        best = -math.inf
        for i in range(max(0, j - radius), min(S, j + radius + 1)):
            if cand[i] and x[i] > best:
                best = x[i]
        out[j] = best
    return out


def mix(cs, weights):
    """Mixture of calibrated distributions, sum_m w_m c^(m) (probability domain)."""
    out = np.zeros_like(np.asarray(cs[0], dtype=np.float64))
    for c, w in zip(cs, weights):
        out = out + float(w) * np.asarray(c, dtype=np.float64)
    return out


def order_desc(values, idx):
    """Slots `idx` ordered by value descending, ties to the larger slot index."""
    vals = np.asarray(values)
    return sorted((int(j) for j in idx), key=lambda j: (-float(vals[j]), -j))


def topk_mass(c, cand, k: int) -> float:
    """M_k(c): sum of the k largest candidate entries (Sec. 3.2, Problem 1)."""
    order = order_desc(c, np.nonzero(cand)[0])
    return float(sum(float(c[j]) for j in order[:k]))


def quantise_p(p: float) -> int:
    """p_q = round-half-even(p * 10^6), evaluated in float64."""
    return int(round(float(p) * P_QUANT))


def fixed_weight(cv: float) -> int:
    """w = floor(c * 2^40); NaN -> 0, values clamped to [0, 1].  Exact for fp32 c."""
    if cv != cv:
        return 0
    cv = min(max(float(cv), 0.0), 1.0)
    return int(math.floor(cv * float(1 << MASS_BITS)))


@dataclass
class ToppResult:
    sel: np.ndarray          # bool [S]
    k: int
    total: int               # integer mass of all candidates
    target: int              # integer mass the selection must reach
    sel_mass: int            # integer mass of the selected set
    order: list = field(default_factory=list)


def topp_head(c, cand, p: float, k_min: int = 1, k_max: int = 0) -> ToppResult:
    """Head-adaptive Top-p budget: the smallest prefix (in the order c desc, ties
    to the larger slot) whose mass reaches p of the total (Sec. 3.2, Problem 1).

    Integer rule:  w_j = floor(c_j 2^40), Total = sum w, p_q = round(p 1e6),
    target = ceil(p_q Total / 1e6), k = min{k : sum_{first k} w >= target}
    (k = 0 when target = 0), clamped to [min(k_min, n), min(k_max or n, n)].
    Pinned by: brute force over all subsets for n <= 12, uniform -> ceil(p n),
    one-hot -> 1, p = 1 -> all positive-weight slots, and the two-sided mass
    invariant; hand-derived golden cases.
    """
    c = np.asarray(c)
    idx = np.nonzero(cand)[0]
    n = len(idx)
    # inputs are probabilities: NaN counts as 0 and values are clamped to [0, 1]
    # before both the ordering and the fixed-point weights
    order = order_desc(np.clip(np.where(np.isnan(c), 0.0, c), 0.0, 1.0), idx)
    w = {j: fixed_weight(float(c[j])) for j in idx}
    total = sum(w.values())
    pq = quantise_p(p)
    target = -(-(pq * total) // P_QUANT)
    k = 0
    if target > 0:
        cum = 0
        for r, j in enumerate(order):
            cum += w[j]
            if cum >= target:
                k = r + 1
                break
    lo = min(max(k_min, 0), n)
    hi = n if k_max <= 0 else min(k_max, n)
    k = max(lo, min(k, hi))
    sel = np.zeros(c.shape[0], dtype=bool)
    sel[order[:k]] = True
    return ToppResult(sel=sel, k=k, total=total, target=target,
                      sel_mass=sum(w[j] for j in order[:k]), order=order)


def solve_T_head(x, cand, k: int, target_mass: float, T_lo: float = 1e-4,
                 T_hi: float = 1e4, iters: int = 40) -> float:
    """Temperature for Problem 1 by bisection (App. D.1, binary search on T).

    f(T) = M_k(Softmax(x / T)) - target_mass, where the Top-k set is that of x
    itself (order invariance, App. D.2 theorem).  Lower T sharpens and raises
    M_k, so f decreases in T.  The search runs on log T over [T_lo, T_hi] for a
    fixed number of halvings: if f(T_mid) > 0 the lower end moves up, otherwise
    the upper end moves down; the result is the midpoint of the final bracket.
    Pinned by: the two-level closed form T* = (a-b) / ln(m(n-k) / (k(1-m))).
    """
    x = np.asarray(x, dtype=np.float64)
    idx = np.nonzero(cand)[0]
    top = order_desc(x, idx)[:k]
    xs_all = x[idx]
    xs_top = x[top]
    a, b = math.log(T_lo), math.log(T_hi)
    for _ in range(iters):
        mid = 0.5 * (a + b)
        T = math.exp(mid)
        mass = math.exp(logsumexp(xs_top / T) - logsumexp(xs_all / T)) if k > 0 else 0.0
        if mass - target_mass > 0.0:
            a = mid
        else:
            b = mid
    return math.exp(0.5 * (a + b))


def topk_mass_and_grad(x, top, theta: float):
    """M_k(Softmax(x / T)) over the candidates x (1-D) with T = exp(theta), where `top`
    marks the Top-k members (fixed in T, App. D.2 theorem), and its derivative in theta:
    with u = 1/T, dM/du = M (E_top[x] - E_all[x]) (expectations under the top-k and the
    full softmax), and du/dtheta = -u.  Terms whose exponential is 0 add nothing to the
    expectations (so a candidate at -inf is simply absent)."""
    x = np.asarray(x, dtype=np.float64)
    if x.size == 0:                       # no candidates: no mass, no gradient (R16)
        return 0.0, 0.0
    u = math.exp(-theta)
    z = u * x
    zmax = float(np.max(z))
    if zmax == -math.inf:
        return 0.0, 0.0
    e = np.exp(z - zmax)
    s_all, s_top = float(e.sum()), float(e[top].sum())
    if s_top == 0.0:
        return 0.0, 0.0
    M = s_top / s_all
    with np.errstate(invalid="ignore"):
        xe = np.where(e > 0.0, x * e, 0.0)  # a term of weight 0 adds 0 (also for x = -inf)
    e_top = float(xe[top].sum()) / s_top
    e_all = float(xe.sum()) / s_all
    return M, -u * M * (e_top - e_all)


def solve_T_gd_head(x, cand, k: int, target_mass: float, T_init: float = 1.0,
                    lr: float = 0.05, iters: int = 200, tol: float = 0.0):
    """Temperature for Problem 1 by gradient descent (Alg. 1, Solution 2 form): the
    parameter is theta = log T (T stays positive), the loss the squared gap
    l = (M_k(Softmax(x / T)) - target)^2, the optimiser Adam (beta 0.9 / 0.999, eps 1e-8,
    bias-corrected, no weight decay).  Iterates until l < tol or `iters` updates.
    Returns (T, final loss).
    Pinned by: the two-level closed form T* = (a-b) / ln(m(n-k) / (k(1-m))) is reached;
    the gradient equals finite differences of scipy's softmax mass; iters = 0 returns
    T_init; the loss never ends above its start on monotone problems.
    """
    x = np.asarray(x, dtype=np.float64)
    idx = np.nonzero(cand)[0]
    xs = x[idx]
    order = order_desc(x, idx)[:k]
    top = np.isin(idx, np.asarray(order, dtype=np.int64))
    theta = math.log(T_init)
    m = v = 0.0
    b1, b2, eps = 0.9, 0.999, 1e-8
    loss = 0.0
    for t in range(1, iters + 1):
        M, dM = topk_mass_and_grad(xs, top, theta) if k > 0 else (0.0, 0.0)
        gap = M - target_mass
        loss = gap * gap
        if loss < tol:
            break
        g = 2.0 * gap * dM
        m = b1 * m + (1.0 - b1) * g
        v = b2 * v + (1.0 - b2) * g * g
        mh = m / (1.0 - b1 ** t)
        vh = v / (1.0 - b2 ** t)
        theta -= lr * mh / (math.sqrt(vh) + eps)
    if iters > 0:
        M, _ = topk_mass_and_grad(xs, top, theta) if k > 0 else (0.0, 0.0)
        loss = (M - target_mass) ** 2
    return math.exp(theta), loss


# ---------------------------------------------------------------------------
# a4: Cascade-Cache rewrite (Sec. 3.1 Step 3, Sec. 3.3.1 Rewrite Cache / Sparse Loading)
# ---------------------------------------------------------------------------
@dataclass
class PageEntry:
    kind: str                # "new" (condensed, rewritten) | "sparse" | "dense"
    mask: int                # 16-bit slot mask
    phys: int = -1           # kept physical id for sparse/dense pages
    src: list = field(default_factory=list)   # for "new": [(phys, slot)] per filled slot


@dataclass
class CompactResult:
    pages: list              # list[PageEntry], new logical page order
    freed: list              # physical ids released, in release order per head
    n_new: int               # number of freshly allocated pages


def compact_head(table_row, mask_row, n_pages: int, sel, L_dense: int, L_sparse: int):
    """Rewrite one head's page list into Cascade-Cache tiers.

    sel[j] marks the selected logical slots (only condensed and sparse bands are
    consulted).  Condensed band: every selected valid slot is copied, in
    ascending logical order, into fresh pages filled 16 at a time (all full but
    the last) -- the Rewrite Cache operation.  Sparse band: pages stay in place
    with mask &= selection (Sparse Loading); a page left empty is released.
    Dense band: untouched.  New order: [condensed][sparse][dense].
    Pinned by: byte equality with np.take of the selected rows, strictly
    ascending logical order, packing, count conservation, disjoint live/freed sets.
    """
    nc, ns, nd = tier_pages(n_pages, L_dense, L_sparse)
    sel = np.asarray(sel, dtype=bool)
    pages, freed = [], []
    gathered = []
    for pp in range(nc):
        m = int(mask_row[pp])
        for t in range(PAGE):
            if (m >> t) & 1 and sel[pp * PAGE + t]:
                gathered.append((int(table_row[pp]), t))
        freed.append(int(table_row[pp]))
    n_new = 0
    for start in range(0, len(gathered), PAGE):
        chunk = gathered[start:start + PAGE]
        pages.append(PageEntry(kind="new", mask=(1 << len(chunk)) - 1, src=chunk))
        n_new += 1
    for pp in range(nc, nc + ns):
        m = int(mask_row[pp])
        word = 0
        for t in range(PAGE):
            if sel[pp * PAGE + t]:
                word |= 1 << t
        m2 = m & word
        if m2 == 0:
            freed.append(int(table_row[pp]))
        else:
            pages.append(PageEntry(kind="sparse", mask=m2, phys=int(table_row[pp])))
    for pp in range(nc + ns, n_pages):
        pages.append(PageEntry(kind="dense", mask=int(mask_row[pp]), phys=int(table_row[pp])))
    return CompactResult(pages=pages, freed=freed, n_new=n_new)


# ---------------------------------------------------------------------------
# a5: paged decode attention (App. F)
# ---------------------------------------------------------------------------
def decode_head(q, keys, vals, valid, sm_scale: float):
    """Attention of G query heads over one KV head's valid slots.

    o_g = sum_j Softmax_j(sm_scale q_g . k_j) v_j,   lse_g = log sum_j exp(sm_scale q_g . k_j)
    (App. F standard attention and SE).  No valid slot -> o = 0, lse = -inf.
    Pinned by: a single slot gives o = v exactly, the merge operator over any
    partition equals the whole, scipy softmax.
    """
    q = np.atleast_2d(np.asarray(q, dtype=np.float64))
    k = np.asarray(keys, dtype=np.float64)[valid]
    v = np.asarray(vals, dtype=np.float64)[valid]
    G, D = q.shape
    if k.shape[0] == 0:
        return np.zeros((G, v.shape[1] if v.ndim == 2 else D)), np.full(G, -math.inf)
    z = sm_scale * (q @ k.T)
    lse = np.array([logsumexp(z[g]) for g in range(G)])
    pr = np.exp(z - lse[:, None])
    return pr @ v, lse


def merge_states(o1, lse1, o2, lse2):
    """Merge operator on attention states (App. F):
    o(I u J) = (o(I) SE(I) + o(J) SE(J)) / (SE(I) + SE(J)),  SE(I u J) = SE(I) + SE(J),
    carried in log form, lse = log SE."""
    o1, o2 = np.asarray(o1, np.float64), np.asarray(o2, np.float64)
    lse1, lse2 = np.asarray(lse1, np.float64), np.asarray(lse2, np.float64)
    m = np.maximum(lse1, lse2)
    m = np.where(np.isneginf(m), 0.0, m)
    a1, a2 = np.exp(lse1 - m), np.exp(lse2 - m)
    den = a1 + a2
    safe = np.where(den > 0, den, 1.0)
    o = (o1 * a1[..., None] + o2 * a2[..., None]) / safe[..., None]
    lse = np.where(den > 0, m + np.log(safe), -math.inf)
    return o, lse


# ---------------------------------------------------------------------------
# a6: dense-tail append (Sec. 3.1 Step 1)
# ---------------------------------------------------------------------------
def append_position(mask_row, n_pages: int):
    """Where the next token of a head goes: one past the highest valid slot of the
    newest page, or slot 0 of a new page when the table is empty or that page's
    slot 15 is taken.  Returns (page_position, slot, needs_new_page)."""
    if n_pages == 0:
        return 0, 0, True
    m = int(mask_row[n_pages - 1])
    top = m.bit_length()          # one past the highest set bit
    if top >= PAGE:
        return n_pages, 0, True
    return n_pages - 1, top, False


# ---------------------------------------------------------------------------
# Step 4 of the pipeline (Sec. 3.1): hard budget with Cautious Update voting and
# attention sinks; budget thresholds L_lower / L_upper (Sec. 3.3.1)
# ---------------------------------------------------------------------------
KEEP, SPARSE, REWRITE = 0, 1, 2      # hard-budget state of a head


def score_rows_head(q_rows, keys, valid, cand_len: int, sm_scale: float, row_lse):
    """Each window row's own attention probabilities over the candidates of one head:
    a[r, j] = exp(z[r, j] - LSE_r) for candidates j, 0 for every other slot, with
    z = sm_scale * q_r . k_j (App. F) and LSE_r the row's log-sum-exp over the valid slots.
    These are the distributions that the Cautious Update strategy (Sec. 3.1) lets vote
    one by one instead of through their mean (exp of score_head's s is that mean).
    Pinned by: every row equals scipy's softmax of its logits over the valid slots; the
    mean over rows equals exp(score_head's s); masked slots equal removed slots.
    """
    q = np.asarray(q_rows, dtype=np.float64)
    k = np.asarray(keys, dtype=np.float64)
    z = sm_scale * (q @ k.T)
    lse = np.asarray(row_lse, dtype=np.float64)
    cand = candidate_mask(valid, cand_len)
    a = np.zeros((q.shape[0], k.shape[0]), dtype=np.float64)
    for r in range(q.shape[0]):
        for j in np.nonzero(cand)[0]:
            a[r, j] = math.exp(z[r, j] - lse[r])
    return a


def vote_head(a_rows, cand, p: float):
    """Cautious Update votes (Sec. 3.1): the window is a voting period in which every
    query keeps its own selection.  Row r of a_rows is one window query's attention over
    the slots; it selects its own head-adaptive Top-p set of the candidates (the a3 rule,
    topp_head with k_min = 1), and the vote of slot j is the number of rows whose set
    holds j.  The cumulative selection mask is votes >= 1.
    Returns (votes [S] int, row_k [R] int, row_sel [R, S] bool).
    Pinned by: one row reproduces topp_head; equal rows give votes in {0, R}; the row
    order does not matter; a hand-worked three-row case.
    """
    a_rows = np.asarray(a_rows)
    R, S = a_rows.shape
    votes = np.zeros(S, dtype=np.int64)
    row_k = np.zeros(R, dtype=np.int64)
    row_sel = np.zeros((R, S), dtype=bool)
    for r in range(R):
        res = topp_head(a_rows[r], cand, p)
        row_sel[r] = res.sel
        row_k[r] = res.k
        votes += res.sel
    return votes, row_k, row_sel


def budget_plan_head(n_pages: int, mask_row, L_dense: int, L_lower: int, L_upper: int):
    """Hard-budget state of one head at a compression point (Sec. 3.3.1: above L_lower a
    selection is applied by sparse loading; above L_upper the cache is rewritten into
    contiguous pages; the budget k caps the usage at L_upper, Sec. 4 settings).
      used  = 16 * n_pages      slots of memory the head holds
      valid = its valid slots
      REWRITE  if used > L_upper
      SPARSE   elif valid > L_lower
      KEEP     otherwise.
    k_cap (REWRITE only; -1 = no cap) = max(0, 16 * floor(L_upper / 16) - 16 * nd), nd the
    dense pages: the rewritten candidates then fill at most floor(L_upper/16) - nd pages,
    so the head's new row stays within L_upper.
    Pinned by: hand cases on each side of both thresholds, and the bound
    16 * n_pages_after <= L_upper after budget_select + compact_mode_head.
    """
    nd = min(n_pages, -(-L_dense // PAGE))
    used = PAGE * n_pages
    valid = sum(bin(int(m) & 0xFFFF).count("1") for m in mask_row[:n_pages])
    if used > L_upper:
        return REWRITE, max(0, PAGE * (L_upper // PAGE) - PAGE * nd)
    if valid > L_lower:
        return SPARSE, -1
    return KEEP, -1


def budget_select_head(cand, votes=None, c=None, sel_in=None, mode: int = REWRITE,
                       k_cap: int = -1, n_sink: int = 0):
    """Step 4 selection under the hard budget (Sec. 3.1).
      KEEP: every candidate (the head is left as it is).
      otherwise:
        sinks = candidates j < n_sink, always kept (the attention sinks that the dense tier
                preserves, Sec. 3.1 Tier 1, and that the paper's baselines retain, Sec. 4);
        base  = the other candidates, restricted to votes[j] >= 1 when votes are given
                (the Cautious Update cumulative mask) and to sel_in[j] when given;
        base is ranked by (votes desc, c desc, slot desc) -- the vote ranking of Sec. 3.1, with
        the calibrated probability and then recency breaking ties; absent keys count as 0
        and c is clamped to [0, 1] with NaN as 0, as in topp_head -- and its first
        min(|base|, cap) entries are kept, cap = max(0, k_cap - |sinks|) (no cap if k_cap < 0).
    Returns (sel [S] bool, k = |sel|).
    Pinned by: without votes and with sel_in = a Top-p set, the cap reproduces topp_head
    with k_max; a cap at or above |base| keeps base; caps nest; brute force over the
    orderings of small sets.
    """
    cand = np.asarray(cand, dtype=bool)
    S = cand.shape[0]
    if mode == KEEP:
        return cand.copy(), int(cand.sum())
    j_all = np.arange(S)
    sinks = cand & (j_all < n_sink)
    base = cand & ~sinks
    if votes is not None:
        base &= np.asarray(votes) >= 1
    if sel_in is not None:
        base &= np.asarray(sel_in, dtype=bool)
    vv = np.zeros(S, dtype=np.int64) if votes is None else np.asarray(votes, dtype=np.int64)
    if c is None:
        cc = np.zeros(S)
    else:
        cc = np.asarray(c, dtype=np.float64)
        cc = np.clip(np.where(np.isnan(cc), 0.0, cc), 0.0, 1.0)
    order = sorted((int(j) for j in np.nonzero(base)[0]),
                   key=lambda j: (-int(vv[j]), -float(cc[j]), -j))
    n_s = int(sinks.sum())
    cap = len(order) if k_cap < 0 else min(len(order), max(0, k_cap - n_s))
    sel = sinks.copy()
    sel[order[:cap]] = True
    return sel, int(sel.sum())


def compact_mode_head(table_row, mask_row, n_pages: int, sel, L_dense: int, mode: int):
    """Cascade-Cache rewrite under the head's hard-budget state (Sec. 3.3.1):
      REWRITE  every page older than the dense tier is rewritten (Rewrite Cache);
      SPARSE   every page older than the dense tier keeps its place under the selection
               mask (Sparse Loading), emptied pages released;
      KEEP     nothing changes.
    The first two are compact_head with the sparse band sized to nothing or to every
    non-dense page.
    """
    if mode == KEEP:
        pages = [PageEntry(kind="dense", mask=int(mask_row[pp]), phys=int(table_row[pp]))
                 for pp in range(n_pages)]
        return CompactResult(pages=pages, freed=[], n_new=0)
    L_sparse = 0 if mode == REWRITE else PAGE * n_pages
    return compact_head(table_row, mask_row, n_pages, sel, L_dense, L_sparse)

"""GrowPage decode-step oracle: plain fp64 NumPy, test infrastructure only.

This module is the reference the HIP path is checked against.  It is imported
only by ``tests/``, by ``__graft_entry__.smoke()`` and by the CPU-baseline leg of
``bench.py``; the library and its Python binding never import it.  It shares no
code with the HIP path.

Paper: "GrowPage: On-Demand KV Budgeting for Efficient LLM Reasoning Serving"
(arXiv 2609.03494).  Each function names the passage it follows.  Arithmetic is
fp64 on inputs widened exactly from their storage type (float32 or bfloat16).
Where a floating-point value decides an integer (top-p working-set sizes,
Top-K selection), the decision is taken on the values rounded to float32: the
boundary interface hands the token scores over as float32 (one score per
candidate and KV head), so selection is defined on float32 scores, and the
working-set sizes are taken on the float32 weights those scores are the
maximum of, so that both decisions rest on the same numbers.  Sums taken on
the way are fp64.

Readings of points the paper leaves open (each one also listed in the design
notes) are marked "reading:" below.

Every function is pinned by tests against values fixed independently of it
(closed forms, brute force on small inputs, library routines, hand-worked
cases).  Parity unpinned: the end-to-end Delta values and the grow/compress
split that the full pipeline yields on the synthetic workloads -- the paper
prints no worked example for them (its grow ratio is measured on real model
activations), so they are reported, not asserted.

Storage conventions (the library's header fixes the same layout):
  K/V pools  [pool_pages][num_kv_heads][b][head_dim]
  page table [num_reqs][max_pages] int32, free-page stack free_list[:free_count]
  qstate     [slots][2][num_q_heads][head_dim] float32, view 0 = S, 1 = L
"""
from __future__ import annotations

from dataclasses import dataclass
from fractions import Fraction

import numpy as np

__all__ = [
    "COMPRESS", "GROW", "FALLBACK", "PREEMPT", "NOT_BOUNDARY", "SHRINK",
    "POLICIES", "METRICS",
    "Params", "widen", "narrow",
    "ema_update", "update_summaries",
    "softmax", "attention", "renormalised_subset_output", "worst_case_error",
    "gather_tokens", "decode_attention",
    "rms", "calibrate", "rope", "view_distributions", "top_p_count", "top_p_fragile",
    "entropy_count", "entropy_fragile",
    "token_scores", "score_request",
    "demand_trend", "decide_and_allocate",
    "local_quota", "select_retained", "compact_tokens",
    "PageState", "boundary_step",
    "append_token", "serve_step",
]

# decision codes
COMPRESS, GROW, FALLBACK, PREEMPT, NOT_BOUNDARY, SHRINK = 0, 1, 2, 3, 4, 5

# capacity-control policies (App. "alternative capacity-control policies") and
# demand metrics (Sec. 3.2; the signal ablation replaces top-p by entropy)
POLICIES = ("growpage", "fixed", "random", "inverse", "shrink")
METRICS = ("top_p", "entropy")


@dataclass
class Params:
    """Method constants.  Defaults: beta_S = 0.9, beta_L = 0.999 (Sec. 3.2),
    p = 0.99 (Sec. 3.2, working-set equation), tau = 0 (Sec. 3.2),
    k_loc = b/4 = 4 at b = 16 (reading: the paper's k_loc = 64 at b = 256,
    App. D.2, keeps a quarter of each block).  scale = 1/sqrt(head_dim)
    (reading: the paper does not restate the attention scale).

    Policy variants (App., alternative capacity-control policies):
    ``fixed`` grows only while the capacity is below ``fixed_pages`` pages
    (4096 tokens at b = 16) and compresses at every boundary after that;
    ``random`` compresses with probability ``compress_prob`` = 0.7 (a draw per
    boundary request, passed in) and grows otherwise; ``inverse`` grows iff
    Delta <= tau; ``shrink`` shrinks iff Delta < ``shrink_threshold`` = -0.005
    and the capacity after shrinking stays at least ``min_capacity_pages``
    pages (1024 tokens), grows iff Delta > tau, and compresses otherwise.
    ``metric``: ``top_p`` (default) or ``entropy`` (signal ablation).
    ``layout``: ``shift`` (default, the stable compaction) or ``fill`` (the
    hole-filling variant of ``compact_tokens``)."""
    beta_s: float = 0.9
    beta_l: float = 0.999
    p: float = 0.99
    tau: float = 0.0
    k_loc: int = 4
    rope_theta: float = 1.0e6
    reserve_pages: int = 0
    scale: float | None = None
    policy: str = "growpage"
    fixed_pages: int = 256
    compress_prob: float = 0.7
    shrink_threshold: float = -0.005
    min_capacity_pages: int = 64
    metric: str = "top_p"
    layout: str = "shift"

    def as_f32(self, head_dim: int) -> "Params":
        """The same constants rounded to float32, the precision in which the
        library receives them, with the scale made explicit."""
        f = lambda v: float(np.float32(v))
        sc = self.scale if self.scale is not None else 1.0 / np.sqrt(head_dim)
        return Params(f(self.beta_s), f(self.beta_l), f(self.p), f(self.tau), int(self.k_loc),
                      f(self.rope_theta), int(self.reserve_pages), f(sc), self.policy,
                      int(self.fixed_pages), f(self.compress_prob), f(self.shrink_threshold),
                      int(self.min_capacity_pages), self.metric, self.layout)


# ----------------------------------------------------------------------------
# storage <-> fp64
# ----------------------------------------------------------------------------

def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of stored float32 or bfloat16 (uint16 bit pattern) data."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return bits.view(np.float32).astype(np.float64)


def narrow(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 to the storage type, to nearest with ties to even.

    bfloat16 keeps 8 significant bits: the fp64 significand is rounded at bit
    45 directly (no intermediate float32 rounding)."""
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f32":
        return x.astype(np.float32)
    u = x.view(np.uint64)
    keep = (u >> np.uint64(45)) & np.uint64(1)
    rounded = ((u + np.uint64((1 << 44) - 1) + keep) >> np.uint64(45)) << np.uint64(45)
    f32 = rounded.view(np.float64).astype(np.float32)   # exact: 8 significant bits
    out = (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    out[nan] = np.uint16(0x7FC0)
    return out


# ----------------------------------------------------------------------------
# A1: dual-timescale query summaries (Sec. 3.2, eq. dual_ema; App. E.1)
# ----------------------------------------------------------------------------

def ema_update(qbar: np.ndarray, q: np.ndarray, beta: float) -> np.ndarray:
    """One step of qbar_t = beta * qbar_{t-1} + (1 - beta) * q_t (fp64)."""
    return beta * qbar + (1.0 - beta) * q


def update_summaries(q_pre, dtype, slot_ids, init, qstate, beta_s, beta_l):
    """Both summaries of every request, in a copy of the float32 summary pool.

    A request whose ``init`` flag is set is on the first decode step of its
    slot: both summaries become the current normalised pre-RoPE query,
    overwriting whatever the slot held (App. E.1).  Otherwise each view takes
    one EMA step with its own decay (Sec. 3.2).  Results are stored as float32.
    """
    out = np.array(qstate, dtype=np.float32, copy=True)
    q = widen(q_pre, dtype)
    for r in range(q.shape[0]):
        s = int(slot_ids[r])
        if init[r]:
            out[s, 0] = q[r].astype(np.float32)
            out[s, 1] = q[r].astype(np.float32)
        else:
            old = out[s].astype(np.float64)
            out[s, 0] = ema_update(old[0], q[r], beta_s).astype(np.float32)
            out[s, 1] = ema_update(old[1], q[r], beta_l).astype(np.float32)
    return out


# ----------------------------------------------------------------------------
# A2: attention (Sec. 3.1, eq. attention_outputs) and the paged decode
# ----------------------------------------------------------------------------

def softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max())
    return e / e.sum()


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """o = sum_i a_i v_i with a = softmax(scale * K q): returns (o, a)."""
    a = softmax(scale * (K @ q))
    return a @ V, a


def renormalised_subset_output(a: np.ndarray, V: np.ndarray, S) -> np.ndarray:
    """o_hat(S) = sum_{i in S} a_i / m(S) v_i, m(S) = sum_{i in S} a_i (Sec. 3.1)."""
    S = np.asarray(S)
    mS = a[S].sum()
    return (a[S] / mS) @ V[S]


def worst_case_error(a: np.ndarray, S, v_max: float) -> float:
    """Exact worst case of ||o - o_hat(S)|| over ||v_i|| <= V_max: 2 V_max (1 - m(S))
    (Sec. 3.1, eq. worst_case_error; proof in App. C)."""
    return 2.0 * v_max * (1.0 - float(np.asarray(a)[np.asarray(S)].sum()))


def gather_tokens(pool, table_row, m: int, b: int) -> np.ndarray:
    """Logical tokens [0, m) of one request: token i sits in page table_row[i // b],
    slot i % b.  ``pool`` is indexable by physical page id -> [Hkv, b, d].
    Returns [m, Hkv, d] in the storage type."""
    ids = [int(table_row[j]) for j in range((m + b - 1) // b)]
    if not ids:
        raise ValueError("empty request")
    if min(ids) < 0:
        raise ValueError("page table entry -1 inside the resident range")
    pages = [pool[pid] for pid in ids]
    stacked = np.stack(pages)                     # [P, Hkv, b, d]
    tok = stacked.transpose(0, 2, 1, 3).reshape(-1, stacked.shape[1], stacked.shape[3])
    return tok[:m]


def decode_attention(k_pool, v_pool, dtype, page_table, seq_lens, q_post, num_q_heads,
                     scale, b=16, requests=None):
    """Paged decode attention over each request's resident tokens (Sec. 3.1,
    eq. attention_outputs, evaluated token by token over the logical sequence).
    Query head g reads KV head g // (Hq / Hkv) (grouped-query attention).
    Returns fp64 [R, Hq, d] (only rows in ``requests`` are filled if given)."""
    q = widen(q_post, dtype)
    R, Hq, d = q.shape
    out = np.full((R, Hq, d), np.nan)
    reqs = range(R) if requests is None else requests
    for r in reqs:
        m = int(seq_lens[r])
        if m == 0:
            out[r] = 0.0          # reading: no resident token -> zero output
            continue
        K = widen(gather_tokens(k_pool, page_table[r], m, b), dtype)
        V = widen(gather_tokens(v_pool, page_table[r], m, b), dtype)
        G = Hq // K.shape[1]
        for g in range(Hq):
            out[r, g], _ = attention(q[r, g], K[:, g // G], V[:, g // G], scale)
    return out


# ----------------------------------------------------------------------------
# A4-A6: boundary scoring (Sec. 3.2, App. E.1)
# ----------------------------------------------------------------------------

def rms(x: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64)
    return float(np.sqrt(np.mean(x * x)))


def calibrate(q_t: np.ndarray, qbar: np.ndarray) -> np.ndarray:
    """gamma = RMS(q_t) / RMS(qbar), q_tilde = gamma * qbar, per query head
    (App. E.1, eq. rms_calibration).  reading: a summary with RMS 0 stays 0."""
    den = rms(qbar)
    if den == 0.0:
        return np.zeros_like(qbar, dtype=np.float64)
    return (rms(q_t) / den) * np.asarray(qbar, dtype=np.float64)


def rope(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotary position embedding at position ``pos`` (App. E.1: the calibrated
    summaries are rotated at the current position).  reading: the half-split
    pairing (dims i and i + d/2, angle pos * theta^(-2i/d)) used by Qwen3,
    theta = 1e6."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    i = np.arange(half, dtype=np.float64)
    ang = float(pos) * theta ** (-2.0 * i / d)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def view_distributions(K_cand: np.ndarray, q_t: np.ndarray, qbar_s: np.ndarray,
                       qbar_l: np.ndarray, pos: int, theta: float, scale: float) -> np.ndarray:
    """Attention distributions of the two aligned summaries over the candidate
    keys, per KV head: a[x, h, i] for x in (S, L).

    For every query head g of KV head h: calibrate the summary to RMS(q_t),
    rotate it at the current position, softmax of scale * (k_i . q_tilde) over
    the candidates (Sec. 3.2, App. E.1).  reading: the G query heads of a KV
    head are merged by averaging their distributions (the paper keeps the
    native GQA head mapping and indexes the working set by KV head)."""
    C, Hkv, d = K_cand.shape
    Hq = q_t.shape[0]
    G = Hq // Hkv
    a = np.zeros((2, Hkv, C))
    for x, qbar in enumerate((qbar_s, qbar_l)):
        for g in range(Hq):
            qt = rope(calibrate(q_t[g], qbar[g]), pos, theta)
            a[x, g // G] += softmax(scale * (K_cand[:, g // G] @ qt))
        a[x] /= G
    return a


def top_p_count(a32: np.ndarray, p: float) -> int:
    """K = min{k : sum of the k largest weights >= p} (Sec. 3.1, eq.
    attention_demand; Sec. 3.2, eq. working_set_ratio).  Weights are the
    float32 values; the running sum is fp64 in descending order.  If the whole
    mass stays below p, K = len(a)."""
    v = np.sort(np.asarray(a32, dtype=np.float32).astype(np.float64))[::-1]
    csum = np.cumsum(v)
    hit = np.nonzero(csum >= p)[0]
    return int(hit[0]) + 1 if hit.size else int(v.size)


def top_p_fragile(a32: np.ndarray, p: float, eps: float = 1e-6) -> bool:
    """True when the running sum passes p within eps, so that float rounding in
    another implementation may move K by one."""
    v = np.sort(np.asarray(a32, dtype=np.float32).astype(np.float64))[::-1]
    csum = np.cumsum(v)
    k = top_p_count(a32, p)
    near = abs(csum[k - 1] - p) <= eps
    if k >= 2:
        near = near or abs(csum[k - 2] - p) <= eps
    return bool(near)


def entropy_count(a32: np.ndarray) -> int:
    """Working-set size from the attention entropy (the signal ablation's
    alternative to top-p): H = -sum a ln a over the float32 weights (fp64,
    zero weights contribute nothing), K = exp(H) rounded to the nearest
    integer, at least 1 and at most len(a).
    reading: the paper names the metric without defining the size; exp(H) is
    the number of equally weighted tokens with the same entropy."""
    v = np.asarray(a32, dtype=np.float32).astype(np.float64)
    v = v[v > 0]
    if v.size == 0:
        return 1
    H = -float(np.sum(v * np.log(v)))
    k = int(np.floor(np.exp(H) + 0.5))
    return max(1, min(k, int(np.asarray(a32).size)))


def entropy_fragile(a32: np.ndarray, eps: float = 1e-6) -> bool:
    """True when exp(H) lies within eps (relative) of a rounding midpoint."""
    v = np.asarray(a32, dtype=np.float32).astype(np.float64)
    v = v[v > 0]
    if v.size == 0:
        return False
    e = float(np.exp(-np.sum(v * np.log(v))))
    frac = e - np.floor(e)
    return bool(abs(frac - 0.5) <= eps * max(1.0, e))


def token_scores(a_s32: np.ndarray, a_l32: np.ndarray) -> np.ndarray:
    """s_i = max(a^S_i, a^L_i) per KV head (Sec. 3.3, eq. token_score)."""
    return np.maximum(np.asarray(a_s32, np.float32), np.asarray(a_l32, np.float32))


def score_request(tokens, dtype, P, b, q_t, qbar, pos, params: Params, scale):
    """Boundary scoring of one request at one layer.

    tokens: [>= (P-1)b, Hkv, d] logical keys (storage type); the candidate set
    is every cached token except the most recent page, i.e. slots [0, (P-1)b)
    (Sec. 3.2; App. E.1).  qbar: [2, Hq, d] the updated summaries.
    Returns (counts [Hkv, 2] int, scores [Hkv, C] float32, a32 [2, Hkv, C]).
    reading: with P <= 1 the candidate set is empty and both counts are 0."""
    C = (P - 1) * b
    Hkv = tokens.shape[1]
    if C <= 0:
        return (np.zeros((Hkv, 2), np.int64), np.zeros((Hkv, 0), np.float32),
                np.zeros((2, Hkv, 0), np.float32))
    K = widen(tokens[:C], dtype)
    a = view_distributions(K, widen(q_t, dtype), np.asarray(qbar[0], np.float64),
                           np.asarray(qbar[1], np.float64), pos, params.rope_theta, scale)
    a32 = a.astype(np.float32)
    if params.metric == "entropy":
        count = lambda w: entropy_count(w)
    else:
        count = lambda w: top_p_count(w, params.p)
    counts = np.array([[count(a32[x, h]) for x in range(2)] for h in range(Hkv)], dtype=np.int64)
    return counts, token_scores(a32[0], a32[1]), a32


# ----------------------------------------------------------------------------
# A7: demand trend, decision and page allocation (Sec. 3.2, 3.3, 4.2; App. E.2)
# ----------------------------------------------------------------------------

def demand_trend(k_s, k_l, C: int) -> Fraction:
    """Delta = r^S - r^L with r^x the mean over (layer, KV head) of K^x / |C|
    (Sec. 3.2, eq. demand_aggregation), as an exact rational."""
    k_s = np.asarray(k_s).ravel()
    k_l = np.asarray(k_l).ravel()
    n = k_s.size
    r_s = sum(Fraction(int(k), C) for k in k_s) / n
    r_l = sum(Fraction(int(k), C) for k in k_l) / n
    return r_s - r_l


@dataclass
class PageState:
    page_table: np.ndarray
    num_pages: np.ndarray
    seq_lens: np.ndarray
    refcount: np.ndarray
    free_list: np.ndarray
    free_count: int

    def copy(self) -> "PageState":
        return PageState(self.page_table.copy(), self.num_pages.copy(), self.seq_lens.copy(),
                         self.refcount.copy(), self.free_list.copy(), int(self.free_count))


def _wants(policy_params: Params, dl, P: int, draw):
    """(want_grow, want_shrink) of one boundary request at P >= 2 pages with
    demand trend dl (an exact rational, or None when the threshold is
    infinite)."""
    pp = policy_params
    tau = Fraction(float(pp.tau)) if np.isfinite(pp.tau) else None
    above = (pp.tau < 0) if tau is None else dl > tau          # Delta > tau
    if pp.policy == "growpage":
        return above, False
    if pp.policy == "inverse":
        return not above, False
    if pp.policy == "fixed":
        return P < pp.fixed_pages, False
    if pp.policy == "random":
        # reading: the draw is uniform in [0, 1); compress iff draw < prob
        return not (float(np.float32(draw)) < float(np.float32(pp.compress_prob))), False
    if pp.policy == "shrink":
        # reading: a shrink keeps at least two pages (one page of survivors
        # plus one of free slots), whatever the floor says
        shrink = (dl < Fraction(float(pp.shrink_threshold))) and (P - 1 >= max(pp.min_capacity_pages, 2))
        return above, shrink
    raise ValueError(f"unknown policy {pp.policy!r}")


def decide_and_allocate(state: PageState, bnd, counts, b: int, params: Params, draws=None):
    """Decision and allocation for the boundary requests, in list order.

    counts[i]: [layers, Hkv, 2] working-set sizes of boundary request i.
    Grow by One Page iff Delta > tau (Sec. 3.2), popping the top of the
    free-page stack and appending it to the block table (Sec. 3.3, 4.2).
    If no page can be granted the request compresses instead (fallback,
    Sec. 4.2).  Compress & Hold keeps the allocation (Sec. 3.3); pages shared
    with other requests are never written, so a compressing request first takes
    one new private page per shared page and drops its reference to the shared
    one (App. E.2); if those pages cannot be had the request is preempted and
    left untouched.  The policy variants (``params.policy``; App., alternative
    capacity-control policies) change only which action is wanted; ``draws``
    [Rb] are the uniform draws of the random policy.  Shrink keeps P - 1 pages:
    the last page leaves the table and loses the request's reference, and
    (P - 2) b tokens stay resident (two pages' worth evicted, one page of free
    slots).
    readings: requests earlier in the list win scarce pages; "safely" granted
    means more than ``reserve_pages`` pages are free and the block table has
    room; a request with P <= 1 cannot compress, so it grows if it can and is
    preempted otherwise (the fixed policy grows below its budget only); a page
    counts as shared if its reference count exceeds one when the call starts;
    references are dropped after every pop of the call and pages whose count
    reaches zero are pushed back onto the stack in ascending page-id order.

    Mutates ``state``; returns (decisions [Rb] int, delta [Rb] float32)."""
    Rb = len(bnd)
    dec = np.zeros(Rb, dtype=np.int64)
    delta = np.zeros(Rb, dtype=np.float32)
    ref_at_start = state.refcount.copy()
    dropped = []
    max_pages = state.page_table.shape[1]
    for i in range(Rb):
        r = int(bnd[i])
        P = int(state.num_pages[r])
        if int(state.seq_lens[r]) != P * b:
            dec[i] = NOT_BOUNDARY
            continue
        draw = None if draws is None else draws[i]
        if P <= 1:
            want_grow = P < params.fixed_pages if params.policy == "fixed" else True
            want_shrink = False
        else:
            C = (P - 1) * b
            cs = np.asarray(counts[i])
            dl = demand_trend(cs[..., 0], cs[..., 1], C)
            delta[i] = np.float32(float(dl))
            want_grow, want_shrink = _wants(params, dl, P, draw)
        can_grow = state.free_count > params.reserve_pages and P < max_pages
        if want_grow and can_grow:
            pid = int(state.free_list[state.free_count - 1])
            state.free_count -= 1
            state.page_table[r, P] = pid
            state.refcount[pid] = 1
            state.num_pages[r] = P + 1
            dec[i] = GROW
            continue
        if P <= 1:
            dec[i] = PREEMPT
            continue
        keep = P - 1 if want_shrink else P          # pages left in the table
        shared = [j for j in range(keep) if ref_at_start[state.page_table[r, j]] > 1]
        if len(shared) > state.free_count:
            dec[i] = PREEMPT
            continue
        for j in shared:
            pid = int(state.free_list[state.free_count - 1])
            state.free_count -= 1
            dropped.append(int(state.page_table[r, j]))
            state.page_table[r, j] = pid
            state.refcount[pid] = 1
        if want_shrink:
            dropped.append(int(state.page_table[r, P - 1]))
            state.page_table[r, P - 1] = -1
            state.num_pages[r] = P - 1
            state.seq_lens[r] = (P - 2) * b
            dec[i] = SHRINK
        else:
            state.seq_lens[r] = (P - 1) * b
            dec[i] = FALLBACK if want_grow else COMPRESS
    for old in dropped:
        state.refcount[old] -= 1
    for pid in sorted({old for old in dropped if state.refcount[old] == 0}):
        state.free_list[state.free_count] = pid
        state.free_count += 1
    return dec, delta


# ----------------------------------------------------------------------------
# A8: selection (Sec. 3.3, eq. local_global_selection)
# ----------------------------------------------------------------------------

def local_quota(P: int, b: int, k_loc: int, drop: int = 1) -> int:
    """Per-block quota: k_loc, capped so the local picks fit in K_t.
    reading: compressing frees exactly one page, so (P-1) b slots stay
    occupied and the b protected recent tokens take one page of them
    (Sec. 3.3; App. E.2); K_t = (P-2) b historical tokens are kept.  A shrink
    evicts ``drop`` = 2 pages' worth, K_t = (P-3) b."""
    K_t = (P - 1 - drop) * b
    return max(0, min(k_loc, K_t // (P - 1)))


def _order(s32: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Indices of idx sorted by score descending, then slot ascending.
    reading: ties go to the earlier slot."""
    return idx[np.lexsort((idx, -s32[idx].astype(np.float64)))]


def select_retained(s32: np.ndarray, P: int, b: int, k_loc: int, drop: int = 1) -> np.ndarray:
    """S = S_loc U TopK_{K_t - |S_loc|}(C minus S_loc), S_loc = union over
    historical blocks B_j of TopK_{k_loc}(B_j) (Sec. 3.3).  Blocks are the
    pages of the candidate set; K_t = (P - 1 - drop) b (drop = 1 for Compress
    & Hold, 2 for a shrink).  Returns the kept slots in ascending order."""
    s32 = np.asarray(s32, dtype=np.float32)
    C = (P - 1) * b
    assert s32.shape[0] == C
    K_t = (P - 1 - drop) * b
    q = local_quota(P, b, k_loc, drop)
    local = []
    for j in range(P - 1):
        blk = np.arange(j * b, (j + 1) * b)
        local.extend(_order(s32, blk)[:q].tolist())
    local = np.array(sorted(local), dtype=np.int64)
    rest = np.setdiff1d(np.arange(C), local)
    glob = _order(s32, rest)[: K_t - local.size]
    return np.sort(np.concatenate([local, glob])).astype(np.int64)


# ----------------------------------------------------------------------------
# A9: compaction (Sec. 3.3; Sec. 4.2; App. E.2)
# ----------------------------------------------------------------------------

def compact_tokens(tokens: np.ndarray, kept: np.ndarray, P: int, b: int, drop: int = 1,
                   layout: str = "shift") -> np.ndarray:
    """New logical contents of one KV head after Compress & Hold (drop = 1) or
    a shrink (drop = 2); the survivors (kept historical tokens and the b
    protected tokens of the last page) end up in slots [0, (P - drop) b).
    Later slots keep their old contents (they are free).

    layout "shift": the kept tokens in their original order, then the
    protected page (reading: the order is stable).
    layout "fill": the hole-filling variant (every survivor below
    T = (P - drop) b stays where it is; the survivors at or above T, in slot
    order, fill the evicted slots below T, in slot order), which moves O(b)
    tokens instead of shifting the whole cache.  Attention over the resident
    tokens does not depend on their order; later events see pages that mix
    old and recent tokens."""
    out = tokens.copy()
    if layout == "shift":
        K_t = (P - 1 - drop) * b
        out[:K_t] = tokens[kept]
        out[K_t:K_t + b] = tokens[(P - 1) * b: P * b]
        return out
    if layout != "fill":
        raise ValueError(f"unknown layout {layout!r}")
    T = (P - drop) * b
    survivors = set(int(x) for x in kept) | set(range((P - 1) * b, P * b))
    holes = [slot for slot in range(T) if slot not in survivors]
    movers = [slot for slot in range(T, P * b) if slot in survivors]
    assert len(holes) == len(movers)
    for dst, src in zip(holes, movers):
        out[dst] = tokens[src]
    return out


# ----------------------------------------------------------------------------
# One boundary event over a whole (small) pool
# ----------------------------------------------------------------------------

def boundary_step(layers, dtype, state: PageState, q_pre, qstate, slot_ids, positions, bnd,
                  params: Params, b: int = 16, draws=None, counts=None):
    """Score, decide, select and compact, for every boundary request, over one or
    more layers.  ``layers`` is a list of (k_pool, v_pool) dense arrays
    [pool_pages, Hkv, b, d] (storage type) that are modified in place, and
    qstate a list with each layer's summary pool.
    ``q_pre`` and ``qstate`` are one array each, or a list with one per layer.
    ``counts`` (optional, [Rb] of [layers, Hkv, 2]): working-set sizes to decide
    with in place of the ones the scoring yields -- a test hook for sizes that
    another implementation obtained where the rounding band excuses a
    difference of one; scores and everything after the decision are computed
    as usual.
    Returns dict(decisions, delta, counts, scores, kept, counters)."""
    n_layers = len(layers)
    q_layers = list(q_pre) if isinstance(q_pre, (list, tuple)) else [q_pre] * n_layers
    s_layers = list(qstate) if isinstance(qstate, (list, tuple)) else [qstate] * n_layers
    d = layers[0][0].shape[-1]
    scale = params.scale if params.scale is not None else 1.0 / np.sqrt(d)
    counts_all, scores_all, weights_all = [], [], []
    for i, r in enumerate(bnd):
        r = int(r)
        P = int(state.num_pages[r])
        per_layer_c, per_layer_s, per_layer_w = [], [], []
        at_boundary = int(state.seq_lens[r]) == P * b
        for ell, (kp, vp) in enumerate(layers):
            if at_boundary and P >= 2:
                toks = gather_tokens(kp, state.page_table[r], P * b, b)
                c, s, a32 = score_request(toks, dtype, P, b, q_layers[ell][r],
                                          s_layers[ell][int(slot_ids[r])], int(positions[r]),
                                          params, scale)
            else:
                Hkv = kp.shape[1]
                c = np.zeros((Hkv, 2), np.int64)
                s = np.zeros((Hkv, 0), np.float32)
                a32 = np.zeros((2, Hkv, 0), np.float32)
            per_layer_c.append(c)
            per_layer_s.append(s)
            per_layer_w.append(a32)
        counts_all.append(np.stack(per_layer_c))
        scores_all.append(per_layer_s)
        weights_all.append(per_layer_w)
    if counts is not None:
        counts_all = [np.asarray(c, np.int64).copy() for c in counts]
    old_tables = {int(r): state.page_table[int(r)].copy() for r in bnd}
    old_pages = {int(r): int(state.num_pages[int(r)]) for r in bnd}
    dec, delta = decide_and_allocate(state, bnd, counts_all, b, params, draws)
    kept_all = {}
    for i, r in enumerate(bnd):
        r = int(r)
        if dec[i] not in (COMPRESS, FALLBACK, SHRINK):
            continue
        drop = 2 if dec[i] == SHRINK else 1
        P = old_pages[r]
        for ell, (kp, vp) in enumerate(layers):
            old = old_tables[r]
            new = state.page_table[r]
            for pool in (kp, vp):
                toks = gather_tokens(pool, old, P * b, b).copy()      # [P b, Hkv, d]
                for h in range(toks.shape[1]):
                    kept = select_retained(scores_all[i][ell][h], P, b, params.k_loc, drop)
                    kept_all[(i, ell, h)] = kept
                    toks[:, h] = compact_tokens(toks[:, h], kept, P, b, drop, params.layout)
                # write the resident pages back through the new table
                for j in range(P - drop):
                    pool[int(new[j])] = toks[j * b:(j + 1) * b].transpose(1, 0, 2)
    counters = np.zeros(4, dtype=np.int64)
    for code in dec:
        if code == SHRINK:
            counters[COMPRESS] += 1          # reading: a shrink counts as a compression
        elif code < 4:
            counters[code] += 1
    return dict(decisions=dec, delta=delta, counts=counts_all, scores=scores_all,
                weights=weights_all, kept=kept_all, counters=counters)


# ----------------------------------------------------------------------------
# A decode loop: one token per request and step, boundary events as they come,
# compaction asynchronous to the next step (App. E.3)
# ----------------------------------------------------------------------------

def append_token(pools, state: PageState, r: int, kv_new, b: int = 16) -> bool:
    """Write the current token's K and V ([Hkv, d] each, per layer) of request
    r at slot m_r of its paged cache and count it resident.  A request whose
    pages are full (m_r = P_r b) cannot take a token: it is at a capacity
    boundary and waits for a decision (Sec. 3.3).  Returns whether it
    appended."""
    m, P = int(state.seq_lens[r]), int(state.num_pages[r])
    if m >= P * b:
        return False
    pid = int(state.page_table[r, m // b])
    for (kp, vp), (k_new, v_new) in zip(pools, kv_new):
        kp[pid, :, m % b] = k_new
        vp[pid, :, m % b] = v_new
    state.seq_lens[r] = m + 1
    return True


def serve_step(pools, dtype, state: PageState, held, qstate, slot_ids, positions, inputs,
               params: Params, b: int = 16):
    """One decode step of a batch with asynchronous compaction (App. E.3).

    ``held``: requests whose compaction from the previous step is still
    running; they sit this step out (no token, no summary update, no output)
    and rejoin the next one.  Every other request appends its token if it has
    room, updates its summaries (Sec. 3.2; only requests that took a token),
    and decodes over its resident tokens (Sec. 3.1).  Requests whose pages are
    now full take the boundary event (``boundary_step``, in request order);
    those that compress or shrink are held for the next step.

    ``inputs``: dict with k_new, v_new ([R, Hkv, d] per layer, lists) and
    q_pre, q_post ([R, Hq, d]).  ``positions`` (logical index of each
    request's current token) advances with every appended token.
    reading: a request that could not take a token (preempted at its boundary)
    still decodes over its full cache and meets its boundary again.
    Returns (out [R, Hq, d] fp64 with NaN rows for held requests, new qstate,
    new held set, boundary_step result, appended list)."""
    R = state.page_table.shape[0]
    held = set(int(r) for r in held)
    active = [r for r in range(R) if r not in held]
    appended = []
    for r in active:
        kv_r = [(k[r], v[r]) for k, v in zip(inputs["k_new"], inputs["v_new"])]
        if append_token(pools, state, r, kv_r, b):
            positions[r] += 1
            appended.append(r)
    qs = np.array(qstate, dtype=np.float32, copy=True)
    if appended:
        idx = np.array(appended)
        upd = update_summaries(inputs["q_pre"][idx], dtype, slot_ids[idx],
                               np.zeros(idx.size, np.uint8), qs, params.beta_s, params.beta_l)
        qs = upd
    d = pools[0][0].shape[-1]
    scale = params.scale if params.scale is not None else 1.0 / np.sqrt(d)
    Hq = inputs["q_post"].shape[1]
    out = decode_attention(pools[0][0], pools[0][1], dtype, state.page_table, state.seq_lens,
                           inputs["q_post"], Hq, scale, b, requests=active)
    bnd = np.array([r for r in active if int(state.seq_lens[r]) == int(state.num_pages[r]) * b],
                   dtype=np.int32)
    res = boundary_step(pools, dtype, state, inputs["q_pre"], qs, slot_ids, positions, bnd, params, b)
    new_held = {int(bnd[i]) for i, dec in enumerate(res["decisions"])
                if dec in (COMPRESS, FALLBACK, SHRINK)}
    return out, qs, new_held, res, appended

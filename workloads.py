"""Seeded synthetic inputs for one decode step of GrowPage's hot path.

This module is the only code shared by the oracle tests, the HIP-path tests and
the benchmark.  It draws random numbers and lays them out as a paged KV pool; it
holds none of the method's arithmetic (no attention, no summary update, no RMS
calibration or RoPE, no scoring, no selection, no compaction).

Layout (what the library's header also fixes):
  * K and V pools: ``[pool_pages][num_kv_heads][page_size][head_dim]`` in the
    storage dtype (float32, or bfloat16 kept here as uint16 bit patterns);
  * page table ``[num_reqs][max_pages]`` int32, unused entries = -1;
  * ``num_pages`` (P_r), ``seq_lens`` (m_r, resident tokens), ``positions``
    (logical index of the current token, n_r - 1);
  * ``refcount[pool_pages]``, free-page stack ``free_list[:free_count]``
    (the top of the stack is ``free_list[free_count-1]``);
  * query-summary pool ``qstate[M][2][num_q_heads][head_dim]`` float32
    (index 0 = short view S, 1 = long view L), M = 512 query slots.

Page-budget reading (how configs that name a "budget" map onto GrowPage,
which has no fixed budget): a request that has grown to B pages and generated
n tokens holds P = min(ceil(n/b), B) pages and m = n tokens if n <= B*b, else
(B-1)*b + (n mod b, or b when that is 0) tokens -- it compressed at earlier
boundaries.  It sits at a capacity boundary iff m == P*b, i.e. iff b | n.

Slots of a partially filled last page, summary slots owned by no request and
pool pages owned by no request are filled with NaN so that any read of them
shows up in the results.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

PAGE = 16
SLOTS = 512                      # query-summary slots (max_num_seqs); more when a batch is larger
BF16_NAN = np.uint16(0x7FC0)


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (input synthesis only)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) >> np.uint32(16)).astype(np.uint16)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


@dataclass
class Workload:
    name: str
    dtype: str                     # "f32" or "bf16" (storage of K, V, q)
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    logical_lens: np.ndarray       # n_r
    budgets: np.ndarray | None     # B_r (pages) or None
    page_table: np.ndarray         # [R, max_pages] int32
    num_pages: np.ndarray          # [R] int32
    seq_lens: np.ndarray           # [R] int32
    positions: np.ndarray          # [R] int32
    refcount: np.ndarray           # [pool_pages] int32
    free_list: np.ndarray          # [pool_pages] int32
    free_count: int
    page_row: np.ndarray           # [pool_pages] int32: row of k_data/v_data or -1
    k_data: np.ndarray             # [U, Hkv, b, d] storage dtype
    v_data: np.ndarray
    q_post: np.ndarray             # [R, Hq, d] storage dtype
    q_pre: np.ndarray              # [R, Hq, d] storage dtype
    qstate: np.ndarray             # [M, 2, Hq, d] float32
    slot_ids: np.ndarray           # [R] int32
    init: np.ndarray               # [R] uint8
    boundary: np.ndarray           # [Rb] int32, ascending
    heavy: list = field(default_factory=list)   # per request: [Hkv] arrays of heavy slots
    q_priors: np.ndarray | None = None          # [n, R, Hq, d] (tiny case only)
    meta: dict = field(default_factory=dict)

    @property
    def num_reqs(self) -> int:
        return int(self.num_pages.shape[0])

    @property
    def pool_pages(self) -> int:
        return int(self.refcount.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def storage(self):
        return np.float32 if self.dtype == "f32" else np.uint16

    def dense_pool(self, which: str) -> np.ndarray:
        """Whole pool as one array (small workloads only); empty pages are NaN."""
        data = self.k_data if which == "k" else self.v_data
        shape = (self.pool_pages, self.num_kv_heads, self.page_size, self.head_dim)
        if self.dtype == "f32":
            out = np.full(shape, np.nan, dtype=np.float32)
        else:
            out = np.full(shape, BF16_NAN, dtype=np.uint16)
        has = self.page_row >= 0
        out[has] = data[self.page_row[has]]
        return out

    def request_pages(self, r: int, which: str) -> np.ndarray:
        """The P_r pages of request r, in logical order: [P, Hkv, b, d]."""
        data = self.k_data if which == "k" else self.v_data
        ids = self.page_table[r, : self.num_pages[r]]
        rows = self.page_row[ids]
        assert (rows >= 0).all()
        return data[rows]

    def kv_bytes_resident(self) -> int:
        e = 4 if self.dtype == "f32" else 2
        return int(self.seq_lens.sum()) * self.num_kv_heads * self.head_dim * e * 2


def _pages_and_resident(n: np.ndarray, budgets, b: int):
    P = -(-n // b)
    m = n.copy()
    if budgets is not None:
        over = n > budgets * b
        tail = np.where(n % b == 0, b, n % b)
        P = np.where(over, budgets, P)
        m = np.where(over, (budgets - 1) * b + tail, n)
    return P.astype(np.int32), m.astype(np.int32)


def _force_boundaries(rng, n: np.ndarray, n_boundary: int, b: int, lo: int) -> np.ndarray:
    """Put exactly n_boundary requests at a boundary (b | n) and no other."""
    n = n.copy()
    R = n.shape[0]
    chosen = np.zeros(R, dtype=bool)
    chosen[rng.choice(R, size=n_boundary, replace=False)] = True
    for r in range(R):
        if chosen[r]:
            n[r] -= n[r] % b
            if n[r] < max(lo, b):
                n[r] += b
        elif n[r] % b == 0:
            n[r] += 1
    return n


def _slow_rotary_dims(d: int, pairs: int) -> np.ndarray:
    """Dimensions of the slowest rotary pairs in the half-split rotary layout
    (pair i couples dims i and i + d/2; frequency falls with i)."""
    half = d // 2
    lo = np.arange(half - pairs, half)
    return np.concatenate([lo, lo + half])


def _build(*, name, seed, dtype, Hq, Hkv, d, n, budgets, free_pages, heavy_mode,
           heavy_frac, summary_mode, prefix_len=0, max_pages=None, pool_pages=None,
           pool_factor=None, extra_meta=None) -> Workload:
    b = PAGE
    R = int(n.shape[0])
    ss = np.random.SeedSequence(seed)
    (ss_layout, ss_q, ss_state, ss_prefix, ss_req) = ss.spawn(5)
    rng = np.random.default_rng(ss_layout)
    P, m = _pages_and_resident(n, budgets, b)
    prefix_pages = prefix_len // b
    assert prefix_len % b == 0
    if prefix_pages:
        assert (m >= prefix_len).all() and budgets is None
    private = P - prefix_pages
    used = prefix_pages + int(private.sum())
    if pool_pages is None:
        if pool_factor is not None:
            pool_pages = int(np.ceil(pool_factor * used))
        else:
            pool_pages = used + free_pages
    assert pool_pages >= used
    if max_pages is None:
        max_pages = int(P.max()) + 4
    perm = rng.permutation(pool_pages).astype(np.int32)
    page_table = np.full((R, max_pages), -1, dtype=np.int32)
    refcount = np.zeros(pool_pages, dtype=np.int32)
    shared_ids = perm[:prefix_pages]
    refcount[shared_ids] = R
    cursor = prefix_pages
    for r in range(R):
        page_table[r, :prefix_pages] = shared_ids
        ids = perm[cursor: cursor + private[r]]
        cursor += private[r]
        page_table[r, prefix_pages: P[r]] = ids
        refcount[ids] = 1
    free_list = np.zeros(pool_pages, dtype=np.int32)
    free = perm[cursor:]
    free_list[: free.shape[0]] = free
    free_count = int(free.shape[0])

    # content rows: shared prefix pages first, then each request's private pages
    page_row = np.full(pool_pages, -1, dtype=np.int32)
    page_row[perm[:used]] = np.arange(used, dtype=np.int32)
    store = np.float32 if dtype == "f32" else np.uint16
    k_data = np.empty((used, Hkv, b, d), dtype=store)
    v_data = np.empty((used, Hkv, b, d), dtype=store)

    # queries
    rq = np.random.default_rng(ss_q)
    q_post32 = rq.standard_normal((R, Hq, d), dtype=np.float32)
    q_pre32 = rq.standard_normal((R, Hq, d), dtype=np.float32)
    G = Hq // Hkv

    # per-request summary direction u[r, h] on slow rotary dims (used by "coin")
    rs = np.random.default_rng(ss_state)
    slow = _slow_rotary_dims(d, max(2, d // 16))
    u = np.zeros((R, Hkv, d), dtype=np.float64)
    u[:, :, slow] = rs.standard_normal((R, Hkv, slow.shape[0]))
    u /= np.linalg.norm(u, axis=-1, keepdims=True)

    if np.ndim(heavy_frac) == 1:
        heavy_frac_r = rs.choice(np.asarray(heavy_frac, dtype=np.float64), size=R)
    else:
        heavy_frac_r = np.full(R, float(heavy_frac))

    def finish_tokens(rr, K, V, first_slot, rng_r):
        """Apply heavy-token synthesis to logical K of tokens [first_slot, first_slot+len)."""
        T = K.shape[0]
        heavy = []
        for h in range(Hkv):
            if heavy_mode == "query":
                # 3 heavy slots inside the candidate region, scaled x4 along the
                # current query direction of the KV group
                C = int(max(P[rr] - 1, 0)) * b
                cnt = min(3, C)
                slots = np.sort(rng_r.choice(C, size=cnt, replace=False)) if cnt else np.zeros(0, int)
                qd = q_post32[rr, h * G:(h + 1) * G].astype(np.float64).sum(0)
                qd /= np.linalg.norm(qd)
                for s in slots:
                    c = float(K[s, h].astype(np.float64) @ qd)
                    K[s, h] = (K[s, h] + (4.0 * abs(c) - c) * qd).astype(np.float32)
                heavy.append(slots.astype(np.int32))
                continue
            cnt = int(round(heavy_frac_r[rr] * T))
            slots = np.sort(rng_r.choice(T, size=cnt, replace=False)) if cnt else np.zeros(0, int)
            if heavy_mode == "scaled":
                K[slots, h] *= np.float32(4.0)
            elif heavy_mode == "aligned":
                c = np.sqrt(15.0 * d)
                K[slots, h] = (K[slots, h] + c * u[rr, h]).astype(np.float32)
            heavy.append((slots + first_slot).astype(np.int32))
        return heavy

    def to_pages(K, npages):
        T = K.shape[0]
        full = np.full((npages * b, Hkv, d), np.nan, dtype=np.float32)
        full[:T] = K
        pages = full.reshape(npages, b, Hkv, d).transpose(0, 2, 1, 3)
        if dtype == "f32":
            return np.ascontiguousarray(pages)
        out = _to_bf16_bits(np.ascontiguousarray(pages))
        return out

    # shared prefix content (identical for every request)
    heavy_prefix = [np.zeros(0, np.int32)] * Hkv
    if prefix_pages:
        rp = np.random.default_rng(ss_prefix)
        Kp = rp.standard_normal((prefix_len, Hkv, d), dtype=np.float32)
        Vp = rp.standard_normal((prefix_len, Hkv, d), dtype=np.float32)
        heavy_prefix = finish_tokens(0, Kp, Vp, 0, rp)
        k_data[:prefix_pages] = to_pages(Kp, prefix_pages)
        v_data[:prefix_pages] = to_pages(Vp, prefix_pages)
        del Kp, Vp

    req_seeds = ss_req.spawn(R)
    row_start = np.concatenate([[prefix_pages], prefix_pages + np.cumsum(private)[:-1]]).astype(np.int64)
    heavy_all = [None] * R

    def one_request(rr):
        rng_r = np.random.default_rng(req_seeds[rr])
        T = int(m[rr]) - prefix_len
        K = rng_r.standard_normal((T, Hkv, d), dtype=np.float32)
        V = rng_r.standard_normal((T, Hkv, d), dtype=np.float32)
        hv = finish_tokens(rr, K, V, prefix_len, rng_r)
        if prefix_pages:
            hv = [np.concatenate([heavy_prefix[h], hv[h]]) for h in range(Hkv)]
        heavy_all[rr] = hv
        lo = row_start[rr]
        k_data[lo: lo + private[rr]] = to_pages(K, int(private[rr]))
        v_data[lo: lo + private[rr]] = to_pages(V, int(private[rr]))

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(one_request, range(R)))

    # query-summary pool: slots owned by no request stay NaN
    nslots = max(SLOTS, R)
    slot_ids = rs.permutation(nslots)[:R].astype(np.int32)
    qstate = np.full((nslots, 2, Hq, d), np.nan, dtype=np.float32)
    if summary_mode == "random":
        qstate[slot_ids] = rs.standard_normal((R, 2, Hq, d), dtype=np.float32)
    elif summary_mode == "coin":
        # one view points along u (the direction heavy keys follow), the other
        # does not; which one is a seeded coin per request
        coin = rs.integers(0, 2, size=R)
        for rr in range(R):
            for x in range(2):
                a = 3.0 if x == coin[rr] else 0.0
                for h in range(Hkv):
                    eps = rs.standard_normal((G, d))
                    qstate[slot_ids[rr], x, h * G:(h + 1) * G] = (
                        a * np.sqrt(d) * u[rr, h] + eps).astype(np.float32)
    elif summary_mode == "priors":
        pass
    else:
        raise ValueError(summary_mode)

    q_priors = None
    if summary_mode == "priors":
        q_priors = rs.standard_normal((8, R, Hq, d), dtype=np.float32)

    if dtype == "f32":
        q_post, q_pre = q_post32, q_pre32
    else:
        q_post, q_pre = _to_bf16_bits(q_post32), _to_bf16_bits(q_pre32)

    boundary = np.nonzero(m == P * b)[0].astype(np.int32)
    meta = dict(seed=seed, heavy_mode=heavy_mode, prefix_len=prefix_len)
    if extra_meta:
        meta.update(extra_meta)
    return Workload(
        name=name, dtype=dtype, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
        page_size=b, logical_lens=n.astype(np.int32),
        budgets=None if budgets is None else budgets.astype(np.int32),
        page_table=page_table, num_pages=P, seq_lens=m, positions=(n - 1).astype(np.int32),
        refcount=refcount, free_list=free_list, free_count=free_count, page_row=page_row,
        k_data=k_data, v_data=v_data, q_post=q_post, q_pre=q_pre, qstate=qstate,
        slot_ids=slot_ids, init=np.zeros(R, dtype=np.uint8), boundary=boundary,
        heavy=heavy_all, q_priors=q_priors, meta=meta)


# --------------------------------------------------------------------------
# The five workloads.  Defaults are the full sizes; keyword overrides give the
# reduced sizes that the oracle finishes in seconds.
# --------------------------------------------------------------------------

def tiny(seed: int = 1) -> Workload:
    """2 requests, 4 query / 2 KV heads, d = 64, fp32, logical lengths 48 and 80,
    budget 3 pages each (request 1 has compressed before), pool of 16 pages."""
    n = np.array([48, 80], dtype=np.int64)
    budgets = np.array([3, 3], dtype=np.int64)
    return _build(name="tiny_fp32", seed=seed, dtype="f32", Hq=4, Hkv=2, d=64, n=n,
                  budgets=budgets, free_pages=10, heavy_mode="query", heavy_frac=0.0,
                  summary_mode="priors", max_pages=6)


def qwen3_8b(seed: int = 2, num_reqs: int = 64, len_lo: int = 1024, len_hi: int = 8192,
             budget_choices=(64, 128, 256), boundary_frac: float = 1 / 16,
             free_pages: int = 200_000, heavy_frac: float = 0.01) -> Workload:
    """Qwen3-8B attention layer: 32 query / 8 KV heads, d = 128, bf16."""
    rng = np.random.default_rng([seed, 101])
    n = rng.integers(len_lo, len_hi + 1, size=num_reqs)
    budgets = rng.choice(np.asarray(budget_choices), size=num_reqs)
    n = _force_boundaries(rng, n, max(1, int(round(num_reqs * boundary_frac))), PAGE, len_lo)
    return _build(name="qwen3_8b_bf16", seed=seed, dtype="bf16", Hq=32, Hkv=8, d=128, n=n,
                  budgets=budgets, free_pages=free_pages, heavy_mode="scaled",
                  heavy_frac=heavy_frac, summary_mode="random",
                  extra_meta=dict(len_range=(len_lo, len_hi)))


def long_reasoning(seed: int = 3, num_reqs: int = 32, len_lo: int = 16384, len_hi: int = 32768,
                   heavy_fracs=(0.001, 0.01, 0.1), free_pages: int = 200_000) -> Workload:
    """Qwen3-8B heads, bf16, every request at a boundary, heavy fraction per request."""
    rng = np.random.default_rng([seed, 101])
    n = rng.integers(len_lo, len_hi + 1, size=num_reqs)
    n = np.maximum(n - n % PAGE, PAGE)
    return _build(name="long_reasoning_bf16", seed=seed, dtype="bf16", Hq=32, Hkv=8, d=128,
                  n=n, budgets=None, free_pages=free_pages, heavy_mode="aligned",
                  heavy_frac=np.asarray(heavy_fracs), summary_mode="coin")


def high_concurrency(seed: int = 4, num_reqs: int = 256, median: float = 2048, sigma: float = 0.8,
                     lo: int = 256, hi: int = 16384, boundary_frac: float = 1 / 8,
                     pool_factor: float = 1.1, heavy_frac: float = 0.01) -> Workload:
    """256 requests, lognormal lengths, pool = 1.1 x pages in use."""
    rng = np.random.default_rng([seed, 101])
    z = rng.standard_normal(num_reqs)
    n = np.clip(np.round(np.exp(np.log(median) + sigma * z)), lo, hi).astype(np.int64)
    n = _force_boundaries(rng, n, max(1, int(round(num_reqs * boundary_frac))), PAGE, lo)
    n = np.minimum(n, hi)
    return _build(name="high_concurrency_bf16", seed=seed, dtype="bf16", Hq=32, Hkv=8, d=128,
                  n=n, budgets=None, free_pages=0, pool_factor=pool_factor,
                  heavy_mode="scaled", heavy_frac=heavy_frac, summary_mode="random")


def prefix_shared(seed: int = 5, num_reqs: int = 128, prefix_len: int = 2048, tail_lo: int = 512,
                  tail_hi: int = 8192, boundary_frac: float = 1 / 16, num_q_heads: int = 64,
                  free_pages: int = 200_000, heavy_frac: float = 0.01) -> Workload:
    """Qwen3-32B attention layer (64 query / 8 KV heads), a refcounted shared prefix."""
    rng = np.random.default_rng([seed, 101])
    n = prefix_len + rng.integers(tail_lo, tail_hi + 1, size=num_reqs)
    n = _force_boundaries(rng, n, max(1, int(round(num_reqs * boundary_frac))), PAGE,
                          prefix_len + tail_lo)
    return _build(name="prefix_shared_bf16", seed=seed, dtype="bf16", Hq=num_q_heads, Hkv=8,
                  d=128, n=n, budgets=None, free_pages=free_pages, heavy_mode="scaled",
                  heavy_frac=heavy_frac, summary_mode="random", prefix_len=prefix_len)


CONFIGS = {
    "tiny": tiny,
    "qwen3_8b": qwen3_8b,
    "long_reasoning": long_reasoning,
    "high_concurrency": high_concurrency,
    "prefix_shared": prefix_shared,
}


def make(name: str, **kw) -> Workload:
    return CONFIGS[name](**kw)


def policy_draws(seed: int, n: int) -> np.ndarray:
    """Uniform float32 draws in [0, 1), one per boundary request, for the
    random capacity policy (the draw is an input to both implementations)."""
    return np.random.default_rng(seed).random(n, dtype=np.float32)


def layer_variant(w: Workload, layer: int) -> Workload:
    """The same batch seen at another attention layer: the page tables, lengths,
    positions and summary slots are shared by every layer, the contents differ.
    Layer 0 is ``w`` itself; layer l > 0 mixes each value of layer 0 with a
    fresh seeded N(0, 1) draw, 0.6 x + 0.8 z (unit variance, heavy keys stay
    somewhat heavy).  Empty slots and unowned summary slots stay NaN."""
    if layer == 0:
        return w
    rng = np.random.default_rng([int(w.meta.get("seed", 0)), 7919, layer])

    def mix(a, storage):
        x = a.astype(np.float32) if storage == "f32" else \
            (a.astype(np.uint32) << np.uint32(16)).view(np.float32)
        z = rng.standard_normal(x.shape, dtype=np.float32)
        y = (np.float32(0.6) * x + np.float32(0.8) * z).astype(np.float32)
        return y if storage == "f32" else _to_bf16_bits(y)

    st = w.dtype
    return dataclasses.replace(
        w, k_data=mix(w.k_data, st), v_data=mix(w.v_data, st), q_pre=mix(w.q_pre, st),
        q_post=mix(w.q_post, st), qstate=mix(w.qstate, "f32"), q_priors=None,
        meta=dict(w.meta, layer=layer))


def step_inputs(w: Workload, n_steps: int, seed: int = 0, n_layers: int = 1) -> list:
    """Per decode step, the new token of every request: its keys and values
    ([R, Hkv, d] per layer), pre- and post-RoPE queries ([R, Hq, d]), all
    seeded N(0, 1) in the workload's storage type.  The loop's synthetic
    continuation of the batch."""
    rng = np.random.default_rng([int(w.meta.get("seed", 0)), 104729, seed])
    R, Hq, Hkv, d = w.num_reqs, w.num_q_heads, w.num_kv_heads, w.head_dim

    def draw(shape):
        x = rng.standard_normal(shape, dtype=np.float32)
        return x if w.dtype == "f32" else _to_bf16_bits(x)

    out = []
    for _ in range(n_steps):
        out.append(dict(k_new=[draw((R, Hkv, d)) for _ in range(n_layers)],
                        v_new=[draw((R, Hkv, d)) for _ in range(n_layers)],
                        q_pre=draw((R, Hq, d)), q_post=draw((R, Hq, d))))
    return out

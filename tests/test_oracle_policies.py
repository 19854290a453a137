"""Pins of the oracle's capacity-policy variants and the entropy demand metric
(App., alternative capacity-control policies and the signal ablation):
closed forms of the entropy size, brute force of the shrink selection on tiny
inputs, the piecewise policy definitions on hand-made counts with exact Delta,
and the invariants of a shrink event.

Every test here runs on the CPU (no GPU marker)."""
import itertools
import math

import numpy as np
import pytest

import oracle as O
import workloads as W


# ----------------------------------------------------------- entropy size ----

def test_entropy_count_closed_forms():
    for n in (1, 2, 7, 100, 4093):
        assert O.entropy_count(np.full(n, 1.0 / n, np.float32)) == n
    one_hot = np.zeros(50, np.float32)
    one_hot[17] = 1.0
    assert O.entropy_count(one_hot) == 1
    # k equal weights among zeros: exp(H) = k
    for k in (3, 9, 31):
        a = np.zeros(64, np.float32)
        a[:k] = 1.0 / k
        assert O.entropy_count(a) == k
    # (1/2, 1/4, 1/4): H = 1.5 ln 2, exp(H) = 2^1.5 = 2.83 -> 3
    assert O.entropy_count(np.array([0.5, 0.25, 0.25], np.float32)) == 3
    # (0.9, 0.1): exp(H) = 0.9^-0.9 * 0.1^-0.1 = 1.384 -> 1
    assert O.entropy_count(np.array([0.9, 0.1], np.float32)) == 1
    assert math.isclose(0.9 ** -0.9 * 0.1 ** -0.1, 1.3841, rel_tol=1e-4)


def test_entropy_count_is_bounded_and_permutation_invariant():
    rng = np.random.default_rng(5)
    for _ in range(20):
        a = rng.dirichlet(np.full(200, 0.3)).astype(np.float32)
        k = O.entropy_count(a)
        assert 1 <= k <= a.size
        assert O.entropy_count(rng.permutation(a)) == k


# ------------------------------------------------------ shrink selection ----

def _key_order(s, idx):
    return sorted(idx, key=lambda i: (-float(s[i]), i))


def _brute_select_shrink(s, P, b, k_loc):
    """Shrink keeps K_t = (P - 3) b of the (P - 1) b candidates: among all
    size-K_t subsets that hold every block's top q (q = min(k_loc, K_t // (P-1))),
    the one whose other members are best under (score desc, slot asc)."""
    C = (P - 1) * b
    K_t = (P - 3) * b
    q = max(0, min(k_loc, K_t // (P - 1)))
    must = set()
    for j in range(P - 1):
        must |= set(_key_order(s, range(j * b, (j + 1) * b))[:q])
    best = None
    for S in itertools.combinations(range(C), K_t):
        if not must <= set(S):
            continue
        key = [(-float(s[i]), i) for i in _key_order(s, set(S) - must)]
        if best is None or key < best[0]:
            best = (key, S)
    return np.array(sorted(best[1]))


def test_shrink_selection_brute_force_small():
    rng = np.random.default_rng(21)
    for trial in range(30):
        b = 2
        P = int(rng.integers(3, 6))
        k_loc = int(rng.integers(0, 3))
        s = rng.choice([0.1, 0.2, 0.3, 0.7], size=(P - 1) * b).astype(np.float32)
        if trial % 2:
            s = rng.uniform(0, 1, (P - 1) * b).astype(np.float32)
        kept = O.select_retained(s, P, b, k_loc, drop=2)
        assert np.array_equal(kept, _brute_select_shrink(s, P, b, k_loc))


def test_shrink_compaction_layout():
    P, b = 5, 4
    toks = np.arange(P * b) * 10
    kept = np.array([1, 4, 6, 9, 10, 13, 14, 15])           # K_t = (P - 3) b = 8
    out = O.compact_tokens(toks, kept, P, b, drop=2)
    assert out[:8].tolist() == [10, 40, 60, 90, 100, 130, 140, 150]
    assert out[8:12].tolist() == [160, 170, 180, 190]        # the protected last page
    assert out[12:].tolist() == toks[12:].tolist()           # free slots keep their contents


# --------------------------------------------------------- policy choice ----

def _state(P_list, b=16, free=8, extra=0):
    """One request per entry, each exactly at a boundary with P pages; pages
    numbered consecutively, the rest on the free stack."""
    R = len(P_list)
    max_pages = max(P_list) + 2
    used = sum(P_list)
    pool = used + free + extra
    table = np.full((R, max_pages), -1, np.int32)
    nxt = 0
    for r, P in enumerate(P_list):
        table[r, :P] = np.arange(nxt, nxt + P)
        nxt += P
    refc = np.zeros(pool, np.int32)
    refc[:used] = 1
    fl = np.zeros(pool, np.int32)
    fl[:pool - used] = np.arange(used, pool)[::-1]
    return O.PageState(table, np.array(P_list, np.int32), np.array(P_list, np.int32) * b, refc, fl,
                       pool - used)


def _counts(ks, kl):
    return [np.array([[[a, c]]]) for a, c in zip(ks, kl)]


def test_policy_definitions_on_exact_trends():
    b = 16
    # P = 6: |C| = 80, one head, one layer -> Delta = (kS - kL) / 80
    ks, kl = [10, 10, 11], [11, 10, 10]                       # Delta = -1/80, 0, +1/80
    cases = {
        "growpage": [O.COMPRESS, O.COMPRESS, O.GROW],
        "inverse": [O.GROW, O.GROW, O.COMPRESS],
        "shrink": [O.SHRINK, O.COMPRESS, O.GROW],
    }
    for policy, want in cases.items():
        st = _state([6, 6, 6])
        p = O.Params(policy=policy, min_capacity_pages=4).as_f32(128)
        dec, delta = O.decide_and_allocate(st, [0, 1, 2], _counts(ks, kl), b, p)
        assert dec.tolist() == want, policy
        assert delta.tolist() == [np.float32(-1 / 80), 0.0, np.float32(1 / 80)]
    # shrink's middle band: -0.005 <= Delta <= 0 compresses (P = 21: Delta = -1/320)
    st = _state([21])
    p = O.Params(policy="shrink", min_capacity_pages=4).as_f32(128)
    assert O.decide_and_allocate(st, [0], _counts([10], [11]), b, p)[0].tolist() == [O.COMPRESS]
    # below the minimum capacity a shrink becomes a compression
    st = _state([6])
    p = O.Params(policy="shrink", min_capacity_pages=6).as_f32(128)
    assert O.decide_and_allocate(st, [0], _counts([10], [11]), b, p)[0].tolist() == [O.COMPRESS]


def test_fixed_and_random_policies():
    b = 16
    st = _state([6, 8, 9])
    p = O.Params(policy="fixed", fixed_pages=8).as_f32(128)
    dec, _ = O.decide_and_allocate(st, [0, 1, 2], _counts([1, 1, 1], [90, 90, 90]), b, p)
    assert dec.tolist() == [O.GROW, O.COMPRESS, O.COMPRESS]   # trend ignored
    st = _state([6, 6, 6, 6])
    p = O.Params(policy="random").as_f32(128)
    draws = np.array([0.0, 0.69, 0.7, 0.999], np.float32)
    dec, _ = O.decide_and_allocate(st, [0, 1, 2, 3], _counts([5] * 4, [5] * 4), b, p, draws)
    assert dec.tolist() == [O.COMPRESS, O.COMPRESS, O.GROW, O.GROW]


def test_shrink_releases_the_last_page():
    b = 16
    st = _state([6, 7], free=3)
    before = st.copy()
    p = O.Params(policy="shrink", min_capacity_pages=4).as_f32(128)
    dec, _ = O.decide_and_allocate(st, [0, 1], _counts([10, 10], [20, 10]), b, p)
    assert dec.tolist() == [O.SHRINK, O.COMPRESS]
    last = int(before.page_table[0, 5])
    assert st.num_pages.tolist() == [5, 7] and st.seq_lens.tolist() == [4 * b, 6 * b]
    assert st.page_table[0, 5] == -1 and st.refcount[last] == 0
    assert st.free_count == before.free_count + 1 and st.free_list[st.free_count - 1] == last


# ----------------------------------------------------------- shrink event ----

def test_shrink_event_invariants():
    w = W._build(name="shrink_f32", seed=41, dtype="f32", Hq=4, Hkv=2, d=64,
                 n=np.array([96, 160, 100]), budgets=None, free_pages=6, heavy_mode="scaled",
                 heavy_frac=0.05, summary_mode="random")
    b = w.page_size
    k0, v0 = w.dense_pool("k"), w.dense_pool("v")
    k, v = k0.copy(), v0.copy()
    st = O.PageState(w.page_table.copy(), w.num_pages.copy(), w.seq_lens.copy(), w.refcount.copy(),
                     w.free_list.copy(), w.free_count)
    # threshold +inf for "grow" and a threshold above every trend make every
    # boundary request shrink
    p = O.Params(policy="shrink", tau=math.inf, shrink_threshold=10.0, min_capacity_pages=2)
    res = O.boundary_step([(k, v)], w.dtype, st, w.q_pre, w.qstate, w.slot_ids, w.positions,
                          w.boundary, p)
    assert len(w.boundary) >= 1
    for i, r in enumerate(w.boundary):
        P = int(w.num_pages[r])
        assert res["decisions"][i] == O.SHRINK
        assert st.num_pages[r] == P - 1 and st.seq_lens[r] == (P - 2) * b
        released = int(w.page_table[r, P - 1])
        assert st.refcount[released] == 0 and released in st.free_list[: st.free_count].tolist()
        assert np.array_equal(k[released], k0[released])        # released, not written
        for pool0, pool in ((k0, k), (v0, v)):
            before = O.gather_tokens(pool0, w.page_table[r], P * b, b)
            after = O.gather_tokens(pool, st.page_table[r], (P - 1) * b, b)
            for h in range(w.num_kv_heads):
                kept = res["kept"][(i, 0, h)]
                K_t = (P - 3) * b
                assert kept.size == K_t
                assert np.array_equal(after[:K_t, h], before[kept, h])
                assert np.array_equal(after[K_t:(P - 2) * b, h], before[(P - 1) * b:, h])
    assert res["counters"].tolist()[O.COMPRESS] == len(w.boundary)
    # every page is either held or free, once
    held = set()
    for r in range(w.num_reqs):
        held |= set(st.page_table[r, : st.num_pages[r]].tolist())
    free = set(st.free_list[: st.free_count].tolist())
    assert not (held & free) and held | free == set(range(w.pool_pages))


def test_params_reject_unknown_policy():
    st = _state([6])
    with pytest.raises(ValueError):
        O.decide_and_allocate(st, [0], _counts([1], [2]), 16, O.Params(policy="sometimes"))

"""Pins of the CPU oracle against facts that do not come from the oracle itself:
closed forms, brute force on tiny inputs, invariants the paper's definitions
imply, library routines, and hand-worked examples under tests/golden/.

Every test here runs on the CPU (no GPU marker)."""
import itertools
import json
import math
from fractions import Fraction
import os

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- storage ----

def test_bf16_widen_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(10000) * 10.0 ** rng.integers(-6, 6, 10000)).astype(np.float32)
    t = torch.from_numpy(x).to(torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.widen(bits, "bf16"), t.to(torch.float64).numpy())


def test_bf16_narrow_is_nearest_even():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000) * 10.0 ** rng.integers(-5, 5, 20000)
    bits = O.narrow(x, "bf16")
    y = O.widen(bits, "bf16")
    # neighbours one bf16 step away on each side are never closer
    up = O.widen((bits.astype(np.int32) + 1).astype(np.uint16), "bf16")
    dn = O.widen((bits.astype(np.int32) - 1).astype(np.uint16), "bf16")
    err = np.abs(y - x)
    assert (err <= np.abs(up - x)).all() and (err <= np.abs(dn - x)).all()
    # float32-representable inputs: same as torch's round-to-nearest-even
    x32 = x.astype(np.float32)
    tb = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.narrow(x32.astype(np.float64), "bf16"), tb)


# ------------------------------------------------------------ attention ----

def test_p1_softmax_rows_sum_to_one():
    rng = np.random.default_rng(2)
    for scale in (1.0, 30.0, 300.0):
        z = rng.standard_normal(1000) * scale
        a = O.softmax(z)
        assert abs(a.sum() - 1.0) <= 1e-12 and (a >= 0).all()


def test_p2_paged_equals_unpaged_and_page_ids_do_not_matter():
    rng = np.random.default_rng(3)
    b, Hkv, d, G = 16, 2, 8, 3
    m = 53
    K = rng.standard_normal((m, Hkv, d)).astype(np.float32)
    V = rng.standard_normal((m, Hkv, d)).astype(np.float32)
    q = rng.standard_normal((1, Hkv * G, d)).astype(np.float32)
    P = 4
    for trial in range(3):
        ids = rng.permutation(10)[:P]
        pool_k = np.full((10, Hkv, b, d), np.nan, np.float32)
        pool_v = np.full((10, Hkv, b, d), np.nan, np.float32)
        for j in range(P):
            lo, hi = j * b, min(m, (j + 1) * b)
            pool_k[ids[j], :, : hi - lo] = K[lo:hi].transpose(1, 0, 2)
            pool_v[ids[j], :, : hi - lo] = V[lo:hi].transpose(1, 0, 2)
        table = np.full((1, 6), -1, np.int32)
        table[0, :P] = ids
        out = O.decode_attention(pool_k, pool_v, "f32", table, np.array([m]), q, Hkv * G, 0.3)
        for g in range(Hkv * G):
            ref, _ = O.attention(q[0, g].astype(np.float64), K[:, g // G].astype(np.float64),
                                 V[:, g // G].astype(np.float64), 0.3)
            assert np.array_equal(out[0, g], ref)


def test_p3_closed_forms():
    rng = np.random.default_rng(4)
    d = 16
    v = rng.standard_normal((5, d))
    k = rng.standard_normal((5, d))
    q = rng.standard_normal(d)
    o, a = O.attention(q, k[:1], v[:1], 0.25)
    assert np.array_equal(o, v[0]) and a[0] == 1.0
    o, _ = O.attention(q, np.repeat(k[:1], 5, 0), v, 0.25)
    assert np.allclose(o, v.mean(0), rtol=0, atol=1e-15)
    o, _ = O.attention(np.zeros(d), k, v, 0.25)
    assert np.allclose(o, v.mean(0), rtol=0, atol=1e-15)


def test_p4_worst_case_error_is_tight_and_an_upper_bound():
    rng = np.random.default_rng(5)
    N, d, vmax = 12, 6, 2.5
    for _ in range(20):
        a = O.softmax(rng.standard_normal(N) * 2)
        S = np.sort(rng.choice(N, size=rng.integers(1, N), replace=False))
        u = rng.standard_normal(d)
        u /= np.linalg.norm(u)
        V = np.where(np.isin(np.arange(N), S)[:, None], -vmax * u, vmax * u)
        o = a @ V
        err = np.linalg.norm(o - O.renormalised_subset_output(a, V, S))
        assert abs(err - O.worst_case_error(a, S, vmax)) <= 1e-12
        for _ in range(5):
            Vr = rng.standard_normal((N, d))
            Vr *= (vmax * rng.uniform(0, 1, N) / np.linalg.norm(Vr, axis=1))[:, None]
            e = np.linalg.norm(a @ Vr - O.renormalised_subset_output(a, Vr, S))
            assert e <= O.worst_case_error(a, S, vmax) + 1e-12


def test_p4_attention_over_kept_subset_is_renormalised_output():
    rng = np.random.default_rng(6)
    N, d = 40, 8
    K, V, q = rng.standard_normal((N, d)), rng.standard_normal((N, d)), rng.standard_normal(d)
    _, a = O.attention(q, K, V, 0.4)
    S = np.sort(rng.choice(N, 17, replace=False))
    o_sub, _ = O.attention(q, K[S], V[S], 0.4)
    assert np.allclose(o_sub, O.renormalised_subset_output(a, V, S), rtol=0, atol=1e-14)


# ------------------------------------------------------------- top-p / D_p ----

def _brute_min_subset(a, p):
    N = len(a)
    for k in range(1, N + 1):
        for S in itertools.combinations(range(N), k):
            if sum(float(a[i]) for i in S) >= p:
                return k
    return N


def test_p5_top_p_count_equals_brute_force():
    rng = np.random.default_rng(7)
    for N in range(1, 11):
        for _ in range(6):
            a = O.softmax(rng.standard_normal(N) * rng.uniform(0.1, 4)).astype(np.float32)
            for p in (0.3, 0.5, 0.9, 0.99):
                assert O.top_p_count(a, p) == _brute_min_subset(a.astype(np.float64), p)


def test_p5_top_p_special_cases():
    one_hot = np.zeros(50, np.float32)
    one_hot[17] = 1.0
    assert O.top_p_count(one_hot, 0.99) == 1
    for N in (7, 10, 33, 1000):
        uni = np.full(N, 1.0 / N)
        p = 0.99
        if math.isclose(p * N, round(p * N)):
            continue
        assert O.top_p_count(uni, p) == math.ceil(p * N)


def test_p5_theorem_capacity_equals_demand():
    """C^wc_delta = D_{1 - delta / (2 Vmax)} (Sec. 3.1, theorem), with C^wc found by
    brute force over subsets using the exact worst-case error."""
    rng = np.random.default_rng(8)
    vmax = 1.5
    for _ in range(10):
        N = int(rng.integers(2, 9))
        a = O.softmax(rng.standard_normal(N) * 2)
        delta = float(rng.uniform(0.05, 2.9))
        best = N
        for k in range(1, N + 1):
            if any(O.worst_case_error(a, list(S), vmax) <= delta
                   for S in itertools.combinations(range(N), k)):
                best = k
                break
        p = 1.0 - delta / (2 * vmax)
        assert best == _brute_min_subset(a, p)
        # the float32 form used at boundaries agrees away from rounding ties
        if not O.top_p_fragile(a.astype(np.float32), p, 1e-6):
            assert O.top_p_count(a.astype(np.float32), p) == best


def test_golden_top_p():
    g = _golden("top_p_worked.json")
    for case in g["cases"]:
        assert O.top_p_count(np.array(case["a"], np.float32), case["p"]) == case["K"]


# ------------------------------------------------------------- summaries ----

def test_p6_ema_closed_form_and_special_cases():
    rng = np.random.default_rng(9)
    Hq, d, n = 2, 8, 12
    qs = rng.standard_normal((n, 1, Hq, d)).astype(np.float32)
    st = np.full((4, 2, Hq, d), np.nan, np.float32)
    slot = np.array([2])
    for t in range(n):
        st = O.update_summaries(qs[t], "f32", slot, np.array([t == 0], np.uint8), st, 0.9, 0.999)
    for x, beta in enumerate((0.9, 0.999)):
        closed = beta ** (n - 1) * qs[0, 0].astype(np.float64)
        for j in range(1, n):
            closed += (1 - beta) * beta ** (n - 1 - j) * qs[j, 0]
        assert np.allclose(st[2, x], closed, rtol=1e-5, atol=1e-6)
    assert np.isnan(st[[0, 1, 3]]).all()            # other slots untouched
    # beta = 0 reduces to the current query
    st0 = O.update_summaries(qs[5], "f32", slot, np.array([0], np.uint8), st, 0.0, 0.0)
    assert np.array_equal(st0[2, 0], qs[5, 0]) and np.array_equal(st0[2, 1], qs[5, 0])
    # a constant query is a fixed point
    c = np.full((1, Hq, d), 0.625, np.float32)
    stc = O.update_summaries(c, "f32", slot, np.array([1], np.uint8), st, 0.9, 0.999)
    for _ in range(5):
        stc = O.update_summaries(c, "f32", slot, np.array([0], np.uint8), stc, 0.9, 0.999)
    assert np.array_equal(stc[2], np.full((2, Hq, d), 0.625, np.float32))


def test_p6_init_overwrites_a_poisoned_slot():
    st = np.full((3, 2, 1, 4), np.nan, np.float32)
    q = np.array([[[1.0, -2.0, 3.0, 0.5]]], np.float32)
    out = O.update_summaries(q, "f32", np.array([1]), np.array([1], np.uint8), st, 0.9, 0.999)
    assert np.array_equal(out[1, 0], q[0]) and np.array_equal(out[1, 1], q[0])


# ---------------------------------------------------- calibration / RoPE ----

def test_p7_calibration_matches_rms():
    rng = np.random.default_rng(10)
    for _ in range(10):
        qt, qb = rng.standard_normal(64) * 3, rng.standard_normal(64) * 0.01
        assert math.isclose(O.rms(O.calibrate(qt, qb)), O.rms(qt), rel_tol=1e-13)
    assert (O.calibrate(np.ones(4), np.zeros(4)) == 0).all()


def test_p7_rope_properties():
    rng = np.random.default_rng(11)
    d, theta = 64, 1e6
    x, y = rng.standard_normal(d), rng.standard_normal(d)
    assert np.array_equal(O.rope(x, 0, theta), x)
    for pos in (1, 77, 32767):
        assert math.isclose(np.linalg.norm(O.rope(x, pos, theta)), np.linalg.norm(x), rel_tol=1e-13)
    d1 = O.rope(x, 100, theta) @ O.rope(y, 40, theta)
    d2 = O.rope(x, 1060, theta) @ O.rope(y, 1000, theta)
    assert math.isclose(d1, d2, rel_tol=1e-10, abs_tol=1e-10)
    assert np.allclose(O.rope(O.rope(x, 300, theta), 700, theta), O.rope(x, 1000, theta), atol=1e-12)
    # one rotary pair rotates by the position itself (frequency theta^0 = 1)
    assert np.allclose(O.rope(np.array([1.0, 0.0]), 0.5, theta), [math.cos(0.5), math.sin(0.5)])
    # half-split pairing: dims i and i + d/2 rotate together at theta^(-2i/d)
    e = np.zeros(8)
    e[1] = 1.0
    r = O.rope(e, 3, 10.0)
    ang = 3 * 10.0 ** (-2 / 8)
    assert np.allclose(r[[1, 5]], [math.cos(ang), math.sin(ang)]) and abs(r).sum() - abs(r[[1, 5]]).sum() < 1e-15


# -------------------------------------------------------------- decision ----

def _tiny_state(w):
    return O.PageState(w.page_table.copy(), w.num_pages.copy(), w.seq_lens.copy(),
                       w.refcount.copy(), w.free_list.copy(), w.free_count)


def _tiny_run(w, params, state=None, qstate=None):
    k, v = w.dense_pool("k"), w.dense_pool("v")
    qs = w.qstate if qstate is None else qstate
    st = _tiny_state(w) if state is None else state
    res = O.boundary_step([(k, v)], w.dtype, st, w.q_pre, qs, w.slot_ids, w.positions,
                          w.boundary, params)
    return res, st, k, v


def _tiny_summaries(w):
    st = w.qstate
    for j in range(w.q_priors.shape[0]):
        st = O.update_summaries(w.q_priors[j], "f32", w.slot_ids,
                                np.full(w.num_reqs, j == 0, np.uint8), st, 0.9, 0.999)
    return O.update_summaries(w.q_pre, "f32", w.slot_ids, np.zeros(w.num_reqs, np.uint8),
                              st, 0.9, 0.999)


def test_p8_equal_summaries_give_zero_trend_and_compress():
    w = W.tiny()
    qs = w.qstate.copy()
    for s in w.slot_ids:
        qs[s, 0] = qs[s, 1] = np.arange(w.num_q_heads * w.head_dim, dtype=np.float32).reshape(
            w.num_q_heads, w.head_dim) % 7 - 3
    res, st, _, _ = _tiny_run(w, O.Params(), qstate=qs)
    for c in res["counts"]:
        assert np.array_equal(c[..., 0], c[..., 1])
    assert (res["delta"] == 0).all() and (res["decisions"] == O.COMPRESS).all()


def test_p8_threshold_extremes_force_the_branch():
    w = W.tiny()
    qs = _tiny_summaries(w)
    res, st, _, _ = _tiny_run(w, O.Params(tau=-math.inf), qstate=qs)
    assert (res["decisions"] == O.GROW).all()
    res, st, _, _ = _tiny_run(w, O.Params(tau=math.inf), qstate=qs)
    assert (res["decisions"] == O.COMPRESS).all()


def test_demand_trend_is_exact():
    assert O.demand_trend([[3, 5]], [[4, 4]], 7) == 0
    assert O.demand_trend([[2]], [[1]], 32) == Fraction(1, 32)


# ------------------------------------------------------------- selection ----

def _key_order(s, idx):
    return sorted(idx, key=lambda i: (-float(s[i]), i))


def _brute_select(s, P, b, k_loc):
    """Among all size-K_t subsets of C that hold every block's top-q_loc, the one
    whose members are best under (score desc, slot asc) compared greedily."""
    C = (P - 1) * b
    K_t = (P - 2) * b
    q = O.local_quota(P, b, k_loc)
    must = set()
    for j in range(P - 1):
        must |= set(_key_order(s, range(j * b, (j + 1) * b))[:q])
    best = None
    for S in itertools.combinations(range(C), K_t):
        if not must <= set(S):
            continue
        key = [(-float(s[i]), i) for i in sorted(set(S) - must, key=lambda i: (-float(s[i]), i))]
        if best is None or key < best[0]:
            best = (key, S)
    return np.array(sorted(best[1]))


def test_p9_selection_brute_force_small():
    rng = np.random.default_rng(12)
    for trial in range(40):
        b = 4
        P = int(rng.integers(2, 5))
        k_loc = int(rng.integers(0, 4))
        s = rng.choice([0.1, 0.2, 0.3, 0.05, 0.7], size=(P - 1) * b).astype(np.float32)
        if trial % 2:
            s = rng.uniform(0, 1, (P - 1) * b).astype(np.float32)
        kept = O.select_retained(s, P, b, k_loc)
        assert np.array_equal(kept, _brute_select(s, P, b, k_loc))


def test_p9_selection_invariants():
    rng = np.random.default_rng(13)
    b = 16
    for P in (2, 3, 4, 9, 40):
        s = rng.uniform(0, 1, (P - 1) * b).astype(np.float32)
        s[rng.choice(s.size, s.size // 3)] = 0.25            # many ties
        for k_loc in (0, 4, 16):
            kept = O.select_retained(s, P, b, k_loc)
            assert kept.size == (P - 2) * b and np.unique(kept).size == kept.size
            q = O.local_quota(P, b, k_loc)
            loc = set()
            for j in range(P - 1):
                top = _key_order(s, range(j * b, (j + 1) * b))[:q]
                loc |= set(top)
                assert set(top) <= set(kept)
            # exchange: no evicted token outranks a kept token outside the local picks
            ev = set(range((P - 1) * b)) - set(kept)
            kept_glob = set(kept) - loc
            if kept_glob:
                worst = max(kept_glob, key=lambda i: (-float(s[i]), i))
                for e in ev:
                    assert (-float(s[e]), e) > (-float(s[worst]), worst)


def test_golden_selection():
    g = _golden("selection_worked.json")
    for case in g["cases"]:
        kept = O.select_retained(np.array(case["scores"], np.float32), case["P"], case["b"],
                                 case["k_loc"])
        assert kept.tolist() == case["kept"]
        toks = np.arange(case["P"] * case["b"])
        comp = O.compact_tokens(toks, kept, case["P"], case["b"])
        assert comp[: (case["P"] - 1) * case["b"]].tolist() == case["compacted"]


# ----------------------------------------------------- boundary events ----

def _pool_consistency(st: O.PageState, pool_pages: int):
    refs = np.zeros(pool_pages, np.int64)
    for r in range(st.num_pages.shape[0]):
        row = st.page_table[r, : st.num_pages[r]]
        assert (row >= 0).all() and np.unique(row).size == row.size
        np.add.at(refs, row, 1)
        assert (st.page_table[r, st.num_pages[r]:] == -1).all()
    assert np.array_equal(refs, st.refcount)
    free = st.free_list[: st.free_count]
    assert np.unique(free).size == free.size
    assert not (set(free.tolist()) & set(np.nonzero(st.refcount > 0)[0].tolist()))
    assert set(free.tolist()) | set(np.nonzero(st.refcount > 0)[0].tolist()) == set(range(pool_pages))


def test_p10_p12_compress_invariants_tiny():
    w = W.tiny()
    qs = _tiny_summaries(w)
    k0, v0 = w.dense_pool("k"), w.dense_pool("v")
    res, st, k, v = _tiny_run(w, O.Params(tau=math.inf), qstate=qs)
    b = w.page_size
    for i, r in enumerate(w.boundary):
        P = int(w.num_pages[r])
        assert res["decisions"][i] == O.COMPRESS
        assert st.seq_lens[r] == (P - 1) * b and st.num_pages[r] == P
        assert np.array_equal(st.page_table[r], w.page_table[r])
        for pool0, pool in ((k0, k), (v0, v)):
            before = O.gather_tokens(pool0, w.page_table[r], P * b, b)
            after = O.gather_tokens(pool, st.page_table[r], P * b, b)
            for h in range(w.num_kv_heads):
                kept = res["kept"][(i, 0, h)]
                K_t = (P - 2) * b
                assert kept.size == K_t
                assert np.array_equal(after[:K_t, h], before[kept, h])
                assert np.array_equal(after[K_t:(P - 1) * b, h], before[(P - 1) * b:, h])
    _pool_consistency(st, w.pool_pages)


def test_p11_grow_invariants_tiny():
    w = W.tiny()
    qs = _tiny_summaries(w)
    k0 = w.dense_pool("k")
    res, st, k, v = _tiny_run(w, O.Params(tau=-math.inf), qstate=qs)
    top = list(w.free_list[: w.free_count][::-1])
    for i, r in enumerate(w.boundary):
        P = int(w.num_pages[r])
        assert res["decisions"][i] == O.GROW
        assert st.num_pages[r] == P + 1 and st.seq_lens[r] == w.seq_lens[r]
        assert st.page_table[r, P] == top[i] and st.refcount[top[i]] == 1
    assert st.free_count == w.free_count - len(w.boundary)
    assert np.array_equal(np.nan_to_num(k, nan=7.0), np.nan_to_num(k0, nan=7.0))
    _pool_consistency(st, w.pool_pages)


def test_p13_fallback_when_no_page_is_free():
    w = W.tiny()
    qs = _tiny_summaries(w)
    st = _tiny_state(w)
    st.free_count = 0
    # pages that are no longer on the stack count as owned elsewhere for this test
    res, st2, _, _ = _tiny_run(w, O.Params(tau=-math.inf), state=st, qstate=qs)
    assert (res["decisions"] == O.FALLBACK).all()
    assert (st2.num_pages[w.boundary] == w.num_pages[w.boundary]).all()
    st = _tiny_state(w)
    st.free_count = 1
    res, st3, _, _ = _tiny_run(w, O.Params(tau=-math.inf), state=st, qstate=qs)
    assert res["decisions"].tolist() == [O.GROW, O.FALLBACK]


def test_prefix_sharing_never_writes_shared_pages():
    w = W.prefix_shared(num_reqs=4, prefix_len=32, tail_lo=20, tail_hi=90, free_pages=40,
                        boundary_frac=0.5)
    k0, v0 = w.dense_pool("k"), w.dense_pool("v")
    k, v = k0.copy(), v0.copy()
    st = _tiny_state(w)
    p = O.Params(tau=math.inf)
    res = O.boundary_step([(k, v)], w.dtype, st, w.q_pre, w.qstate, w.slot_ids, w.positions,
                          w.boundary, p)
    shared = np.nonzero(w.refcount > 1)[0]
    assert shared.size == 2
    assert np.array_equal(k[shared], k0[shared]) and np.array_equal(v[shared], v0[shared])
    for i, r in enumerate(w.boundary):
        assert res["decisions"][i] == O.COMPRESS
        assert not (set(st.page_table[r, : st.num_pages[r]].tolist()) & set(shared.tolist()))
    assert (st.refcount[shared] == w.num_reqs - len(w.boundary)).all()
    _pool_consistency(st, w.pool_pages)
    # not enough free pages for the replacements: preempt, state untouched
    st = _tiny_state(w)
    st.free_count = 1
    before = st.copy()
    res = O.boundary_step([(k0.copy(), v0.copy())], w.dtype, st, w.q_pre, w.qstate, w.slot_ids,
                          w.positions, w.boundary, p)
    assert (res["decisions"] == O.PREEMPT).all()
    assert np.array_equal(st.page_table, before.page_table) and st.free_count == 1


def test_not_boundary_is_reported_and_untouched():
    w = W.qwen3_8b(num_reqs=6, len_lo=40, len_hi=120, budget_choices=(3, 5), free_pages=10)
    nb = np.array([r for r in range(6) if r not in set(w.boundary.tolist())][:1], np.int32)
    st = _tiny_state(w)
    res = O.boundary_step([(w.dense_pool("k"), w.dense_pool("v"))], w.dtype, st, w.q_pre,
                          w.qstate, w.slot_ids, w.positions, nb, O.Params())
    assert res["decisions"].tolist() == [O.NOT_BOUNDARY]
    assert np.array_equal(st.seq_lens, w.seq_lens)


# ------------------------------------------------ library-routine pins ----

def test_decode_attention_matches_torch_sdpa():
    """Paged decode attention equals torch's scaled_dot_product_attention on the
    gathered keys/values (fp64, CPU), with grouped-query heads expanded."""
    w = W.qwen3_8b(seed=3, num_reqs=3, len_lo=40, len_hi=200, budget_choices=(4, 16), free_pages=5)
    scale = 1.0 / math.sqrt(w.head_dim)
    kp, vp = w.dense_pool("k"), w.dense_pool("v")
    out = O.decode_attention(kp, vp, "bf16", w.page_table, w.seq_lens, w.q_post, w.num_q_heads, scale)
    G = w.num_q_heads // w.num_kv_heads
    for r in range(w.num_reqs):
        m = int(w.seq_lens[r])
        K = torch.from_numpy(O.widen(O.gather_tokens(kp, w.page_table[r], m, 16), "bf16"))
        V = torch.from_numpy(O.widen(O.gather_tokens(vp, w.page_table[r], m, 16), "bf16"))
        q = torch.from_numpy(O.widen(w.q_post[r], "bf16"))               # [Hq, d]
        Kx = K.permute(1, 0, 2).repeat_interleave(G, 0)                  # [Hq, m, d]
        Vx = V.permute(1, 0, 2).repeat_interleave(G, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(q[:, None, :], Kx, Vx, scale=scale)[:, 0]
        assert np.allclose(out[r], ref.numpy(), rtol=0, atol=1e-12)


def test_view_distributions_special_case_is_softmax():
    """At position 0 (no rotation) with both summaries equal to the current query
    (unit calibration), each view is the mean over the G query heads of
    torch.softmax of the scaled key products."""
    rng = np.random.default_rng(14)
    C, Hkv, G, d = 50, 2, 3, 16
    K = rng.standard_normal((C, Hkv, d))
    qt = rng.standard_normal((Hkv * G, d))
    a = O.view_distributions(K, qt, qt, qt, 0, 1e6, 0.25)
    for h in range(Hkv):
        ref = torch.stack([torch.softmax(0.25 * torch.from_numpy(K[:, h]) @ torch.from_numpy(qt[h * G + g]), 0)
                           for g in range(G)]).mean(0).numpy()
        assert np.allclose(a[0, h], ref, rtol=0, atol=1e-15) and np.allclose(a[1, h], ref, rtol=0, atol=1e-15)


def test_cpu_baseline_child_runs_the_oracle_on_worker_processes():
    """The benchmark's all-core CPU leg: a GPU-free child process that forks
    workers running the oracle's decode attention over the tiny workload."""
    import json
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    cp = subprocess.run([sys.executable, "-m", "oracle.cpu_baseline", "tiny", "0.3", "2"], cwd=root,
                        capture_output=True, text=True, timeout=120)
    assert cp.returncode == 0, cp.stderr[-500:]
    res = json.loads(cp.stdout.strip().splitlines()[-1])
    assert res["workers"] == 2 and res["passes"] >= 2 and res["bytes"] > 0 and res["seconds"] > 0


# ------------------------------------------- token scores and fragility ----

def test_golden_token_scores():
    """s = max(a^S, a^L) per KV head (Sec. 3.3, token-score equation) through
    the whole scoring of one request: keys built so that each view's softmax is
    a hand-chosen distribution (tests/golden/token_score_worked.json)."""
    g = _golden("token_score_worked.json")
    b, P = g["b"], g["P"]
    heads = g["heads"]
    Hkv = len(heads)
    C = (P - 1) * b
    tokens = np.zeros((P * b, Hkv, 2), np.float32)
    for h, hd in enumerate(heads):
        tokens[:C, h] = np.array(hd["keys"], np.float32)
    tokens[C:] = 0.0                                       # the protected page is not scored
    q_t = np.tile(np.float32([1.0, 0.0]), (Hkv, 1))          # [Hq = Hkv, d]
    qbar = np.zeros((2, Hkv, 2), np.float32)
    qbar[0, :, 0] = 1.0                                    # short summary (1, 0)
    qbar[1, :, 1] = 1.0                                    # long summary (0, 1)
    params = O.Params(p=0.85, scale=1.0)
    counts, scores, a32 = O.score_request(tokens, "f32", P, b, q_t, qbar, 0, params, 1.0)
    for h, hd in enumerate(heads):
        np.testing.assert_allclose(a32[0, h], hd["a_s"], rtol=1e-6, atol=0)
        np.testing.assert_allclose(a32[1, h], hd["a_l"], rtol=1e-6, atol=0)
        np.testing.assert_allclose(scores[h], hd["scores"], rtol=1e-6, atol=0)
    # the direct form on the golden weights
    for hd in heads:
        s = O.token_scores(np.float32(hd["a_s"]), np.float32(hd["a_l"]))
        np.testing.assert_array_equal(s, np.float32(hd["scores"]))


def test_golden_top_p_fragile():
    """Fragility of the top-p size at the 1e-6 band, just inside and just
    outside it on either side of the K-th and (K-1)-th running sums
    (tests/golden/top_p_fragile_worked.json)."""
    g = _golden("top_p_fragile_worked.json")
    a = np.float32(g["a"])
    for case in g["cases"]:
        assert O.top_p_count(a, case["p"]) == case["K"], case
        assert O.top_p_fragile(a, case["p"], g["eps"]) == case["fragile"], case
        # order of the weights does not matter
        assert O.top_p_fragile(a[::-1].copy(), case["p"], g["eps"]) == case["fragile"], case


def test_golden_entropy_fragile():
    """Fragility of the entropy size: exp(H) within 1e-6 (relative) of a rounding
    midpoint, tested at 1.5 +- 5e-7 (inside) and 1.5 +- 2e-6 (outside), plus
    integer and far-from-midpoint cases (tests/golden/entropy_fragile_worked.json).
    The golden's own claims are checked too: its q solves the binary-entropy
    closed form, and scipy's entropy of each vector is the exp(H) the file
    states (the normalisation scipy applies moves it by far less than the
    tolerance)."""
    from scipy.stats import entropy as scipy_entropy
    g = _golden("entropy_fragile_worked.json")
    q = g["q_star"]
    assert abs(-q * math.log(q) - (1 - q) * math.log(1 - q) - math.log(1.5)) < 1e-15
    for case in g["cases"]:
        a = np.float32(case["a"])
        w = a.astype(np.float64)
        e_lib = float(np.exp(scipy_entropy(w / w.sum())))
        assert abs(e_lib - case["exp_H"]) <= 5e-8 * case["exp_H"], case
        assert O.entropy_fragile(a, g["eps"]) == case["fragile"], case
        if not case["fragile"]:
            assert O.entropy_count(a) == int(math.floor(case["exp_H"] + 0.5)), case

"""Pins of the oracle's hole-filling compaction layout: hand-worked cases,
the invariants that define it, and its equivalence with the stable layout
for attention (softmax over the resident tokens does not depend on their
order).  CPU only."""
import numpy as np

import oracle as O
import workloads as W


def test_fill_hand_worked_compress():
    # P = 4, b = 4: candidates 0..11, protected 12..15, T = 12
    P, b = 4, 4
    toks = np.arange(P * b) * 10
    kept = np.array([0, 2, 3, 5, 6, 8, 9, 11])              # evicts 1, 4, 7, 10
    out = O.compact_tokens(toks, kept, P, b, drop=1, layout="fill")
    # the protected 120..150 fill slots 1, 4, 7, 10 in order
    assert out.tolist() == [0, 120, 20, 30, 130, 50, 60, 140, 80, 90, 150, 110, 120, 130, 140, 150]


def test_fill_hand_worked_shrink():
    # P = 5, b = 4: T = 12, K_t = 8 kept of 16 candidates; 12..15 is page P-2
    P, b = 5, 4
    toks = np.arange(P * b) * 10
    kept = np.array([1, 4, 6, 9, 10, 13, 14, 15])            # evicted: 0 2 3 5 7 8 11 12
    out = O.compact_tokens(toks, kept, P, b, drop=2, layout="fill")
    # holes below 12: 0 2 3 5 7 8 11 (7 of them); movers at or above 12:
    # 13 14 15 (kept) and 16..19 (protected)
    assert out[:12].tolist() == [130, 10, 140, 150, 40, 160, 60, 170, 180, 90, 100, 190]
    assert out[12:].tolist() == toks[12:].tolist()


def test_fill_invariants_random():
    rng = np.random.default_rng(8)
    for _ in range(200):
        b = int(rng.choice([2, 4, 16]))
        drop = int(rng.integers(1, 3))
        P = int(rng.integers(drop + 1, 9))
        s = rng.uniform(0, 1, (P - 1) * b).astype(np.float32)
        kept = O.select_retained(s, P, b, int(rng.integers(0, b + 1)), drop)
        toks = np.arange(P * b) + 1000
        out = O.compact_tokens(toks, kept, P, b, drop, layout="fill")
        shift = O.compact_tokens(toks, kept, P, b, drop, layout="shift")
        T = (P - drop) * b
        # same resident multiset as the stable layout
        assert sorted(out[:T].tolist()) == sorted(shift[:T].tolist())
        # kept tokens below T never move; slots at or above T keep their contents
        for slot in kept[kept < T]:
            assert out[slot] == toks[slot]
        assert np.array_equal(out[T:], toks[T:])
        # at most drop * b tokens move, each into a slot below T, in slot order
        moved = [i for i in range(T) if out[i] != toks[i]]
        assert len(moved) <= drop * b
        assert all(out[moved[k]] < out[moved[k + 1]] for k in range(len(moved) - 1))


def test_fill_same_attention_as_shift():
    """Decode attention over a request compacted either way agrees to
    rounding: the layouts hold the same tokens."""
    w = W.tiny()
    b = w.page_size
    G = w.num_q_heads // w.num_kv_heads
    rng = np.random.default_rng(3)
    for r in range(w.num_reqs):
        P = int(w.num_pages[r])
        n = (P - 1) * b
        toks = {x: O.gather_tokens(w.dense_pool(x), w.page_table[r], P * b, b) for x in ("k", "v")}
        kept = [O.select_retained(rng.uniform(0, 1, n).astype(np.float32), P, b, 4)
                for _ in range(w.num_kv_heads)]
        outs = []
        for layout in ("shift", "fill"):
            c = {x: t.copy() for x, t in toks.items()}
            for x in ("k", "v"):
                for h in range(w.num_kv_heads):
                    c[x][:, h] = O.compact_tokens(toks[x][:, h], kept[h], P, b, 1, layout)
            kk, vv = O.widen(c["k"][:n], "f32"), O.widen(c["v"][:n], "f32")
            q = O.widen(w.q_post[r], "f32")
            outs.append(np.stack([O.attention(q[g], kk[:, g // G], vv[:, g // G], 0.125)[0]
                                  for g in range(w.num_q_heads)]))
        assert not np.array_equal(c["k"], toks["k"])
        np.testing.assert_allclose(outs[0], outs[1], rtol=1e-12, atol=1e-12)


def test_boundary_step_fill_matches_shift_up_to_order():
    """A whole boundary event (compress, shrink) with either layout: the same
    decisions and page state, and per head the same resident tokens."""
    w = W._build(name="layout", seed=41, dtype="f32", Hq=4, Hkv=2, d=64,
                 n=np.array([96, 160, 100, 48]), budgets=None, free_pages=6, heavy_mode="scaled",
                 heavy_frac=0.05, summary_mode="random")
    b = w.page_size
    for kw in (dict(tau=np.inf), dict(policy="shrink", tau=np.inf, shrink_threshold=10.0,
                                      min_capacity_pages=2)):
        res, pools, states = [], [], []
        for layout in ("shift", "fill"):
            k, v = w.dense_pool("k"), w.dense_pool("v")
            st = O.PageState(w.page_table.copy(), w.num_pages.copy(), w.seq_lens.copy(),
                             w.refcount.copy(), w.free_list.copy(), w.free_count)
            res.append(O.boundary_step([(k, v)], w.dtype, st, w.q_pre, w.qstate, w.slot_ids,
                                       w.positions, w.boundary, O.Params(layout=layout, **kw)))
            pools.append((k, v))
            states.append(st)
        assert np.array_equal(res[0]["decisions"], res[1]["decisions"])
        assert np.array_equal(states[0].page_table, states[1].page_table)
        assert np.array_equal(states[0].seq_lens, states[1].seq_lens)
        for r in w.boundary:
            m = int(states[0].seq_lens[r])
            for x in range(2):
                a = O.gather_tokens(pools[0][x], states[0].page_table[r], m, b)
                c = O.gather_tokens(pools[1][x], states[1].page_table[r], m, b)
                for h in range(w.num_kv_heads):
                    ka = sorted(map(bytes, a[:, h]))
                    kc = sorted(map(bytes, c[:, h]))
                    assert ka == kc

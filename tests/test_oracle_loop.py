"""Pins of the oracle's decode loop (one token per request and step, boundary
events as they come, compaction asynchronous to the next step, App. E.3):
with every boundary growing the cache is the initial tokens followed by every
appended token and each step's output is plain attention over it; a
compressing request sits exactly one step out; the page pool stays
consistent over many steps.  CPU only."""
import math

import numpy as np
import torch

import oracle as O
import workloads as W


def _small(seed=61, free_pages=60):
    return W._build(name="loop", seed=seed, dtype="f32", Hq=4, Hkv=2, d=64,
                    n=np.array([30, 47, 64, 15, 100, 81]), budgets=None, free_pages=free_pages,
                    heavy_mode="scaled", heavy_frac=0.05, summary_mode="random")


def _state(w):
    return O.PageState(w.page_table.copy(), w.num_pages.copy(), w.seq_lens.copy(), w.refcount.copy(),
                       w.free_list.copy(), w.free_count)


def test_always_grow_cache_is_the_whole_sequence():
    w = _small()
    b = w.page_size
    st = _state(w)
    pools = [(w.dense_pool("k"), w.dense_pool("v"))]
    seqs = {r: [O.gather_tokens(pools[0][x], w.page_table[r], int(w.seq_lens[r]), b) for x in range(2)]
            for r in range(w.num_reqs)}
    qs, pos, held = w.qstate.copy(), w.positions.copy(), set()
    p = O.Params(tau=-math.inf)
    for t, inp in enumerate(W.step_inputs(w, 40)):
        out, qs, held, res, app = O.serve_step(pools, "f32", st, held, qs, w.slot_ids, pos, inp, p)
        assert not held
        for r in app:
            seqs[r][0] = np.concatenate([seqs[r][0], inp["k_new"][0][r][None]])
            seqs[r][1] = np.concatenate([seqs[r][1], inp["v_new"][0][r][None]])
        for r in range(w.num_reqs):
            K, V = seqs[r]
            assert int(st.seq_lens[r]) == K.shape[0]
            assert np.array_equal(O.gather_tokens(pools[0][0], st.page_table[r], K.shape[0], b), K)
            # plain attention over the whole sequence (torch, fp64)
            q = torch.from_numpy(inp["q_post"][r].astype(np.float64))
            Kt = torch.from_numpy(K.astype(np.float64)).repeat_interleave(2, dim=1).transpose(0, 1)
            Vt = torch.from_numpy(V.astype(np.float64)).repeat_interleave(2, dim=1).transpose(0, 1)
            a = torch.softmax((Kt @ q[:, :, None])[..., 0] * 0.125, dim=-1)
            ref = (a[:, None, :] @ Vt)[:, 0]
            np.testing.assert_allclose(out[r], ref.numpy(), rtol=1e-12, atol=1e-12)
    # a request full at the start stalls one step, every other appends every step
    full0 = [r for r in range(w.num_reqs) if w.seq_lens[r] == w.num_pages[r] * b]
    for r in range(w.num_reqs):
        assert pos[r] == w.positions[r] + 40 - (1 if r in full0 else 0)


def test_compressing_request_sits_one_step_out():
    w = _small()
    b = w.page_size
    st = _state(w)
    pools = [(w.dense_pool("k"), w.dense_pool("v"))]
    qs, pos, held = w.qstate.copy(), w.positions.copy(), set()
    p = O.Params(tau=math.inf)
    seen = 0
    for t, inp in enumerate(W.step_inputs(w, 40)):
        m_before = st.seq_lens.copy()
        P_before = st.num_pages.copy()
        qs_before = qs.copy()
        was_held = set(held)
        out, qs, held, res, app = O.serve_step(pools, "f32", st, held, qs, w.slot_ids, pos, inp, p)
        for r in was_held:
            seen += 1
            assert np.isnan(out[r]).all() and r not in app
            assert st.seq_lens[r] == m_before[r] == (st.num_pages[r] - 1) * b
            assert np.array_equal(qs[w.slot_ids[r]], qs_before[w.slot_ids[r]])
        for r in held:
            assert st.seq_lens[r] == (st.num_pages[r] - 1) * b
        assert app == [r for r in range(w.num_reqs) if r not in was_held and m_before[r] < P_before[r] * b]
    assert seen >= 10


def test_pool_consistent_over_many_steps_mixed():
    w = _small(free_pages=8)
    b = w.page_size
    st = _state(w)
    pools = [(w.dense_pool("k"), w.dense_pool("v"))]
    qs, pos, held = w.qstate.copy(), w.positions.copy(), set()
    decisions = set()
    for t, inp in enumerate(W.step_inputs(w, 60, seed=1)):
        p = O.Params(tau=0.0 if t % 3 else -math.inf)
        out, qs, held, res, app = O.serve_step(pools, "f32", st, held, qs, w.slot_ids, pos, inp, p)
        decisions |= set(res["decisions"].tolist())
        refs = np.zeros_like(st.refcount)
        for r in range(w.num_reqs):
            P = int(st.num_pages[r])
            assert 0 <= st.seq_lens[r] <= P * b
            assert (st.page_table[r, :P] >= 0).all() and (st.page_table[r, P:] == -1).all()
            np.add.at(refs, st.page_table[r, :P], 1)
        assert np.array_equal(refs, st.refcount)
        free = st.free_list[: st.free_count]
        assert len(set(free.tolist())) == free.size and (refs[free] == 0).all()
        assert free.size + int((refs > 0).sum()) == w.pool_pages
    assert {O.GROW, O.COMPRESS} <= decisions

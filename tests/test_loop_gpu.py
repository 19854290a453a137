"""GPU parity of the split boundary calls and of the decode loop with
asynchronous compaction (App. E.3): select / decide / compact against
gp_boundary_apply, held requests in decode attention, the step prologue
(KV append + summaries) against the oracle, and whole multi-step loops run
the asynchronous way on the GPU (compaction on a second stream beside the
next step's decode) against the oracle's decode loop, step by step."""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_03494_amd as gp
import workloads as W
from _harness import (DEV, AbsPool, DeviceCase, assert_rows_close, bf16_rounding_ok, fp32_elementwise_ok,
                      library_params, oracle_state,
                      to_numpy, to_torch, torch_dtype)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gp.load()


def _say(*a):
    print(*a, flush=True)


def _small(seed=61, free_pages=60, dtype="f32"):
    return W._build(name="loop", seed=seed, dtype=dtype, Hq=4, Hkv=2, d=64,
                    n=np.array([30, 47, 64, 15, 100, 81]), budgets=None, free_pages=free_pages,
                    heavy_mode="scaled", heavy_frac=0.05, summary_mode="random")


def _bytes(t):
    return to_numpy(t).tobytes()


# ------------------------------------------------------ split == apply --

@pytest.mark.parametrize("case", ["tau0", "compress", "shrink_fill", "tau0_big_pool", "grow_big_pool",
                                  "random_big_pool"])
def test_split_calls_equal_apply(case):
    """select + decide + compact (hold 0), and with hold 1 then release, give
    the bytes of one gp_boundary_apply; so does the split with the selection
    told that the counts are final (it then skips the requests that can only
    grow, as gp_boundary_apply always does).  With a big free pool most or
    all grows are skipped; with 30 free pages none can be."""
    big = case.endswith("big_pool")
    w = W.qwen3_8b(seed=7, num_reqs=12, len_lo=300, len_hi=4000, budget_choices=(8, 60, 200),
                   boundary_frac=0.5, free_pages=5000 if big else 30)
    Rb = len(w.boundary)
    draws = torch.from_numpy(np.random.default_rng(3).random(Rb).astype(np.float32)).to(DEV)
    p = {"tau0": O.Params(), "compress": O.Params(tau=math.inf),
         "shrink_fill": O.Params(tau=math.inf, policy="shrink", shrink_threshold=10.0, min_capacity_pages=2,
                                 layout="fill"),
         "tau0_big_pool": O.Params(), "grow_big_pool": O.Params(tau=-math.inf),
         "random_big_pool": O.Params(policy="random", compress_prob=0.5)}[case]
    gparams = library_params(p, w.head_dim)
    if case == "random_big_pool":
        gparams = dataclasses.replace(gparams, draws=draws)
    results = []
    for mode in ("apply", "split", "split_hold", "split_skip"):
        _say(f"split: {case}, {mode}")
        dc = DeviceCase(w)
        Rb = len(w.boundary)
        dt = torch_dtype(w)
        bnd = torch.from_numpy(w.boundary.astype(np.int32)).to(DEV)
        max_cand = (w.max_pages - 1) * w.page_size
        counts = torch.zeros((1, Rb, w.num_kv_heads, 2), dtype=torch.int32, device=DEV)
        scores = torch.zeros((1, Rb, w.num_kv_heads, max_cand), device=DEV)
        ws_s = gp.workspace(gp.GP_OP_SCORE, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads, w.head_dim,
                            w.max_pages, dt)
        ws_a = gp.workspace(gp.GP_OP_APPLY, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads, w.head_dim,
                            w.max_pages, dt)
        gp.gp_boundary_score(dc.layers[0], dc.ps, dc.q_pre, dc.qstate, dc.slot_ids, dc.positions, bnd,
                             gparams, counts[0], scores[0], ws_s)
        dec = torch.full((Rb,), -1, dtype=torch.int32, device=DEV)
        delta = torch.zeros(Rb, device=DEV)
        ctr = torch.zeros(4, dtype=torch.int64, device=DEV)
        mp = dataclasses.replace(gparams, select_skip_grows=1) if mode == "split_skip" else gparams
        args = (dc.layers, dc.ps, bnd, counts, scores, mp, dec, delta, ctr, ws_a)
        if mode == "apply":
            gp.gp_boundary_apply(*args)
        else:
            gp.gp_boundary_select(*args)
            gp.gp_boundary_decide(*args, hold=(mode == "split_hold"))
            if mode == "split_hold":
                torch.cuda.synchronize()
                sl = dc.ps.seq_lens.cpu().numpy()
                d_ = dec.cpu().numpy()
                for i, r in enumerate(w.boundary):
                    assert (sl[r] < 0) == (d_[i] in (gp.GP_COMPRESS, gp.GP_FALLBACK, gp.GP_SHRINK))
            gp.gp_boundary_compact(*args)
            if mode == "split_hold":
                gp.gp_release_held(dc.ps)
        torch.cuda.synchronize()
        results.append([_bytes(t) for t in (dec, delta, ctr, dc.ps.page_table, dc.ps.num_pages, dc.ps.seq_lens,
                                             dc.ps.refcount, dc.ps.free_list, dc.ps.free_count,
                                             dc.layers[0].k, dc.layers[0].v)])
    names = ("decisions", "delta", "counters", "page_table", "num_pages", "seq_lens", "refcount", "free_list",
             "free_count", "k", "v")
    for other in results[1:]:
        for n, a, b in zip(names, results[0], other):
            assert a == b, f"{case}: {n} differs from gp_boundary_apply"


def test_skipped_request_that_does_not_grow_is_preempted():
    """The selection skips requests whose counts say they grow (a big free
    pool); if the decision then gets counts that say compress -- the caller
    broke the contract that the counts are final -- every skipped request is
    preempted: decisions PREEMPT, counters [0, 0, 0, Rb], and the page state
    and the cache rows untouched by the decision and the compaction."""
    w = W.qwen3_8b(seed=9, num_reqs=10, len_lo=300, len_hi=3000, budget_choices=(8, 60, 200),
                   boundary_frac=0.5, free_pages=5000)
    dc = DeviceCase(w)
    Rb = len(w.boundary)
    gparams = dataclasses.replace(library_params(O.Params(), w.head_dim), select_skip_grows=1)
    bnd = torch.from_numpy(w.boundary.astype(np.int32)).to(DEV)
    max_cand = (w.max_pages - 1) * w.page_size
    grow_counts = torch.zeros((1, Rb, w.num_kv_heads, 2), dtype=torch.int32, device=DEV)
    grow_counts[..., 0] = 16                      # K^S > K^L: Delta > 0, wants to grow
    compress_counts = grow_counts.flip(-1).contiguous()   # K^S < K^L: wants to compress
    scores = torch.rand((1, Rb, w.num_kv_heads, max_cand), device=DEV)
    ws_a = gp.workspace(gp.GP_OP_APPLY, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads, w.head_dim,
                        w.max_pages, torch_dtype(w))
    dec = torch.full((Rb,), -1, dtype=torch.int32, device=DEV)
    delta = torch.zeros(Rb, device=DEV)
    ctr = torch.zeros(4, dtype=torch.int64, device=DEV)
    before = [_bytes(t) for t in (dc.ps.page_table, dc.ps.num_pages, dc.ps.seq_lens, dc.ps.refcount,
                                  dc.ps.free_list, dc.ps.free_count, dc.layers[0].k, dc.layers[0].v)]
    _say("skip safety: select with grow counts, decide and compact with compress counts")
    gp.gp_boundary_select(dc.layers, dc.ps, bnd, grow_counts, scores, gparams, dec, delta, ctr, ws_a)
    args = (dc.layers, dc.ps, bnd, compress_counts, scores, gparams, dec, delta, ctr, ws_a)
    gp.gp_boundary_decide(*args, hold=False)
    gp.gp_boundary_compact(*args)
    torch.cuda.synchronize()
    assert (dec.cpu().numpy() == gp.GP_PREEMPT).all()
    assert ctr.cpu().numpy().tolist() == [0, 0, 0, Rb]
    after = [_bytes(t) for t in (dc.ps.page_table, dc.ps.num_pages, dc.ps.seq_lens, dc.ps.refcount,
                                 dc.ps.free_list, dc.ps.free_count, dc.layers[0].k, dc.layers[0].v)]
    names = ("page_table", "num_pages", "seq_lens", "refcount", "free_list", "free_count", "k", "v")
    for n, a, b in zip(names, before, after):
        assert a == b, f"{n} changed"


# ------------------------------------------------------- held requests --

def test_decode_leaves_held_requests_out():
    w = W.qwen3_8b(seed=5, num_reqs=16, len_lo=200, len_hi=3000, budget_choices=(20, 100),
                   boundary_frac=0.3, free_pages=20)
    dc = DeviceCase(w)
    scale = float(np.float32(1 / math.sqrt(w.head_dim)))
    ref = dc.decode(scale)
    held = [1, 4, 5, 11]
    sl = dc.ps.seq_lens.clone()
    for r in held:
        dc.ps.seq_lens[r] = -int(w.seq_lens[r]) - 1
    _say("held: decode with requests", held, "held")
    out = torch.full_like(dc.q_post, float("nan"))
    gp.gp_decode_attention(dc.layers[0], dc.ps, dc.q_post, scale, out, dc.ws_decode)
    # the fused step leaves their summaries alone as well
    qs0 = dc.qstate.clone()
    init = torch.zeros(w.num_reqs, dtype=torch.uint8, device=DEV)
    out2 = torch.full_like(dc.q_post, float("nan"))
    gp.gp_decode_step(dc.layers[0], dc.ps, dc.q_post, dc.q_pre, scale, out2, dc.slot_ids, init, dc.qstate,
                      0.9, 0.999, dc.ws_decode)
    torch.cuda.synchronize()
    got = O.widen(to_numpy(out), w.dtype)
    got2 = O.widen(to_numpy(out2), w.dtype)
    qs = dc.qstate.cpu().numpy()
    for r in range(w.num_reqs):
        if r in held:
            assert np.isnan(got[r]).all() and np.isnan(got2[r]).all()
            assert np.array_equal(qs[w.slot_ids[r]], qs0.cpu().numpy()[w.slot_ids[r]], equal_nan=True)
        else:
            assert np.array_equal(got[r], ref[r]) and np.array_equal(got2[r], ref[r])
            assert not np.array_equal(qs[w.slot_ids[r]], qs0.cpu().numpy()[w.slot_ids[r]])
    gp.gp_release_held(dc.ps)
    torch.cuda.synchronize()
    assert torch.equal(dc.ps.seq_lens, sl)


# ---------------------------------------------------------- step prologue --

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_append_step_matches_oracle(dtype):
    """KV append + summary update of every request with room, over two
    layers; full and held requests untouched."""
    w = _small(dtype=dtype)
    L = 2
    dc = DeviceCase(w, n_layers=L, distinct_layers=True)
    b = w.page_size
    held = 4
    inp = W.step_inputs(w, 1, seed=3, n_layers=L)[0]
    full = [r for r in range(w.num_reqs) if w.seq_lens[r] == w.num_pages[r] * b]
    assert full, "the case needs a request with full pages"
    # oracle
    st = oracle_state(w)
    st.seq_lens[held] = w.seq_lens[held]          # held: skipped below
    pools = [(wl.dense_pool("k"), wl.dense_pool("v")) for wl in dc.layer_workloads]
    qs_ref = [wl.qstate.copy() for wl in dc.layer_workloads]
    pos = w.positions.copy()
    app = []
    for r in range(w.num_reqs):
        if r == held:
            continue
        kv = [(inp["k_new"][l][r], inp["v_new"][l][r]) for l in range(L)]
        if O.append_token(pools, st, r, kv, b):
            pos[r] += 1
            app.append(r)
    idx = np.array(app)
    p32 = O.Params().as_f32(w.head_dim)
    for l in range(L):
        qs_ref[l] = O.update_summaries(inp["q_pre"][idx], dtype, w.slot_ids[idx], np.zeros(idx.size, np.uint8),
                                       qs_ref[l], p32.beta_s, p32.beta_l)
    # GPU
    dc.ps.seq_lens[held] = -int(w.seq_lens[held]) - 1
    positions = dc.positions.clone()
    qstate = torch.stack(dc.qstate_layers).contiguous()
    k_new = torch.stack([to_torch(x, dtype) for x in inp["k_new"]]).contiguous()
    v_new = torch.stack([to_torch(x, dtype) for x in inp["v_new"]]).contiguous()
    q_pre = torch.stack([to_torch(inp["q_pre"], dtype)] * L).contiguous()
    _say(f"append step: {dtype}, two layers, held request {held}, full requests {full}")
    gp.gp_append_step(dc.layers, dc.ps, positions, k_new, v_new, q_pre, dc.slot_ids, None, qstate,
                      p32.beta_s, p32.beta_l)
    gp.gp_release_held(dc.ps)
    torch.cuda.synchronize()
    assert np.array_equal(dc.ps.seq_lens.cpu().numpy(), st.seq_lens)
    assert np.array_equal(positions.cpu().numpy(), pos)
    got_qs = qstate.cpu().numpy()
    for l in range(L):
        assert np.array_equal(got_qs[l], qs_ref[l], equal_nan=True), f"summaries of layer {l}"
        for r in range(w.num_reqs):
            m = int(st.seq_lens[r])
            for x, which in enumerate(("k", "v")):
                want = O.gather_tokens(pools[l][x], st.page_table[r], m, b)
                have = dc.gather(st.page_table[r], m, which, layer=l)
                assert np.array_equal(want, have), f"{which} of request {r}, layer {l}"


# ------------------------------------- the token folded into the decode step --

def _step_case(case):
    if case == "f32":
        return _small(dtype="f32")
    if case == "bf16_qwen3":
        return W.qwen3_8b(seed=71, num_reqs=9, len_lo=30, len_hi=5000, budget_choices=(4, 40, 400),
                          boundary_frac=0.25, free_pages=32)
    return W.prefix_shared(num_reqs=5, prefix_len=256, tail_lo=20, tail_hi=700, free_pages=40)


@pytest.mark.parametrize("case", ["f32", "bf16_qwen3", "bf16_g8"])
def test_decode_step_with_token_against_oracle(case):
    """gp_decode_step with the step's token folded in (Sec. 4.1): K and V
    written at slot m_r of every request with room, the summaries of those
    requests updated, decode attention over m_r + 1 tokens, lengths and
    positions advanced; a held request and requests with full pages as in the
    loop, a request with nothing resident attends to the new token alone.
    Against the oracle's append_token + update_summaries + decode_attention,
    and bit for bit against gp_append_step followed by gp_decode_attention."""
    w = _step_case(case)
    b, R, dt = w.page_size, w.num_reqs, w.dtype
    inp = W.step_inputs(w, 1, seed=5)[0]
    full = [r for r in range(R) if w.seq_lens[r] == w.num_pages[r] * b]
    # (no empty request under a shared prefix: its first page is shared, so its
    # token would land in a page other requests read)
    empty = 1 if case != "bf16_g8" else None
    held = max(r for r in range(R) if r not in full and r != empty)
    assert full and empty not in full
    init = np.zeros(R, np.uint8)
    init[0] = 1
    p32 = O.Params().as_f32(w.head_dim)
    scale = float(np.float32(1.0 / math.sqrt(w.head_dim)))
    _say(f"decode step with the token folded in: {case}, full {full}, held {held}, empty {empty}")
    # oracle
    st = oracle_state(w)
    if empty is not None:
        st.seq_lens[empty] = 0
    pools = [(w.dense_pool("k"), w.dense_pool("v"))]
    pos = w.positions.copy()
    active = [r for r in range(R) if r != held]
    app = [r for r in active if O.append_token(pools, st, r, [(inp["k_new"][0][r], inp["v_new"][0][r])], b)]
    for r in app:
        pos[r] += 1
    idx = np.array(app)
    qs_ref = O.update_summaries(inp["q_pre"][idx], dt, w.slot_ids[idx], init[idx], w.qstate,
                                p32.beta_s, p32.beta_l)
    ref = O.decode_attention(pools[0][0], pools[0][1], dt, st.page_table, st.seq_lens, inp["q_post"],
                             w.num_q_heads, scale, requests=active)[active]

    def run(fused, advance=True):
        dc = DeviceCase(w)
        if empty is not None:
            dc.ps.seq_lens[empty] = 0
        dc.ps.seq_lens[held] = -int(w.seq_lens[held]) - 1
        positions = dc.positions.clone()
        q_pre, q_post = to_torch(inp["q_pre"], dt), to_torch(inp["q_post"], dt)
        k_new, v_new = to_torch(inp["k_new"][0], dt), to_torch(inp["v_new"][0], dt)
        ini = torch.from_numpy(init).to(DEV)
        out = torch.full_like(q_post, float("nan"))
        if fused:
            gp.gp_decode_step(dc.layers[0], dc.ps, q_post, q_pre, scale, out, dc.slot_ids, ini, dc.qstate,
                              p32.beta_s, p32.beta_l, dc.ws_decode, k_new=k_new, v_new=v_new,
                              positions=positions, advance=advance)
        else:
            gp.gp_append_step(dc.layers, dc.ps, positions, k_new[None].contiguous(), v_new[None].contiguous(),
                              q_pre[None].contiguous(), dc.slot_ids, ini, dc.qstate[None], p32.beta_s,
                              p32.beta_l)
            gp.gp_decode_attention(dc.layers[0], dc.ps, q_post, scale, out, dc.ws_decode)
        torch.cuda.synchronize()
        return dc, positions, out

    dc, positions, out = run(True)
    got = O.widen(to_numpy(out), dt)
    assert np.isnan(got[held]).all(), "the held request's output row was written"
    g = got[active]
    if dt == "f32":
        ref_abs = O.decode_attention(pools[0][0], AbsPool(pools[0][1]), dt, st.page_table, st.seq_lens,
                                     inp["q_post"], w.num_q_heads, scale, requests=active)[active]
        assert_rows_close(g, ref, 1e-5, "decode step fp32")
        assert fp32_elementwise_ok(g, ref, ref_abs), "decode step fp32: element-wise bar"
    else:
        assert_rows_close(g, ref, 2e-2, "decode step bf16")
        assert bf16_rounding_ok(g, ref), "decode step bf16: beyond bf16 rounding of the exact value"
    np.testing.assert_array_equal(dc.qstate.cpu().numpy().view(np.int32), qs_ref.view(np.int32))
    sl = dc.ps.seq_lens.cpu().numpy()
    want_sl = st.seq_lens.copy()
    want_sl[held] = -int(w.seq_lens[held]) - 1
    np.testing.assert_array_equal(sl, want_sl)
    np.testing.assert_array_equal(positions.cpu().numpy(), pos)
    for r in active:
        m = int(st.seq_lens[r])
        for x, which in enumerate(("k", "v")):
            want = O.gather_tokens(pools[0][x], st.page_table[r], m, b)
            assert np.array_equal(want, dc.gather(st.page_table[r], m, which)), f"{which} of request {r}"
    # the two launches of the loop prologue give the same bytes
    dc2, positions2, out2 = run(False)
    assert _bytes(out2) == _bytes(out)        # bytes: the held row is NaN in both
    assert _bytes(dc2.qstate) == _bytes(dc.qstate) and torch.equal(positions2, positions)
    assert torch.equal(dc2.ps.seq_lens, dc.ps.seq_lens)
    assert _bytes(dc2.layers[0].k) == _bytes(dc.layers[0].k) and _bytes(dc2.layers[0].v) == _bytes(dc.layers[0].v)
    # advance = 0 (every layer but the last): the same outputs, the token in the
    # cache, lengths and positions as they were
    dc3, positions3, out3 = run(True, advance=False)
    assert _bytes(out3) == _bytes(out)
    assert _bytes(dc3.layers[0].k) == _bytes(dc.layers[0].k) and _bytes(dc3.layers[0].v) == _bytes(dc.layers[0].v)
    assert torch.equal(positions3, dc3.positions)
    sl3 = dc3.ps.seq_lens.cpu().numpy()
    assert (empty is None or sl3[empty] == 0) and sl3[held] == -int(w.seq_lens[held]) - 1
    assert all(sl3[r] == w.seq_lens[r] for r in range(R) if r not in (empty, held))


# -------------------------------------------------- the decode loop itself --

class Loop:
    """The asynchronous decode loop on the GPU, one layer.  Per step, on the
    main stream: prologue (append + summaries), decode attention; beside it on
    stream B: scoring and selection of every request whose pages are full;
    then (after B and after the previous step's compaction on stream A)
    release of the held requests and the decision with hold; the compaction
    goes to stream A, beside the next step."""

    def __init__(self, w, params: O.Params):
        self.w = w
        self.dc = DeviceCase(w)
        self.p = library_params(params, w.head_dim)
        R, Hq, Hkv, d = w.num_reqs, w.num_q_heads, w.num_kv_heads, w.head_dim
        dt = torch_dtype(w)
        self.dt = dt
        self.bnd = torch.arange(R, dtype=torch.int32, device=DEV)     # every request; the kernels filter
        max_cand = (w.max_pages - 1) * w.page_size
        self.counts = torch.zeros((1, R, Hkv, 2), dtype=torch.int32, device=DEV)
        self.scores = torch.zeros((1, R, Hkv, max_cand), device=DEV)
        self.dec = torch.zeros(R, dtype=torch.int32, device=DEV)
        self.delta = torch.zeros(R, device=DEV)
        self.ctr = torch.zeros(4, dtype=torch.int64, device=DEV)
        self.ws_s = gp.workspace(gp.GP_OP_SCORE, R, R, Hq, Hkv, d, w.max_pages, dt)
        self.ws_a = [gp.workspace(gp.GP_OP_APPLY, R, R, Hq, Hkv, d, w.max_pages, dt) for _ in range(2)]
        self.positions = self.dc.positions
        self.qstate5 = self.dc.qstate.view(1, *self.dc.qstate.shape)
        self.out = torch.empty_like(self.dc.q_post)
        self.side_a = torch.cuda.Stream()
        self.side_b = torch.cuda.Stream()
        self.t = 0

    def step(self, inp):
        dc, w = self.dc, self.w
        main = torch.cuda.current_stream()
        k_new = to_torch(inp["k_new"][0], w.dtype)[None].contiguous()
        v_new = to_torch(inp["v_new"][0], w.dtype)[None].contiguous()
        q_pre = to_torch(inp["q_pre"], w.dtype)
        q_post = to_torch(inp["q_post"], w.dtype)
        self.out.fill_(float("nan"))
        gp.gp_append_step([dc.layers[0]], dc.ps, self.positions, k_new, v_new, q_pre[None].contiguous(),
                          dc.slot_ids, None, self.qstate5, self.p.beta_s, self.p.beta_l)
        self.side_b.wait_stream(main)
        ws = self.ws_a[self.t % 2]
        args = ([dc.layers[0]], dc.ps, self.bnd, self.counts, self.scores, self.p, self.dec, self.delta,
                self.ctr, ws)
        with torch.cuda.stream(self.side_b):
            gp.gp_boundary_score(dc.layers[0], dc.ps, q_pre, dc.qstate, dc.slot_ids, self.positions, self.bnd,
                                 self.p, self.counts[0], self.scores[0], self.ws_s)
            gp.gp_boundary_select(*args)
        gp.gp_decode_attention(dc.layers[0], dc.ps, q_post, self.p.scale, self.out, dc.ws_decode)
        main.wait_stream(self.side_b)
        main.wait_stream(self.side_a)
        gp.gp_release_held(dc.ps)
        gp.gp_boundary_decide(*args, hold=True)
        self.side_a.wait_stream(main)
        with torch.cuda.stream(self.side_a):
            gp.gp_boundary_compact(*args)
        # tensors made on this stream and used on the side streams stay alive
        # until the side streams are joined (the test synchronises every step)
        self.keep = (k_new, v_new, q_pre, q_post)
        self.t += 1


def _run_loop(w, params, n_steps, seed=0, check_every=1):
    b = w.page_size
    loop = Loop(w, params)
    p32 = params.as_f32(w.head_dim)
    st = oracle_state(w)
    pools = [(w.dense_pool("k"), w.dense_pool("v"))]
    qs, pos, held = w.qstate.copy(), w.positions.copy(), set()
    seen = {}
    for t, inp in enumerate(W.step_inputs(w, n_steps, seed=seed)):
        out_o, qs, held, res, app = O.serve_step(pools, w.dtype, st, held, qs, w.slot_ids, pos, inp, p32)
        for dcd in res["decisions"].tolist():
            seen[dcd] = seen.get(dcd, 0) + 1
        loop.step(inp)
        torch.cuda.synchronize()
        # page state (held requests carry -(m + 1) on the GPU)
        gs = loop.dc.host_state()
        sl = gs.seq_lens.copy()
        assert {int(r) for r in np.nonzero(sl < 0)[0]} == held, f"step {t}: held set"
        sl = np.where(sl < 0, -sl - 1, sl)
        assert np.array_equal(sl, st.seq_lens), f"step {t}: seq_lens"
        for name in ("page_table", "num_pages", "refcount"):
            assert np.array_equal(getattr(gs, name), getattr(st, name)), f"step {t}: {name}"
        assert gs.free_count == st.free_count
        assert np.array_equal(gs.free_list[: gs.free_count], st.free_list[: st.free_count])
        assert np.array_equal(loop.positions.cpu().numpy(), pos)
        assert np.array_equal(loop.dc.qstate.cpu().numpy(), qs, equal_nan=True), f"step {t}: summaries"
        # decisions of the requests that met a boundary this step
        dec_g = loop.dec.cpu().numpy()
        bnd_o = [r for r in range(w.num_reqs) if dec_g[r] != gp.GP_NOT_BOUNDARY]
        assert len(bnd_o) == len(res["decisions"])
        assert dec_g[bnd_o].tolist() == res["decisions"].tolist(), f"step {t}: decisions"
        # outputs: requests in the batch within the decode bar, held ones unwritten
        got = O.widen(to_numpy(loop.out), w.dtype)
        act = [r for r in range(w.num_reqs) if not np.isnan(out_o[r]).all()]
        for r in range(w.num_reqs):
            if r not in act:
                assert np.isnan(got[r]).all(), f"step {t}: output written for held request {r}"
        if w.dtype == "f32":
            assert_rows_close(got[act], out_o[act], 1e-5, f"step {t} decode")
        else:
            assert_rows_close(got[act], out_o[act], 2e-2, f"step {t} decode")
            assert bf16_rounding_ok(got[act], out_o[act])
        # resident K/V, exact
        if t % check_every == 0 or t == n_steps - 1:
            for r in range(w.num_reqs):
                m = int(st.seq_lens[r])
                for x, which in enumerate(("k", "v")):
                    want = O.gather_tokens(pools[0][x], st.page_table[r], m, b)
                    have = loop.dc.gather(gs.page_table[r], m, which)
                    assert np.array_equal(want, have), f"step {t}: {which} of request {r}"
    return seen


@pytest.mark.parametrize("tau", [0.0, math.inf, -math.inf])
def test_loop_small_fp32(tau):
    w = _small(free_pages=40)
    _say(f"loop: small fp32 batch, 48 steps, tau {tau}")
    seen = _run_loop(w, O.Params(tau=tau), 48)
    _say("decisions seen", seen)
    if tau == math.inf:
        assert seen.get(O.COMPRESS, 0) >= 10


def test_loop_small_shrink_fill_pressure():
    """Shrink policy and the fill layout with a small pool: grows, shrinks,
    compressions and fallbacks in one loop."""
    w = _small(free_pages=3, seed=62)
    p = O.Params(policy="shrink", shrink_threshold=-0.0001, min_capacity_pages=2, layout="fill")
    _say("loop: small fp32 batch, 48 steps, shrink policy, fill layout, 3 free pages")
    seen = _run_loop(w, p, 48)
    _say("decisions seen", seen)


def test_loop_qwen3_bf16():
    w = W.qwen3_8b(seed=11, num_reqs=10, len_lo=200, len_hi=1500, budget_choices=(20, 60),
                   boundary_frac=0.4, free_pages=30)
    _say("loop: Qwen3-8B heads, 10 requests, bf16, 24 steps")
    seen = _run_loop(w, O.Params(), 24, check_every=6)
    _say("decisions seen", seen)

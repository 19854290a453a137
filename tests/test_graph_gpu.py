"""The decode step captured in HIP graphs gives the same bytes as eager calls,
on every replay, with eager work and synchronisations between replays."""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle as O
import workloads as W
from _harness import DeviceCase

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fork,free", [(False, 40), (True, 40), ("bench", 40), ("bench", 5000)],
                         ids=["one_stream", "score_on_side_stream", "bench_step_layout",
                              "bench_step_layout_big_pool"])
def test_graph_replays_match_eager(fork, free):
    """fork="bench" is the benchmark's step: after the summary update, decode
    attention reads a snapshot of the request metadata while scoring, the
    selection (told that the counts are final, so it skips the certain grows;
    with the big pool it does) and the decision run on a side stream beside
    it, then the compaction; its eager result must also equal the plain
    one-stream sequence."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_03494_amd as gp
    print(f"graph: capture decode + boundary step of a reduced Qwen3-8B batch, fork={fork}", flush=True)
    w = W.qwen3_8b(seed=17, num_reqs=10, len_lo=200, len_hi=3000, budget_choices=(20, 100, 200),
                   boundary_frac=0.4, free_pages=free)
    dc = DeviceCase(w)
    p32 = O.Params().as_f32(w.head_dim)
    params = gp.Params(p32.beta_s, p32.beta_l, p32.p, p32.tau, p32.scale, p32.rope_theta, p32.k_loc, 0)
    Rb = len(w.boundary)
    max_cand = (w.max_pages - 1) * w.page_size
    bnd = torch.from_numpy(w.boundary.astype(np.int32)).cuda()
    counts = torch.zeros((Rb, w.num_kv_heads, 2), dtype=torch.int32, device="cuda")
    scores = torch.zeros((Rb, w.num_kv_heads, max_cand), device="cuda")
    dec = torch.zeros(Rb, dtype=torch.int32, device="cuda")
    delta = torch.zeros(Rb, device="cuda")
    ctr = torch.zeros(4, dtype=torch.int64, device="cuda")
    dt = torch.bfloat16
    ws_s = gp.workspace(gp.GP_OP_SCORE, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads, w.head_dim, w.max_pages, dt)
    ws_a = gp.workspace(gp.GP_OP_APPLY, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads, w.head_dim, w.max_pages, dt)
    out = torch.empty_like(dc.q_post)
    init = torch.zeros(w.num_reqs, dtype=torch.uint8, device="cuda")
    aux = torch.cuda.Stream()          # default priority
    state0 = [t.clone() for t in (dc.ps.page_table, dc.ps.num_pages, dc.ps.seq_lens, dc.ps.refcount,
                                  dc.ps.free_list, dc.ps.free_count)]
    k0, v0, qs0 = dc.layers[0].k.clone(), dc.layers[0].v.clone(), dc.qstate.clone()

    def reset():
        for t, t0 in zip((dc.ps.page_table, dc.ps.num_pages, dc.ps.seq_lens, dc.ps.refcount,
                          dc.ps.free_list, dc.ps.free_count), state0):
            t.copy_(t0)
        dc.layers[0].k.copy_(k0)
        dc.layers[0].v.copy_(v0)
        dc.qstate.copy_(qs0)

    bargs = (dc.layers, dc.ps, bnd, counts, scores, params, dec, delta, ctr, ws_a)

    # decode's snapshot of the request metadata (the benchmark's step)
    snap_pt, snap_np, snap_sl = (torch.empty_like(t) for t in (dc.ps.page_table, dc.ps.num_pages,
                                                                dc.ps.seq_lens))
    ps_dec = gp.PageState(snap_pt, snap_np, snap_sl, dc.ps.refcount, dc.ps.free_list, dc.ps.free_count)

    # the selection runs after the scoring on the side stream: the counts are
    # final, so it may skip the requests that can only grow
    bargs_skip = (dc.layers, dc.ps, bnd, counts, scores, dataclasses.replace(params, select_skip_grows=1), dec,
                  delta, ctr, ws_a)

    def step_bench():
        reset()
        cur = torch.cuda.current_stream()
        for t, t0 in ((snap_pt, dc.ps.page_table), (snap_np, dc.ps.num_pages), (snap_sl, dc.ps.seq_lens)):
            torch.mul(t0, 1, out=t)
        gp.gp_update_summaries(dc.q_pre, dc.slot_ids, init, dc.qstate, p32.beta_s, p32.beta_l)
        aux.wait_stream(cur)
        gp.gp_decode_attention(dc.layers[0], ps_dec, dc.q_post, p32.scale, out, dc.ws_decode)
        with torch.cuda.stream(aux):
            gp.gp_boundary_score(dc.layers[0], dc.ps, dc.q_pre, dc.qstate, dc.slot_ids, dc.positions,
                                 bnd, params, counts, scores, ws_s)
            gp.gp_boundary_select(*bargs_skip)
            gp.gp_boundary_decide(*bargs_skip, hold=False)      # updates the live metadata only
        cur.wait_stream(aux)
        gp.gp_boundary_compact(*bargs_skip)

    def step():
        if fork == "bench":
            step_bench()
            return
        reset()
        gp.gp_update_summaries(dc.q_pre, dc.slot_ids, init, dc.qstate, p32.beta_s, p32.beta_l)
        cur = torch.cuda.current_stream()
        if fork:
            # scoring reads keys only: it may run beside decode attention
            aux.wait_stream(cur)
            with torch.cuda.stream(aux):
                gp.gp_boundary_score(dc.layers[0], dc.ps, dc.q_pre, dc.qstate, dc.slot_ids, dc.positions,
                                     bnd, params, counts, scores, ws_s)
        gp.gp_decode_attention(dc.layers[0], dc.ps, dc.q_post, p32.scale, out, dc.ws_decode)
        if fork:
            cur.wait_stream(aux)
        else:
            gp.gp_boundary_score(dc.layers[0], dc.ps, dc.q_pre, dc.qstate, dc.slot_ids, dc.positions, bnd,
                                 params, counts, scores, ws_s)
        gp.gp_boundary_apply(dc.layers, dc.ps, bnd, counts, scores, params, dec, delta, ctr, ws_a)

    def snapshot():
        torch.cuda.synchronize()
        return [t.detach().clone() for t in (out, counts, scores, dec, delta, dc.ps.page_table,
                                              dc.ps.seq_lens, dc.ps.free_list, dc.ps.free_count,
                                              dc.layers[0].k, dc.layers[0].v, dc.qstate)]

    if fork == "bench":
        # the plain sequence on one stream, with gp_boundary_apply
        fork_saved, fork = fork, False
        step()
        plain = snapshot()
        fork = fork_saved
    step()
    eager = snapshot()
    names = ("out", "counts", "scores", "decisions", "delta", "page_table", "seq_lens", "free_list",
             "free_count", "k_pool", "v_pool", "qstate")

    def same_bits(a, b):
        # compare bit patterns, so that NaN-poisoned slots compare equal
        bits = {torch.bfloat16: torch.int16, torch.float32: torch.int32}.get(a.dtype)
        ai, bi = (a.view(bits), b.view(bits)) if bits is not None else (a, b)
        if not torch.equal(ai, bi):
            print("differs in", int((ai != bi).sum()), "of", ai.numel(), flush=True)
            return False
        return True

    if fork == "bench":
        for name, a, b in zip(names, plain, eager):
            assert same_bits(a, b), f"bench step layout: {name} differs from the one-stream sequence"
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        junk = torch.randn(1 << 20, device="cuda").sum()      # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for name, a, b in zip(names, eager, got):
            assert same_bits(a, b), f"replay {rep}: {name} differs"
        del junk

"""Benchmark: one decode step of GrowPage's hot path at the Qwen3-8B layer shape.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]

A step is one pass of the whole path over the batch: restore the page metadata
to the step's starting state (one device-to-device copy), update both query summaries of every request, paged decode attention
for every request, then boundary scoring, selection, the decision and compaction for the
requests at a capacity boundary.  Inputs are seeded synthetic tensors resident
in HBM before timing starts.  Five consecutive steps are captured as one
HIP graph (as a serving loop captures its decode steps: the graph's launch
cost is paid once per five steps, every step does all of its work) and
replayed K / 5 times (``--graph-steps S`` sets the steps per graph; ``--eager``
launches every call directly).  Decode attention reads
a snapshot of the request metadata (written by the restore, in the same
launch), so scoring, selection and the decision (which updates the live
metadata) run on a second stream beside it; the summary update runs before
the fork (``--layout``); the compaction, which moves cached rows, waits for
both (``--serial`` runs everything on one stream, decode on the live
metadata).

Prints one JSON line.  ``value`` is GB/s of the every-step traffic (summaries
and decode attention, algorithmic bytes) over the whole step's time, boundary
work included in the time but not in the bytes; the timed region holds the K
steps and nothing else.  With a shared prefix (``--workload prefix_shared``)
the step decodes with the shared-prefix call and its bytes count each
resident page once.  The ``roofline`` object covers the dominant kernel
(decode attention: split kernel + merge; the shared-prefix call with a shared
prefix), timed with HIP events around K back-to-back launches on its stream
after the timed steps.  A last,
instrumented pass of K eager steps with events between the phases gives the
time the boundary work adds after decode attention.  ``cpu_baseline`` times
the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0

# workload name -> (metric suffix, description)
WORKLOADS = {
    "qwen3_8b": ("Qwen3-8B layer shape",
                 "qwen3_8b_layer: 64 requests, 32 q / 8 kv heads, d 128, page 16, lengths U[1024,8192] "
                 "under page budgets {64,128,256}, 4 at a boundary, 200k free pages"),
    "long_reasoning": ("long-reasoning shape",
                       "long_reasoning: 32 requests, 32 q / 8 kv heads, d 128, page 16, lengths "
                       "U[16384,32768], all at a boundary, heavy fraction per request in {0.1%,1%,10%}, "
                       "200k free pages"),
    "high_concurrency": ("high-concurrency shape",
                         "high_concurrency: 256 requests, 32 q / 8 kv heads, d 128, page 16, lognormal "
                         "lengths (median 2048, sigma 0.8, [256,16384]), 1/8 at a boundary, pool 1.1x use"),
    "prefix_shared": ("prefix-shared Qwen3-32B layer shape",
                      "prefix_shared: 128 requests, 64 q / 8 kv heads, d 128, page 16, a 2048-token shared "
                      "prefix then private tails U[512,8192], 1/16 at a boundary, 200k free pages"),
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", default="qwen3_8b", choices=sorted(WORKLOADS),
                    help="qwen3_8b is the benchmark; the others report the same fields at their shapes")
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU sample")
    ap.add_argument("--ceiling-mib", type=int, default=4096, help="buffer of the streaming-read ceiling")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "decode_traffic_qwen3_8b.json"))
    ap.add_argument("--eager", action="store_true", help="launch every call directly (no HIP graphs)")
    ap.add_argument("--graph-steps", type=int, default=5,
                    help="steps captured per HIP graph (a divisor of --steps is used)")
    ap.add_argument("--layout", default="summaries-first",
                    choices=["boundary-first", "decode-first", "summaries-first"],
                    help="capture order of the two branches of a step (see step())")
    ap.add_argument("--serial", action="store_true",
                    help="run boundary scoring after decode attention on one stream")
    ap.add_argument("--loop-steps", type=int, default=50,
                    help="steps of the decode-loop measurement (0 skips it)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run a plain device copy of this many MiB (counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the path shards by request or by KV head, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_03494_amd as gp
    import workloads as W

    gp.load()
    dev = "cuda"
    w = W.make(args.workload)
    R, Hq, Hkv, d, b = w.num_reqs, w.num_q_heads, w.num_kv_heads, w.head_dim, w.page_size
    e = 2
    dt = torch.bfloat16

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(dt).to(dev)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev)

    shape = (w.pool_pages, Hkv, b, d)
    k = torch.empty(shape, dtype=dt, device=dev)
    v = torch.empty(shape, dtype=dt, device=dev)
    ids = np.nonzero(w.page_row >= 0)[0]
    idx = torch.from_numpy(ids.astype(np.int64)).to(dev)
    k.index_copy_(0, idx, bf(w.k_data[w.page_row[ids]]))
    v.index_copy_(0, idx, bf(w.v_data[w.page_row[ids]]))
    kv = gp.KVLayer(k, v)
    # all page metadata in one int32 buffer, so that the per-step restore is one copy
    parts = dict(page_table=w.page_table, num_pages=w.num_pages, seq_lens=w.seq_lens,
                 refcount=w.refcount, free_list=w.free_list, free_count=np.array([w.free_count]))
    flat = np.concatenate([np.asarray(v, np.int32).ravel() for v in parts.values()])
    # followed by decode attention's snapshot of the request metadata (page
    # table, page counts, lengths), which the restore writes in the same launch
    n_req_meta = int(w.page_table.size) + 2 * R
    meta0_ext = i32(np.concatenate([flat, flat[:n_req_meta]]))
    meta_ext = meta0_ext.clone()
    meta0, meta = meta0_ext[: flat.size], meta_ext[: flat.size]
    views, off = {}, 0
    for name, arr in parts.items():
        n = int(np.asarray(arr).size)
        views[name] = meta[off: off + n].view(np.asarray(arr).shape)
        off += n
    ps = gp.PageState(**views)
    qstate = torch.from_numpy(w.qstate).to(dev)
    slots, positions = i32(w.slot_ids), i32(w.positions)
    q_pre, q_post = bf(w.q_pre), bf(w.q_post)
    init = torch.zeros(R, dtype=torch.uint8, device=dev)
    out = torch.empty_like(q_post)
    bnd = i32(w.boundary)
    Rb = int(bnd.shape[0])
    max_cand = (w.max_pages - 1) * b
    # (the selection runs after the scoring on one stream: the counts are final,
    # so it may skip the requests that can only grow)
    params = gp.Params(scale=float(np.float32(1 / math.sqrt(d))), select_skip_grows=1)
    counts = torch.zeros((Rb, Hkv, 2), dtype=torch.int32, device=dev)
    scores = torch.zeros((Rb, Hkv, max_cand), device=dev)
    decisions = torch.zeros(Rb, dtype=torch.int32, device=dev)
    delta = torch.zeros(Rb, device=dev)
    counters = torch.zeros(4, dtype=torch.int64, device=dev)
    ws_d = gp.workspace(gp.GP_OP_DECODE, R, 0, Hq, Hkv, d, w.max_pages, dt)
    ws_s = gp.workspace(gp.GP_OP_SCORE, R, Rb, Hq, Hkv, d, w.max_pages, dt)
    ws_a = gp.workspace(gp.GP_OP_APPLY, R, Rb, Hq, Hkv, d, w.max_pages, dt)
    stream = torch.cuda.current_stream()

    def restore():
        # the page metadata goes back to the step's starting state, so that every
        # step meets the same boundary requests; the summaries simply keep
        # evolving from step to step, as they would in serving.  An elementwise
        # kernel rather than a copy: in a HIP graph a memcpy node costs a few
        # microseconds of scheduling before the kernel that follows it
        torch.mul(meta0_ext, 1, out=meta_ext)

    def phase_pre():
        restore()

    def phase_summaries():
        gp.gp_update_summaries(q_pre, slots, init, qstate, params.beta_s, params.beta_l)

    def phase_decode():
        gp.gp_decode_attention(kv, ps, q_post, params.scale, out, ws_d)

    # a workload whose requests share a prefix of pages (App. E.2) decodes in
    # the step with the shared-prefix call, which reads each shared page once
    # per block of requests (its three stages in order on one stream)
    prefix_pages = int(w.meta.get("prefix_len", 0)) // b
    groups = [(0, R, prefix_pages)] if prefix_pages else []

    def phase_decode_snapshot():
        if prefix_pages:
            gp.gp_decode_attention_shared(kv, ps_dec, q_post, params.scale, out, groups, ws_d)
        else:
            gp.gp_decode_attention(kv, ps_dec, q_post, params.scale, out, ws_d)

    bargs = ([kv], ps, bnd, counts, scores, params, decisions, delta, counters, ws_a)
    # Decode attention reads a per-step snapshot of the request metadata
    # (page table, page counts, lengths), so that the decision, which updates
    # the live copy, may run beside it; only the compaction, which moves cached
    # rows, waits for it.  The restore writes the snapshot too (one launch); a
    # serving loop without a restore would take it with one small copy.
    snap = meta_ext[meta.numel():]
    npt = views["page_table"].numel()
    ps_dec = gp.PageState(snap[:npt].view(views["page_table"].shape), snap[npt: npt + R], snap[npt + R:],
                          views["refcount"], views["free_list"], views["free_count"])

    def phase_score():
        # scoring, then the eviction lists every boundary request would use if
        # it compressed: both read keys and scores only
        gp.gp_boundary_score(kv, ps, q_pre, qstate, slots, positions, bnd, params, counts, scores, ws_s)
        gp.gp_boundary_select(*bargs)

    def phase_apply():
        gp.gp_boundary_decide(*bargs, hold=False)
        gp.gp_boundary_compact(*bargs)

    def phase_decide():
        gp.gp_boundary_decide(*bargs, hold=False)

    def phase_compact():
        gp.gp_boundary_compact(*bargs)

    side = torch.cuda.Stream()          # default priority, like the main stream
    phase = dict(pre=phase_pre, summaries=phase_summaries, decode=phase_decode, score=phase_score,
                 apply=phase_apply, decode_snapshot=phase_decode_snapshot,
                 decide=phase_decide, compact=phase_compact)

    def step(marks=None):
        """One step on the current stream.  Unless --serial, the summary
        update, scoring, selection and the decision run beside decode attention
        on a second stream (fork and join by stream waits, which graph capture
        records as dependencies): decode reads its own snapshot of the request
        metadata, which the decision does not touch.  The compaction waits for
        both."""
        cur = torch.cuda.current_stream()

        def mark(name):
            if marks is not None:
                e_ = torch.cuda.Event(enable_timing=True)
                e_.record(cur)
                marks[name].append(e_)

        phase["pre"]()
        if args.serial:
            phase["summaries"]()
            mark("d0")
            phase["decode"]()
            mark("d1")
            phase["score"]()
            phase["apply"]()
        else:
            # decode attention needs only the snapshot of the request metadata
            # (written by the restore): it forks right after it, beside the
            # summary update, scoring, selection and the decision.  The
            # layouts differ in the order of capture (the graph runs the first
            # branch captured on the launch queue) and in where the summary
            # update runs
            if args.layout == "summaries-first":
                phase["summaries"]()
            side.wait_stream(cur)

            def boundary_branch():
                with torch.cuda.stream(side):
                    if args.layout != "summaries-first":
                        phase["summaries"]()
                    phase["score"]()
                    phase["decide"]()

            if args.layout == "boundary-first":
                boundary_branch()
            mark("d0")
            phase["decode_snapshot"]()
            mark("d1")
            if args.layout != "boundary-first":
                boundary_branch()
            cur.wait_stream(side)
            phase["compact"]()
        mark("b1")

    # warm up every call (and the library's lazy state) eagerly first
    for _ in range(2):
        step()
    torch.cuda.synchronize()
    # steps per launch: with HIP graphs, S consecutive steps are captured into
    # one graph (as a serving loop captures its decode steps), so that the
    # graph's launch cost is paid once per S steps; every step still does all
    # of its work, the restore included
    S = 1 if args.eager else max(1, math.gcd(args.graph_steps, args.steps))
    if args.eager:
        run_step = step
    else:
        # S whole steps are one HIP graph: no launch gaps between their kernels
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(S):
                step()
        run_step = graph.replay

    for _ in range(max(1, args.warmup // S)):
        run_step()
    torch.cuda.synchronize()
    counters.zero_()
    # timed region: K whole steps (K / S launches), nothing else on the streams
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps // S):
        run_step()
    t1.record(stream)
    torch.cuda.synchronize()
    step_ms = t0.elapsed_time(t1) / args.steps
    split = counters.cpu().numpy().tolist()

    # decode attention alone: K back-to-back launches of the decode call on its
    # stream, bracketed by HIP events (the roofline's kernel timing)
    restore()
    torch.cuda.synchronize()
    k0 = torch.cuda.Event(enable_timing=True)
    k1 = torch.cuda.Event(enable_timing=True)
    k0.record(stream)
    for _ in range(args.steps):
        phase_decode()
    k1.record(stream)
    torch.cuda.synchronize()
    decode_ms = k0.elapsed_time(k1) / args.steps

    # the same call with the caches cold: a 512 MiB scratch write before each
    # launch evicts L2 and the 256 MB last-level cache, so no K/V byte can come
    # from an earlier call (context for the back-to-back figure above)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold = []
    for _ in range(args.steps):
        flush.fill_(1)
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        phase_decode()
        c1.record(stream)
        cold.append((c0, c1))
    torch.cuda.synchronize()
    cold_t = np.array([x.elapsed_time(y) for x, y in cold])
    decode_cold_ms = float(np.mean(cold_t))
    decode_cold_pct = [round(float(x), 4) for x in np.percentile(cold_t, [10, 50, 90])]
    del flush

    # streaming-read ceiling: the plain read kernel of the library over a
    # buffer far larger than the caches, K back-to-back launches
    ceil_buf = torch.ones(args.ceiling_mib << 20, dtype=torch.uint8, device=dev)
    ceil_out = torch.zeros(1, dtype=torch.int32, device=dev)
    for _ in range(2):
        gp.gp_stream_read(ceil_buf, ceil_out)
    torch.cuda.synchronize()
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(args.steps):
        gp.gp_stream_read(ceil_buf, ceil_out)
    c1.record(stream)
    torch.cuda.synchronize()
    ceiling_gbs = ceil_buf.numel() / (c0.elapsed_time(c1) / args.steps * 1e-3) / 1e9
    del ceil_buf, ceil_out

    # the summary update folded into decode attention (one launch) against the
    # two calls, K back-to-back launches each
    def timed_loop(fn):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    def fused_step():
        gp.gp_decode_step(kv, ps, q_post, q_pre, params.scale, out, slots, init, qstate,
                          params.beta_s, params.beta_l, ws_d)

    def separate_step():
        gp.gp_update_summaries(q_pre, slots, init, qstate, params.beta_s, params.beta_l)
        gp.gp_decode_attention(kv, ps, q_post, params.scale, out, ws_d)

    fused_ms = timed_loop(fused_step)
    separate_ms = timed_loop(separate_step)

    # the step's new token folded in as well (one launch: K/V append into the
    # pages, summaries, decode attention, lengths advanced) against the loop
    # prologue and decode attention as two launches; both restore the page
    # metadata and positions before each call so that every call does the same
    # work
    tok = W.step_inputs(w, 1, seed=1)[0]
    k_tok, v_tok = bf(tok["k_new"][0]), bf(tok["v_new"][0])
    pos0 = positions.clone()

    def token_fused():
        restore()
        positions.copy_(pos0)
        gp.gp_decode_step(kv, ps, q_post, q_pre, params.scale, out, slots, init, qstate,
                          params.beta_s, params.beta_l, ws_d, k_new=k_tok, v_new=v_tok, positions=positions)

    def token_separate():
        restore()
        positions.copy_(pos0)
        gp.gp_append_step([kv], ps, positions, k_tok[None], v_tok[None], q_pre[None], slots, init,
                          qstate[None], params.beta_s, params.beta_l)
        gp.gp_decode_attention(kv, ps, q_post, params.scale, out, ws_d)

    token_fused_ms = timed_loop(token_fused)
    token_separate_ms = timed_loop(token_separate)
    restore()
    positions.copy_(pos0)

    # a workload with a shared prefix: decode attention that reads the shared
    # pages once per block of requests (the prefix pass on a second stream
    # beside the private tails, then the merge), K back-to-back calls
    shared = None
    if prefix_pages:
        side2 = torch.cuda.Stream()

        def shared_call():
            cur = torch.cuda.current_stream()
            side2.wait_stream(cur)
            with torch.cuda.stream(side2):
                gp.gp_decode_attention_shared(kv, ps, q_post, params.scale, out, groups, ws_d,
                                              stages=gp.GP_DECODE_PREFIX)
            gp.gp_decode_attention_shared(kv, ps, q_post, params.scale, out, groups, ws_d,
                                          stages=gp.GP_DECODE_CHUNKS)
            cur.wait_stream(side2)
            gp.gp_decode_attention_shared(kv, ps, q_post, params.scale, out, groups, ws_d,
                                          stages=gp.GP_DECODE_MERGE)

        for _ in range(2):
            shared_call()
        shared_ms = timed_loop(shared_call)
        shared_one_ms = timed_loop(lambda: gp.gp_decode_attention_shared(kv, ps, q_post, params.scale, out,
                                                                        groups, ws_d))
        shared = {"ms": shared_ms, "one_stream_ms": shared_one_ms, "groups": groups}

    # instrumented pass (eager launches, events between phases): how much of a
    # step the boundary work adds after decode attention has finished
    marks = {"d0": [], "d1": [], "b1": []}
    for _ in range(args.steps):
        step(marks)
    torch.cuda.synchronize()
    boundary_ms = float(np.mean([a.elapsed_time(c) for a, c in zip(marks["d1"], marks["b1"])]))
    inline_decode_ms = float(np.mean([a.elapsed_time(c) for a, c in zip(marks["d0"], marks["d1"])]))

    # gp_boundary_apply alone with every boundary request compressing, in each
    # compaction layout: the method's stable shift and the hole-filling variant
    def apply_ms(layout):
        p = dataclasses.replace(params, tau=math.inf, layout=layout)
        ev = []
        for _ in range(args.steps):
            restore()
            phase_score()
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record(stream)
            gp.gp_boundary_apply([kv], ps, bnd, counts, scores, p, decisions, delta, counters, ws_a)
            a1.record(stream)
            ev.append((a0, a1))
        torch.cuda.synchronize()
        return float(np.mean([x.elapsed_time(y) for x, y in ev]))

    apply_layout_ms = {"shift": apply_ms(gp.GP_LAYOUT_SHIFT), "fill": apply_ms(gp.GP_LAYOUT_FILL)}

    # the boundary calls alone, on one stream, as the step runs them (scoring +
    # selection, then the decision + compaction), the state restored before
    # each iteration outside the events; medians over K iterations
    bev = []
    for _ in range(args.steps):
        restore()
        b0, b1, b2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        b0.record(stream)
        phase_score()
        b1.record(stream)
        phase_apply()
        b2.record(stream)
        bev.append((b0, b1, b2))
    torch.cuda.synchronize()
    t_score = float(np.median([x.elapsed_time(y) for x, y, _ in bev]))
    t_apply = float(np.median([y.elapsed_time(z) for _, y, z in bev]))
    bnd_np = np.asarray(w.boundary, dtype=np.int64)
    cand = int(((w.num_pages[bnd_np].astype(np.int64) - 1) * b).sum())
    score_bytes = cand * Hkv * d * e + cand * Hkv * 4         # K of every candidate once + the scores

    # the decode loop itself (App. E.3): every step appends each running
    # request's new token (K/V into its pages, one summary EMA step), decodes,
    # and takes the boundary event of every request whose pages are full.
    # "sync" decides and compacts before the next step; "async" leaves
    # compressing requests held for one step and runs their compaction on a
    # third stream beside the next step's append and decode.  Both start from
    # the same state and see the same seeded tokens; the W + K steps are two
    # HIP graphs (inputs picked by a device-side step counter).
    loop = serving_loops(args, gp, W, w, kv, ps, meta, meta0, qstate, slots, positions, params, k, v) \
        if args.loop_steps > 0 else None

    # algorithmic bytes
    m = w.seq_lens.astype(np.int64)
    decode_bytes = int(m.sum()) * Hkv * d * e * 2 + int(w.num_pages.sum()) * 4 + 2 * R * Hq * d * e
    summary_bytes = R * Hq * d * e + 2 * 2 * R * Hq * d * 4

    # resident (page, slot) pairs counted once: pages shared by a common prefix
    # are read by every request that holds them, but held in HBM once
    slots_all = np.concatenate([w.page_table[r][np.arange(int(w.seq_lens[r])) // b].astype(np.int64) * b
                                + np.arange(int(w.seq_lens[r])) % b for r in range(R)])
    unique_bytes = int(np.unique(slots_all).size) * Hkv * d * e * 2
    # the step's decode bytes: with a shared prefix, the shared pages once
    # (the call the step makes reads them once per block of requests)
    step_decode_bytes = (unique_bytes + decode_bytes - int(m.sum()) * Hkv * d * e * 2) if prefix_pages \
        else decode_bytes
    step_bytes = step_decode_bytes + summary_bytes
    gbs = step_bytes / (step_ms * 1e-3) / 1e9
    dec_gbs = decode_bytes / (decode_ms * 1e-3) / 1e9

    if shared is not None:
        sh_gbs = unique_bytes / (shared["ms"] * 1e-3) / 1e9
        shared = {"ms": round(shared["ms"], 4), "unique_GB/s": round(sh_gbs, 1),
                  "unique_hbm_frac": round(sh_gbs / HBM_PEAK_GBS, 4),
                  "one_stream_ms": round(shared["one_stream_ms"], 4),
                  "one_stream_unique_hbm_frac": round(unique_bytes / (shared["one_stream_ms"] * 1e-3) / 1e9
                                                      / HBM_PEAK_GBS, 4),
                  "plain_call_unique_hbm_frac": round(unique_bytes / (decode_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                  "groups": shared["groups"],
                  "note": "gp_decode_attention_shared: the prefix pass (shared pages read once per block of "
                          "requests, on the matrix cores) on a second stream beside the private tails, then "
                          "the merge; one_stream: the three stages in order on one stream, as the step "
                          "calls it"}
        # the step decodes with the one-stream shared call: it is the roofline's kernel here
        rf_bytes = step_decode_bytes
        rf_gbs = rf_bytes / (shared_one_ms * 1e-3) / 1e9
    else:
        rf_bytes, rf_gbs = decode_bytes, dec_gbs

    traffic = None
    if args.workload == "qwen3_8b" and os.path.exists(args.traffic_json):
        with open(args.traffic_json) as f:
            tj = json.load(f)
        if tj.get("kernel_source_hash") == _kernel_hash():
            traffic = tj.get("hbm_bytes_per_launch")

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src_t = torch.ones(n, dtype=torch.float32, device=dev)
        dst_t = torch.empty_like(src_t)
        for _ in range(2):
            dst_t.copy_(src_t)
        torch.cuda.synchronize()
        del src_t, dst_t

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w, args.workload, args.cpu_seconds)

    line = {
        "metric": "decode attn GB/s (% of HBM peak) + boundary events/s, " + WORKLOADS[args.workload][0],
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) K/V/q with 1% heavy keys; no model weights)",
        "config": {"workload": WORKLOADS[args.workload][1],
                   "resident_tokens": int(m.sum()), "boundary_requests": Rb},
        "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
        "launch": ("eager" if args.eager else f"one HIP graph per {S} step{'s' if S > 1 else ''}") +
                  ("" if args.serial else f", {args.layout}"),
        "decode_attention": {"ms": round(decode_ms, 4), "GB/s": round(dec_gbs, 1),
                             "hbm_frac": round(dec_gbs / HBM_PEAK_GBS, 4), "bytes": decode_bytes,
                             "unique_kv_bytes": unique_bytes, "step_decode_bytes": step_decode_bytes,
                             "ms_inside_step": round(inline_decode_ms, 4),
                             "ms_caches_flushed": round(decode_cold_ms, 4),
                             "ms_caches_flushed_p10_p50_p90": decode_cold_pct,
                             "with_summaries_one_launch_ms": round(fused_ms, 4),
                             "with_summaries_two_launches_ms": round(separate_ms, 4),
                             "with_token_and_summaries_one_launch_ms": round(token_fused_ms, 4),
                             "append_step_then_decode_two_launches_ms": round(token_separate_ms, 4),
                             "shared_prefix": shared},
        "boundary": {"ms_after_decode": round(boundary_ms, 4),
                     "events_per_s": round(Rb / (step_ms * 1e-3), 1),
                     "overlapped_with_decode": not args.serial,
                     "compress_grow_fallback_preempt": split,
                     "apply_ms_all_compress": {k_: round(v_, 4) for k_, v_ in apply_layout_ms.items()},
                     "alone": {"score_select_ms": round(t_score, 4), "decide_compact_ms": round(t_apply, 4),
                               "events_per_s": round(Rb / ((t_score + t_apply) * 1e-3), 1),
                               "score_bytes": score_bytes,
                               "score_GB/s": round(score_bytes / (t_score * 1e-3) / 1e9, 1)}},
        "serving_loop": loop,
        "roofline": {"bound": "hbm", "achieved": round(rf_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(rf_gbs / HBM_PEAK_GBS, 4), "traffic": traffic},
        "stream_read_ceiling": {"GB/s": round(ceiling_gbs, 1), "hbm_frac": round(ceiling_gbs / HBM_PEAK_GBS, 4),
                                "bytes": args.ceiling_mib << 20,
                                "decode_over_ceiling": round(dec_gbs / ceiling_gbs, 4),
                                "kernel": "gp_stream_read: one pass of non-temporal 16-byte loads, one "
                                          "contiguous chunk per workgroup, 16 loads in flight per thread, 8 "
                                          "workgroups of 256 per CU, per-workgroup partials folded by a "
                                          "one-workgroup kernel (the best of a sweep of grid-stride or "
                                          "contiguous chunks, 4/8/16 loads in flight, 4-64 workgroups per CU)"},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def serving_loops(args, gp, W, w, kv, ps, meta, meta0, qstate, slots, positions, params, k, v):
    """Times the decode loop synchronously and with asynchronous compaction,
    from the same starting state; returns the report object."""
    import torch

    dev = "cuda"
    R, Hq, Hkv, d = w.num_reqs, w.num_q_heads, w.num_kv_heads, w.head_dim
    n_warm, n_steps = max(args.warmup, 1), args.loop_steps
    S = n_warm + n_steps
    dt = torch.bfloat16
    inp = W.step_inputs(w, S, seed=0)

    def stack(key, layer0=False):
        a = np.stack([x[key][0] if layer0 else x[key] for x in inp])
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(dt).to(dev)

    k_all, v_all = stack("k_new", True), stack("v_new", True)          # [S][R][Hkv][d]
    qpre_all, qpost_all = stack("q_pre"), stack("q_post")              # [S][R][Hq][d]
    t_idx = torch.zeros(1, dtype=torch.int64, device=dev)
    bnd = torch.arange(R, dtype=torch.int32, device=dev)               # every request; kernels filter
    max_cand = (w.max_pages - 1) * w.page_size
    counts = torch.zeros((1, R, Hkv, 2), dtype=torch.int32, device=dev)
    scores = torch.zeros((1, R, Hkv, max_cand), device=dev)
    dec = torch.zeros(R, dtype=torch.int32, device=dev)
    delta = torch.zeros(R, device=dev)
    ctr = torch.zeros(4, dtype=torch.int64, device=dev)
    out = torch.empty((R, Hq, d), dtype=dt, device=dev)
    ws_d = gp.workspace(gp.GP_OP_DECODE, R, 0, Hq, Hkv, d, w.max_pages, dt)
    ws_s = gp.workspace(gp.GP_OP_SCORE, R, R, Hq, Hkv, d, w.max_pages, dt)
    ws_a = [gp.workspace(gp.GP_OP_APPLY, R, R, Hq, Hkv, d, w.max_pages, dt) for _ in range(2)]
    qstate5 = qstate.view(1, *qstate.shape)
    side_a, side_b = torch.cuda.Stream(), torch.cuda.Stream()

    # the starting state, restored before each variant
    snap = dict(meta=meta0.clone(), qstate=qstate.clone(), positions=positions.clone(), k=k.clone(),
                v=v.clone())

    def restore_all():
        meta.copy_(snap["meta"])
        qstate.copy_(snap["qstate"])
        positions.copy_(snap["positions"])
        k.copy_(snap["k"])
        v.copy_(snap["v"])
        ctr.zero_()
        t_idx.zero_()
        for x in ws_a:
            x.zero_()

    def one_step(async_, parity):
        cur = torch.cuda.current_stream()
        k_new = torch.index_select(k_all, 0, t_idx)                    # [1][R][Hkv][d]
        v_new = torch.index_select(v_all, 0, t_idx)
        q_pre = torch.index_select(qpre_all, 0, t_idx)                 # [1][R][Hq][d]
        q_post = torch.index_select(qpost_all, 0, t_idx)[0]
        gp.gp_append_step([kv], ps, positions, k_new, v_new, q_pre, slots, None, qstate5,
                          params.beta_s, params.beta_l)
        ws = ws_a[parity] if async_ else ws_a[0]
        bargs = ([kv], ps, bnd, counts, scores, params, dec, delta, ctr, ws)
        side_b.wait_stream(cur)
        with torch.cuda.stream(side_b):
            gp.gp_boundary_score(kv, ps, q_pre[0], qstate, slots, positions, bnd, params, counts[0],
                                 scores[0], ws_s)
            gp.gp_boundary_select(*bargs)
        gp.gp_decode_attention(kv, ps, q_post, params.scale, out, ws_d)
        cur.wait_stream(side_b)
        if async_:
            cur.wait_stream(side_a)                                     # the previous compaction
            gp.gp_release_held(ps)
            gp.gp_boundary_decide(*bargs, hold=True)
            side_a.wait_stream(cur)
            with torch.cuda.stream(side_a):
                gp.gp_boundary_compact(*bargs)
        else:
            gp.gp_boundary_decide(*bargs, hold=False)
            gp.gp_boundary_compact(*bargs)
        t_idx.add_(1)
        return k_new, v_new, q_pre, q_post

    def capture(n, async_):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            cur = torch.cuda.current_stream()
            side_a.wait_stream(cur)
            side_b.wait_stream(cur)
            # each step's inputs stay allocated until the capture ends, so no
            # later step reuses memory that a side-stream node still reads
            keep = [one_step(async_, j % 2) for j in range(n)]
            cur.wait_stream(side_a)
            cur.wait_stream(side_b)
        del keep
        return g

    res = {}
    for name, async_ in (("sync", False), ("async", True)):
        restore_all()
        torch.cuda.synchronize()
        g_warm, g_run = capture(n_warm, async_), capture(n_steps, async_)
        restore_all()
        torch.cuda.synchronize()
        g_warm.replay()
        torch.cuda.synchronize()
        pos0 = int(positions.sum().item())
        ctr0 = ctr.cpu().numpy().copy()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g_run.replay()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        tokens = int(positions.sum().item()) - pos0
        split = (ctr.cpu().numpy() - ctr0).tolist()
        res[name] = {"ms_per_step": round(ms / n_steps, 4), "tokens_per_s": round(tokens / (ms * 1e-3), 1),
                     "tokens": tokens, "boundary_events": int(sum(split)),
                     "compress_grow_fallback_preempt": split}
        del g_warm, g_run
    restore_all()
    torch.cuda.synchronize()
    del snap
    res["steps"] = n_steps
    res["async_speedup"] = round(res["async"]["tokens_per_s"] / res["sync"]["tokens_per_s"], 4)
    res["note"] = ("one layer of the workload run as a decode loop: per step, append "
                   "(new K/V into the pages, summary EMA), decode attention, and the boundary event of "
                   "every request whose pages are full; async holds compressing requests for one step "
                   "and overlaps their compaction with the next step (App. E.3)")
    return res


def _kernel_hash() -> str:
    import hashlib
    p = os.path.join(ROOT, "paper_2609_03494_amd", "csrc", "gp_decode.hip")
    with open(p, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def cpu_baseline(w, workload: str, budget_s: float):
    """The fp64 NumPy oracle on the host cores over the requests of the same
    workload in order, each call one BLAS thread: one thread in this process
    for half the time budget, then one worker process per host core (at most
    16, the host share of one GPU) for the other half, in a child process that
    never touches the GPU; plus one boundary-event scoring pass.  Reported as
    decode GB/s-equivalent; `value` is the all-core figure."""
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:           # pragma: no cover
        threadpool_limits = None
    import contextlib
    import subprocess
    import oracle as O

    class View:
        def __init__(self, data):
            self.data = data

        def __getitem__(self, pid):
            return self.data[w.page_row[int(pid)]]

    scale = 1.0 / math.sqrt(w.head_dim)
    kv_k, kv_v = View(w.k_data), View(w.v_data)
    ctx = threadpool_limits(limits=1) if threadpool_limits else contextlib.nullcontext()
    with ctx:
        t_start = time.perf_counter()
        done1, bytes1 = 0, 0
        while time.perf_counter() - t_start < budget_s / 2:
            r = done1 % w.num_reqs
            O.decode_attention(kv_k, kv_v, w.dtype, w.page_table, w.seq_lens, w.q_post, w.num_q_heads, scale,
                               requests=[r])
            bytes1 += int(w.seq_lens[r]) * w.num_kv_heads * w.head_dim * 2 * 2
            done1 += 1
        t1 = time.perf_counter() - t_start
        r = int(w.boundary[0])
        P = int(w.num_pages[r])
        te = time.perf_counter()
        toks = O.gather_tokens(kv_k, w.page_table[r], P * 16, 16)
        O.score_request(toks, w.dtype, P, 16, w.q_pre[r], w.qstate[w.slot_ids[r]], int(w.positions[r]),
                        O.Params().as_f32(w.head_dim), scale)
        t_evt = time.perf_counter() - te
    single = {"value": round(bytes1 / t1 / 1e9, 4), "unit": "GB/s", "cores": 1,
              "sample": f"{done1} request passes ({bytes1 / 1e6:.0f} MB of K/V) in {t1:.1f} s"}
    ncores = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count() or 1))
    env = dict(os.environ, OMP_NUM_THREADS="1", OPENBLAS_NUM_THREADS="1", MKL_NUM_THREADS="1")
    cp = subprocess.run([sys.executable, "-m", "oracle.cpu_baseline", workload, str(budget_s / 2), str(ncores)],
                        cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    res = json.loads(cp.stdout.strip().splitlines()[-1]) if cp.returncode == 0 else None
    if res is None:
        out = dict(single, kind="oracle", boundary_score_s_per_event=round(t_evt, 3),
                   sample=single["sample"] + f"; the all-core leg failed: {cp.stderr.strip()[-200:]}")
        return out
    return {"value": round(res["bytes"] / res["seconds"] / 1e9, 4), "unit": "GB/s", "cores": res["workers"],
            "kind": "oracle",
            "sample": f"decode attention of {res['passes']} request passes over the {w.num_reqs} requests in "
                      f"order ({res['bytes'] / 1e6:.0f} MB of K/V) in {res['seconds']:.1f} s on "
                      f"{res['workers']} worker processes (workload set-up excluded); one boundary scoring "
                      f"pass ({P} pages) in {t_evt:.2f} s",
            "single_thread": single,
            "boundary_score_s_per_event": round(t_evt, 3)}


if __name__ == "__main__":
    main()

"""All-core timing of the oracle's decode attention (test infrastructure: run
by the benchmark's CPU-baseline leg as a child process that never touches a
GPU, so that it may fork worker processes).

usage: python -m oracle.cpu_baseline WORKLOAD SECONDS WORKERS
Prints one JSON line: bytes of K/V read, request passes, seconds, workers.
Each worker runs the oracle unchanged, one BLAS thread, over the workload's
requests in order (worker k starts at request k and steps by WORKERS)."""
import json
import math
import multiprocessing as mp
import os
import sys
import time

_W = None


def _worker(args):
    k, nworkers, seconds, t0 = args
    import numpy as np  # noqa: F401
    try:
        from threadpoolctl import threadpool_limits
        ctx = threadpool_limits(limits=1)
    except ImportError:           # pragma: no cover
        import contextlib
        ctx = contextlib.nullcontext()
    from oracle import growpage_oracle as O
    w = _W

    class View:
        def __init__(self, data):
            self.data = data

        def __getitem__(self, pid):
            return self.data[w.page_row[int(pid)]]

    scale = 1.0 / math.sqrt(w.head_dim)
    kv_k, kv_v = View(w.k_data), View(w.v_data)
    done, nbytes, r = 0, 0, k
    with ctx:
        while time.time() - t0 < seconds:
            rr = r % w.num_reqs
            O.decode_attention(kv_k, kv_v, w.dtype, w.page_table, w.seq_lens, w.q_post, w.num_q_heads,
                               scale, requests=[rr])
            nbytes += int(w.seq_lens[rr]) * w.num_kv_heads * w.head_dim * 2 * 2
            done += 1
            r += nworkers
    return done, nbytes


def main():
    global _W
    name, seconds, nworkers = sys.argv[1], float(sys.argv[2]), int(sys.argv[3])
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import workloads as W
    _W = W.make(name)
    ctx = mp.get_context("fork")      # this process has never touched a GPU
    t0 = time.time()
    with ctx.Pool(nworkers) as pool:
        res = pool.map(_worker, [(k, nworkers, seconds, t0) for k in range(nworkers)])
    dt = time.time() - t0
    print(json.dumps({"bytes": sum(b for _, b in res), "passes": sum(d for d, _ in res), "seconds": dt,
                      "workers": nworkers}), flush=True)


if __name__ == "__main__":
    main()

"""Test-side helpers: move a seeded workload onto the GPU, run the library's
entry points on it, and bring results back as NumPy arrays; plus the
comparison rules shared by the parity tests.

Nothing here computes any part of the method: the HIP library does on one
side and the oracle on the other."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
import paper_2609_03494_amd as gp
import workloads as W

DEV = "cuda"
# floor of the element-wise fp32 decode bar, relative to sum_i a_i |v_i,d|:
# 2^-18 = 64 units of float32 rounding, the worst-case error of a sequential
# fp32 sum of 64 terms (the kernels sum at most a page of tokens per lane and
# step, over at most a few dozen steps, and merge partials in short trees)
FP32_FLOOR = 2.0 ** -18


def torch_dtype(w: W.Workload):
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def to_torch(arr: np.ndarray, dtype_name: str, device=DEV) -> torch.Tensor:
    if dtype_name == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)


def to_numpy(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


class PoolView:
    """Pool pages of a workload indexed by physical id (content rows only)."""

    def __init__(self, w: W.Workload, which: str):
        self.w, self.data = w, (w.k_data if which == "k" else w.v_data)

    def __getitem__(self, pid):
        row = self.w.page_row[int(pid)]
        assert row >= 0, f"page {pid} has no content"
        return self.data[row]


def oracle_state(w: W.Workload) -> O.PageState:
    return O.PageState(w.page_table.copy(), w.num_pages.copy(), w.seq_lens.copy(),
                       w.refcount.copy(), w.free_list.copy(), int(w.free_count))


POLICY_CODES = {"growpage": gp.GP_POLICY_GROWPAGE, "fixed": gp.GP_POLICY_FIXED,
                "random": gp.GP_POLICY_RANDOM, "inverse": gp.GP_POLICY_INVERSE,
                "shrink": gp.GP_POLICY_SHRINK}
METRIC_CODES = {"top_p": gp.GP_METRIC_TOP_P, "entropy": gp.GP_METRIC_ENTROPY}
LAYOUT_CODES = {"shift": gp.GP_LAYOUT_SHIFT, "fill": gp.GP_LAYOUT_FILL}


def library_params(params: O.Params, head_dim: int, draws=None) -> "gp.Params":
    """The oracle's constants, rounded to float32, as the library's struct;
    draws (host float32 [num_bnd]) are copied to the device."""
    p32 = params.as_f32(head_dim)
    d = None if draws is None else torch.from_numpy(np.asarray(draws, np.float32)).to(DEV)
    return gp.Params(p32.beta_s, p32.beta_l, p32.p, p32.tau, p32.scale, p32.rope_theta, p32.k_loc,
                     p32.reserve_pages, POLICY_CODES[p32.policy], METRIC_CODES[p32.metric],
                     p32.fixed_pages, p32.min_capacity_pages, p32.compress_prob, p32.shrink_threshold, d,
                     LAYOUT_CODES[p32.layout])


class DeviceCase:
    """One workload resident on the GPU, with the library's workspaces."""

    def __init__(self, w: W.Workload, poison_free_pages: bool = True, n_layers: int = 1,
                 distinct_layers: bool = False):
        """n_layers K/V pools; with distinct_layers layer l holds the contents of
        W.layer_variant(w, l) (otherwise every layer a copy of w's)."""
        self.w = w
        dt = torch_dtype(w)
        shape = (w.pool_pages, w.num_kv_heads, w.page_size, w.head_dim)
        self.layers = []
        self.layer_workloads = [W.layer_variant(w, l) if distinct_layers else w for l in range(n_layers)]
        for wl in self.layer_workloads:
            k = torch.empty(shape, dtype=dt, device=DEV)
            v = torch.empty(shape, dtype=dt, device=DEV)
            if poison_free_pages:
                k.fill_(float("nan"))
                v.fill_(float("nan"))
            ids = np.nonzero(w.page_row >= 0)[0]
            idx = torch.from_numpy(ids.astype(np.int64)).to(DEV)
            rows = w.page_row[ids]
            k.index_copy_(0, idx, to_torch(wl.k_data[rows], w.dtype))
            v.index_copy_(0, idx, to_torch(wl.v_data[rows], w.dtype))
            self.layers.append(gp.KVLayer(k, v))
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(DEV)
        self.ps = gp.PageState(i32(w.page_table), i32(w.num_pages), i32(w.seq_lens),
                               i32(w.refcount), i32(w.free_list), i32([w.free_count]))
        self.positions = i32(w.positions)
        self.slot_ids = i32(w.slot_ids)
        self.qstate = torch.from_numpy(w.qstate.copy()).to(DEV)
        self.q_pre = to_torch(w.q_pre, w.dtype)
        self.q_post = to_torch(w.q_post, w.dtype)
        self.n_layers = n_layers
        # per-layer queries and summary pools (layer 0: the ones above)
        self.q_pre_layers = [self.q_pre] + [to_torch(wl.q_pre, w.dtype) for wl in self.layer_workloads[1:]]
        self.qstate_layers = [self.qstate] + [torch.from_numpy(wl.qstate.copy()).to(DEV)
                                              for wl in self.layer_workloads[1:]]
        R, Hq, Hkv, d, maxp = w.num_reqs, w.num_q_heads, w.num_kv_heads, w.head_dim, w.max_pages
        self.ws_decode = gp.workspace(gp.GP_OP_DECODE, R, 0, Hq, Hkv, d, maxp, dt)

    # ------------------------------------------------------------------ A1
    def update_summaries(self, q_pre: np.ndarray, init, beta_s: float, beta_l: float):
        q = to_torch(q_pre, self.w.dtype)
        ini = torch.from_numpy(np.asarray(init, np.uint8)).to(DEV)
        gp.gp_update_summaries(q, self.slot_ids, ini, self.qstate, beta_s, beta_l)

    # ------------------------------------------------------------------ A2
    def decode(self, scale: float, layer: int = 0) -> np.ndarray:
        out = torch.empty_like(self.q_post)
        gp.gp_decode_attention(self.layers[layer], self.ps, self.q_post, scale, out, self.ws_decode)
        torch.cuda.synchronize()
        return O.widen(to_numpy(out), self.w.dtype)

    # ------------------------------------------------------------- A3..A9
    def boundary(self, params: O.Params, bnd=None, q_pre_layers=None, qstate_layers=None, draws=None):
        w = self.w
        bnd = w.boundary if bnd is None else np.asarray(bnd, np.int32)
        Rb = int(bnd.shape[0])
        dt = torch_dtype(w)
        gparams = library_params(params, w.head_dim, draws)
        max_cand = (w.max_pages - 1) * w.page_size
        L = self.n_layers
        bnd_t = torch.from_numpy(bnd.astype(np.int32)).to(DEV)
        k_counts = torch.full((L, Rb, w.num_kv_heads, 2), -7, dtype=torch.int32, device=DEV)
        scores = torch.full((L, Rb, w.num_kv_heads, max(max_cand, 4)), -1.0, device=DEV)
        ws_s = gp.workspace(gp.GP_OP_SCORE, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads,
                            w.head_dim, w.max_pages, dt)
        ws_a = gp.workspace(gp.GP_OP_APPLY, w.num_reqs, Rb, w.num_q_heads, w.num_kv_heads,
                            w.head_dim, w.max_pages, dt, n_layers=L)
        for ell in range(L):
            qp = self.q_pre_layers[ell] if q_pre_layers is None else q_pre_layers[ell]
            qs = self.qstate_layers[ell] if qstate_layers is None else qstate_layers[ell]
            gp.gp_boundary_score(self.layers[ell], self.ps, qp, qs, self.slot_ids, self.positions,
                                 bnd_t, gparams, k_counts[ell], scores[ell], ws_s)
        decisions = torch.full((Rb,), -1, dtype=torch.int32, device=DEV)
        delta = torch.full((Rb,), float("nan"), device=DEV)
        counters = torch.zeros(4, dtype=torch.int64, device=DEV)
        gp.gp_boundary_apply(self.layers, self.ps, bnd_t, k_counts, scores, gparams, decisions,
                             delta, counters, ws_a)
        torch.cuda.synchronize()
        return dict(k_counts=k_counts.cpu().numpy(), scores=scores.cpu().numpy(),
                    decisions=decisions.cpu().numpy(), delta=delta.cpu().numpy(),
                    counters=counters.cpu().numpy())

    def host_state(self) -> O.PageState:
        fc = int(self.ps.free_count.cpu().item())
        return O.PageState(self.ps.page_table.cpu().numpy(), self.ps.num_pages.cpu().numpy(),
                           self.ps.seq_lens.cpu().numpy(), self.ps.refcount.cpu().numpy(),
                           self.ps.free_list.cpu().numpy(), fc)

    def gather(self, table_row: np.ndarray, n: int, which: str, layer: int = 0) -> np.ndarray:
        """Logical tokens [0, n) of one request through a page-table row: [n, Hkv, d]."""
        pool = self.layers[layer].k if which == "k" else self.layers[layer].v
        ids = torch.from_numpy(np.asarray(table_row[: (n + 15) // 16], np.int64)).to(DEV)
        pages = to_numpy(pool.index_select(0, ids))
        tok = pages.transpose(0, 2, 1, 3).reshape(-1, pages.shape[1], pages.shape[3])
        return tok[:n]


# ---------------------------------------------------------------- rules ----

def assert_rows_close(got: np.ndarray, ref: np.ndarray, rtol: float, what: str):
    """Every output row (last axis) within rtol of the row's largest |value|."""
    scale = np.maximum(np.abs(ref).max(axis=-1, keepdims=True), 1e-30)
    err = np.abs(got - ref) / scale
    worst = float(np.nanmax(err)) if err.size else 0.0
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    assert worst <= rtol, f"{what}: worst row-relative error {worst:.3e} > {rtol:.1e}"
    return worst


class AbsPool:
    """|values| of a pool view: decode attention over it gives, per output
    element, sum_i a_i |v_i,d|, the magnitude at which the fp32 sums of that
    element round."""

    def __init__(self, view):
        self.view = view

    def __getitem__(self, pid):
        return np.abs(self.view[pid])


def fp32_elementwise_ok(got: np.ndarray, ref: np.ndarray, ref_abs: np.ndarray, rtol: float = 1e-5,
                        floor: float = FP32_FLOOR) -> bool:
    """Element-wise fp32 bar: |got - ref| <= rtol |ref| + floor * sum_i a_i |v_i,d|.
    The floor term is the rounding scale of the weighted sum that produces the
    element (a sum over the resident tokens of terms of size a_i |v_i,d|); it
    keeps elements that nearly cancel from demanding more than fp32 can give."""
    return bool((np.abs(got - ref) <= rtol * np.abs(ref) + floor * ref_abs).all())


def bf16_rounding_ok(got: np.ndarray, ref: np.ndarray, extra: float = 1e-5) -> bool:
    """|got - ref| within half a bfloat16 step of ref plus a small fp32 term."""
    scale = np.abs(ref).max(axis=-1, keepdims=True)
    return bool((np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + extra * scale).all())


def row_index(before: np.ndarray, after: np.ndarray) -> np.ndarray:
    """For each row of ``after`` the index of the identical row of ``before``
    (rows are random vectors, so they are unique); -1 if absent."""
    lut = {before[i].tobytes(): i for i in range(before.shape[0])}
    return np.array([lut.get(after[i].tobytes(), -1) for i in range(after.shape[0])])


def threshold_band(s32: np.ndarray, kept: np.ndarray, P: int, b: int, k_loc: int,
                   rel: float = 1e-5) -> set:
    """Candidates whose score lies within rel of the selection threshold (the
    best evicted non-local score and the worst kept one); a swap among them is
    excused."""
    C = (P - 1) * b
    ev = np.setdiff1d(np.arange(C), kept)
    if ev.size == 0:
        return set()
    theta = float(np.max(s32[ev]))
    band = np.nonzero(np.abs(s32.astype(np.float64) - theta) <= rel * max(theta, 1e-300))[0]
    return set(band.tolist())

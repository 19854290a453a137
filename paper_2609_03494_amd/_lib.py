"""ctypes binding of libgrowpage.so (include/growpage.h).

Argument marshalling only: tensors become device pointers, the current torch
stream becomes the HIP stream, and a non-zero status becomes GrowPageError.
Every step of the computation runs in the library's HIP kernels.  If the
library has not been built, importing a function raises instead of falling
back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgrowpage.so")

GP_F32, GP_BF16 = 0, 1
GP_OP_DECODE, GP_OP_SCORE, GP_OP_APPLY = 0, 1, 2
GP_COMPRESS, GP_GROW, GP_FALLBACK, GP_PREEMPT, GP_NOT_BOUNDARY = 0, 1, 2, 3, 4
GP_SHRINK = 5
GP_POLICY_GROWPAGE, GP_POLICY_FIXED, GP_POLICY_RANDOM, GP_POLICY_INVERSE, GP_POLICY_SHRINK = 0, 1, 2, 3, 4
GP_METRIC_TOP_P, GP_METRIC_ENTROPY = 0, 1
GP_DECODE_CHUNKS, GP_DECODE_MERGE, GP_DECODE_PREFIX = 1, 2, 4
GP_LAYOUT_SHIFT, GP_LAYOUT_FILL = 0, 1
GP_SCORE_WEIGHTS, GP_SCORE_COUNTS = 1, 2
PAGE_SIZE = 16
GP_ERR_SCRATCH = 5

EXPORTS = ("gp_update_summaries", "gp_decode_attention", "gp_decode_attention_noalloc", "gp_decode_attention_shared",
           "gp_decode_attention_stages", "gp_decode_step", "gp_boundary_score", "gp_boundary_score_stages",
           "gp_boundary_apply", "gp_boundary_select", "gp_boundary_decide", "gp_boundary_compact",
           "gp_release_held", "gp_append_step", "gp_workspace_bytes", "gp_status_string", "gp_stream_read")


class GrowPageError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: status {status} ({status_string(status)})")
        self.status = status


class _KVLayer(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("pool_pages", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int)]


class _PageState(ctypes.Structure):
    _fields_ = [("page_table", ctypes.c_void_p), ("num_pages", ctypes.c_void_p),
                ("seq_lens", ctypes.c_void_p), ("refcount", ctypes.c_void_p),
                ("free_list", ctypes.c_void_p), ("free_count", ctypes.c_void_p),
                ("num_reqs", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("pool_pages", ctypes.c_int32)]


class _PrefixGroup(ctypes.Structure):
    _fields_ = [("first_req", ctypes.c_int32), ("num_reqs", ctypes.c_int32), ("prefix_pages", ctypes.c_int32)]


class _Params(ctypes.Structure):
    _fields_ = [("beta_s", ctypes.c_float), ("beta_l", ctypes.c_float), ("p", ctypes.c_float),
                ("tau", ctypes.c_float), ("scale", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("k_loc", ctypes.c_int32), ("reserve_pages", ctypes.c_int32),
                ("policy", ctypes.c_int32), ("metric", ctypes.c_int32), ("fixed_pages", ctypes.c_int32),
                ("min_capacity_pages", ctypes.c_int32), ("compress_prob", ctypes.c_float),
                ("shrink_threshold", ctypes.c_float), ("draws", ctypes.c_void_p), ("layout", ctypes.c_int32),
                ("select_skip_grows", ctypes.c_int32)]


_lib = None


def load() -> ctypes.CDLL:
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_03494_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    lib.gp_status_string.restype = ctypes.c_char_p
    lib.gp_status_string.argtypes = [ctypes.c_int]
    lib.gp_workspace_bytes.restype = sz
    lib.gp_workspace_bytes.argtypes = [i32] * 8 + [ctypes.c_int, i32]
    lib.gp_stream_read.restype = ctypes.c_int
    lib.gp_stream_read.argtypes = [vp, sz, vp, vp]
    lib.gp_update_summaries.restype = ctypes.c_int
    lib.gp_update_summaries.argtypes = [vp, ctypes.c_int, i32, i32, i32, vp, vp, vp, i32, f32, f32, vp]
    lib.gp_decode_attention.restype = ctypes.c_int
    lib.gp_decode_attention.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp, i32,
                                        f32, vp, vp, sz, vp]
    lib.gp_decode_attention_noalloc.restype = ctypes.c_int
    lib.gp_decode_attention_noalloc.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp,
                                                i32, f32, vp, vp]
    lib.gp_decode_attention_shared.restype = ctypes.c_int
    lib.gp_decode_attention_shared.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp, i32,
                                               f32, vp, ctypes.POINTER(_PrefixGroup), i32, i32, vp, sz, vp]
    lib.gp_decode_attention_stages.restype = ctypes.c_int
    lib.gp_decode_attention_stages.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp, i32,
                                               f32, vp, i32, vp, sz, vp]
    lib.gp_decode_step.restype = ctypes.c_int
    lib.gp_decode_step.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp, vp, i32, f32,
                                   vp, vp, vp, vp, i32, f32, f32, vp, vp, vp, i32, vp, sz, vp]
    lib.gp_boundary_score.restype = ctypes.c_int
    lib.gp_boundary_score.argtypes = [ctypes.POINTER(_KVLayer), ctypes.POINTER(_PageState), vp, vp, i32,
                                      vp, vp, vp, i32, i32, ctypes.POINTER(_Params), vp, vp, i32, vp,
                                      sz, vp]
    lib.gp_boundary_score_stages.restype = ctypes.c_int
    lib.gp_boundary_score_stages.argtypes = lib.gp_boundary_score.argtypes + [i32]
    lib.gp_boundary_apply.restype = ctypes.c_int
    apply_args = [ctypes.POINTER(_KVLayer), i32, ctypes.POINTER(_PageState), vp, i32,
                  vp, vp, i32, ctypes.POINTER(_Params), vp, vp, vp, vp, sz, vp]
    for name in ("gp_boundary_apply", "gp_boundary_select", "gp_boundary_compact"):
        getattr(lib, name).restype = ctypes.c_int
        getattr(lib, name).argtypes = apply_args
    lib.gp_boundary_decide.restype = ctypes.c_int
    lib.gp_boundary_decide.argtypes = apply_args + [i32]
    lib.gp_release_held.restype = ctypes.c_int
    lib.gp_release_held.argtypes = [ctypes.POINTER(_PageState), vp]
    lib.gp_append_step.restype = ctypes.c_int
    lib.gp_append_step.argtypes = [ctypes.POINTER(_KVLayer), i32, ctypes.POINTER(_PageState), vp, vp, vp, vp,
                                   i32, vp, vp, vp, i32, f32, f32, vp]
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().gp_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != 0:
        raise GrowPageError(status, where)


def _ptr(t: torch.Tensor | None) -> int | None:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GP_F32
    if t.dtype == torch.bfloat16:
        return GP_BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


@dataclass
class KVLayer:
    """K and V pools [pool_pages, num_kv_heads, 16, head_dim] (float32 or bfloat16)."""
    k: torch.Tensor
    v: torch.Tensor

    def c(self) -> _KVLayer:
        pool, hkv, b, d = self.k.shape
        return _KVLayer(_ptr(self.k), _ptr(self.v), pool, hkv, b, d, _dtype_code(self.k))


@dataclass
class PageState:
    """Device page state (int32 tensors).  free_count is a one-element tensor."""
    page_table: torch.Tensor   # [R, max_pages]
    num_pages: torch.Tensor    # [R]
    seq_lens: torch.Tensor     # [R]
    refcount: torch.Tensor     # [pool_pages]
    free_list: torch.Tensor    # [pool_pages]
    free_count: torch.Tensor   # [1]

    def c(self) -> _PageState:
        R, maxp = self.page_table.shape
        return _PageState(_ptr(self.page_table), _ptr(self.num_pages), _ptr(self.seq_lens),
                          _ptr(self.refcount), _ptr(self.free_list), _ptr(self.free_count),
                          R, maxp, self.refcount.shape[0])


@dataclass
class Params:
    beta_s: float = 0.9
    beta_l: float = 0.999
    p: float = 0.99
    tau: float = 0.0
    scale: float = 1.0 / 128 ** 0.5
    rope_theta: float = 1.0e6
    k_loc: int = 4
    reserve_pages: int = 0
    policy: int = 0                 # GP_POLICY_*
    metric: int = 0                 # GP_METRIC_*
    fixed_pages: int = 256
    min_capacity_pages: int = 64
    compress_prob: float = 0.7
    shrink_threshold: float = -0.005
    draws: torch.Tensor | None = None   # [num_bnd] float32 on the device (RANDOM only)
    layout: int = 0                 # GP_LAYOUT_*
    select_skip_grows: int = 0      # gp_boundary_select: k_counts are final (see the header)

    def c(self) -> _Params:
        if self.draws is not None and (self.draws.dtype != torch.float32 or not self.draws.is_contiguous()):
            raise ValueError("draws must be a contiguous float32 tensor")
        return _Params(self.beta_s, self.beta_l, self.p, self.tau, self.scale, self.rope_theta,
                       self.k_loc, self.reserve_pages, self.policy, self.metric, self.fixed_pages,
                       self.min_capacity_pages, self.compress_prob, self.shrink_threshold,
                       _ptr(self.draws), self.layout, self.select_skip_grows)


def gp_workspace_bytes(op: int, num_reqs: int, num_bnd: int, num_q_heads: int, num_kv_heads: int,
                       head_dim: int, max_pages: int, dtype: torch.dtype, n_layers: int = 1) -> int:
    code = GP_F32 if dtype == torch.float32 else GP_BF16
    n = load().gp_workspace_bytes(op, num_reqs, num_bnd, num_q_heads, num_kv_heads, head_dim,
                                  max_pages, PAGE_SIZE, code, n_layers)
    if n == 0:
        raise GrowPageError(2, "gp_workspace_bytes")
    return int(n)


def workspace(op: int, num_reqs: int, num_bnd: int, num_q_heads: int, num_kv_heads: int,
              head_dim: int, max_pages: int, dtype: torch.dtype, n_layers: int = 1,
              device="cuda") -> torch.Tensor:
    """A zero-filled workspace of the size the library asks for."""
    n = gp_workspace_bytes(op, num_reqs, num_bnd, num_q_heads, num_kv_heads, head_dim, max_pages,
                           dtype, n_layers)
    return torch.zeros(n, dtype=torch.uint8, device=device)


def gp_update_summaries(q_pre: torch.Tensor, slot_ids: torch.Tensor, init: torch.Tensor,
                        qstate: torch.Tensor, beta_s: float, beta_l: float, stream=None) -> None:
    R, Hq, d = q_pre.shape
    st = load().gp_update_summaries(_ptr(q_pre), _dtype_code(q_pre), R, Hq, d, _ptr(slot_ids),
                                    _ptr(init), _ptr(qstate), qstate.shape[0], beta_s, beta_l,
                                    _stream(stream))
    _check(st, "gp_update_summaries")


def gp_decode_attention(kv: KVLayer, ps: PageState, q_post: torch.Tensor, scale: float,
                        out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    c_kv, c_ps = kv.c(), ps.c()
    st = load().gp_decode_attention(ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_post),
                                    q_post.shape[1], scale, _ptr(out), _ptr(ws), ws.numel(),
                                    _stream(stream))
    _check(st, "gp_decode_attention")


def gp_stream_read(src: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """The streaming-read reference kernel over src's bytes (XOR into out[0],
    an int32 device tensor)."""
    st = load().gp_stream_read(_ptr(src), src.numel() * src.element_size(), _ptr(out), _stream(stream))
    _check(st, "gp_stream_read")


def gp_decode_attention_noalloc(kv: KVLayer, ps: PageState, q_post: torch.Tensor, scale: float,
                                out: torch.Tensor, stream=None) -> None:
    """gp_decode_attention with its partials in the library's static scratch
    (no workspace, nothing allocated)."""
    c_kv, c_ps = kv.c(), ps.c()
    st = load().gp_decode_attention_noalloc(ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_post),
                                            q_post.shape[1], scale, _ptr(out), _stream(stream))
    _check(st, "gp_decode_attention_noalloc")


def gp_decode_attention_shared(kv: KVLayer, ps: PageState, q_post: torch.Tensor, scale: float,
                               out: torch.Tensor, groups, ws: torch.Tensor,
                               stages: int = GP_DECODE_PREFIX | GP_DECODE_CHUNKS | GP_DECODE_MERGE,
                               stream=None) -> None:
    """Decode attention with shared-prefix groups: ``groups`` is a list of
    (first_req, num_reqs, prefix_pages); ``stages`` any of GP_DECODE_PREFIX,
    GP_DECODE_CHUNKS, GP_DECODE_MERGE."""
    arr = (_PrefixGroup * max(len(groups), 1))(*[_PrefixGroup(*map(int, g)) for g in groups])
    c_kv, c_ps = kv.c(), ps.c()
    st = load().gp_decode_attention_shared(ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_post),
                                           q_post.shape[1], scale, _ptr(out), arr, len(groups), int(stages),
                                           _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "gp_decode_attention_shared")


def gp_decode_attention_stages(kv: KVLayer, ps: PageState, q_post: torch.Tensor, scale: float,
                               out: torch.Tensor, stages: int, ws: torch.Tensor, stream=None) -> None:
    """Decode attention's chunk pass (GP_DECODE_CHUNKS) and/or merge (GP_DECODE_MERGE)."""
    c_kv, c_ps = kv.c(), ps.c()
    st = load().gp_decode_attention_stages(ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_post),
                                           q_post.shape[1], scale, _ptr(out), stages, _ptr(ws), ws.numel(),
                                           _stream(stream))
    _check(st, "gp_decode_attention_stages")


def gp_decode_step(kv: KVLayer, ps: PageState, q_post: torch.Tensor, q_pre: torch.Tensor, scale: float,
                   out: torch.Tensor, slot_ids: torch.Tensor, init: torch.Tensor, qstate: torch.Tensor,
                   beta_s: float, beta_l: float, ws: torch.Tensor, k_new: torch.Tensor | None = None,
                   v_new: torch.Tensor | None = None, positions: torch.Tensor | None = None,
                   advance: bool = True, stream=None) -> None:
    """The step's new token (k_new, v_new [R][Hkv][d], optional), the summary
    update and decode attention in one launch."""
    c_kv, c_ps = kv.c(), ps.c()
    st = load().gp_decode_step(ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_post), _ptr(q_pre),
                               q_post.shape[1], scale, _ptr(out), _ptr(slot_ids), _ptr(init),
                               _ptr(qstate), qstate.shape[0], beta_s, beta_l, _ptr(k_new), _ptr(v_new),
                               _ptr(positions), int(bool(advance)), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "gp_decode_step")


def gp_boundary_score(kv: KVLayer, ps: PageState, q_pre: torch.Tensor, qstate: torch.Tensor,
                      slot_ids: torch.Tensor, positions: torch.Tensor, bnd: torch.Tensor,
                      params: Params, k_counts: torch.Tensor, scores: torch.Tensor,
                      ws: torch.Tensor, stream=None, stages=None) -> None:
    """stages None: gp_boundary_score; else gp_boundary_score_stages with that
    mask (GP_SCORE_WEIGHTS, GP_SCORE_COUNTS)."""
    c_kv, c_ps, c_p = kv.c(), ps.c(), params.c()
    args = (ctypes.byref(c_kv), ctypes.byref(c_ps), _ptr(q_pre), _ptr(qstate), qstate.shape[0], _ptr(slot_ids),
            _ptr(positions), _ptr(bnd), bnd.shape[0], q_pre.shape[1], ctypes.byref(c_p), _ptr(k_counts),
            _ptr(scores), scores.shape[-1], _ptr(ws), ws.numel(), _stream(stream))
    if stages is None:
        _check(load().gp_boundary_score(*args), "gp_boundary_score")
    else:
        _check(load().gp_boundary_score_stages(*args, stages), "gp_boundary_score_stages")


def _apply_like(name, layers, ps, bnd, k_counts, scores, params, decisions, delta, counters, ws, stream,
                *extra) -> None:
    arr = (_KVLayer * len(layers))(*[layer.c() for layer in layers])
    c_ps, c_p = ps.c(), params.c()
    st = getattr(load(), name)(arr, len(layers), ctypes.byref(c_ps), _ptr(bnd), bnd.shape[0],
                               _ptr(k_counts), _ptr(scores), scores.shape[-1], ctypes.byref(c_p),
                               _ptr(decisions), _ptr(delta), _ptr(counters), _ptr(ws),
                               ws.numel(), _stream(stream), *extra)
    _check(st, name)


def gp_boundary_apply(layers: list[KVLayer], ps: PageState, bnd: torch.Tensor,
                      k_counts: torch.Tensor, scores: torch.Tensor, params: Params,
                      decisions: torch.Tensor, delta: torch.Tensor, counters: torch.Tensor,
                      ws: torch.Tensor, stream=None) -> None:
    _apply_like("gp_boundary_apply", layers, ps, bnd, k_counts, scores, params, decisions, delta, counters,
                ws, stream)


def gp_boundary_select(layers, ps, bnd, k_counts, scores, params, decisions, delta, counters, ws,
                       stream=None) -> None:
    """First part of gp_boundary_apply: eviction lists and saved rows (workspace only)."""
    _apply_like("gp_boundary_select", layers, ps, bnd, k_counts, scores, params, decisions, delta, counters,
                ws, stream)


def gp_boundary_decide(layers, ps, bnd, k_counts, scores, params, decisions, delta, counters, ws,
                       hold: bool = False, stream=None) -> None:
    """Second part: decisions and page metadata; hold=True leaves compressing requests held."""
    _apply_like("gp_boundary_decide", layers, ps, bnd, k_counts, scores, params, decisions, delta, counters,
                ws, stream, int(bool(hold)))


def gp_boundary_compact(layers, ps, bnd, k_counts, scores, params, decisions, delta, counters, ws,
                        stream=None) -> None:
    """Third part: compaction and the release of freed pages."""
    _apply_like("gp_boundary_compact", layers, ps, bnd, k_counts, scores, params, decisions, delta, counters,
                ws, stream)


def gp_release_held(ps: PageState, stream=None) -> None:
    c_ps = ps.c()
    _check(load().gp_release_held(ctypes.byref(c_ps), _stream(stream)), "gp_release_held")


def gp_append_step(layers: list[KVLayer], ps: PageState, positions: torch.Tensor, k_new: torch.Tensor,
                   v_new: torch.Tensor, q_pre: torch.Tensor, slot_ids: torch.Tensor, init: torch.Tensor | None,
                   qstate: torch.Tensor, beta_s: float, beta_l: float, stream=None) -> None:
    """k_new, v_new [L][R][Hkv][d]; q_pre [L][R][Hq][d]; qstate [L][M][2][Hq][d]."""
    L = len(layers)
    if k_new.dim() != 4 or k_new.shape[0] != L or q_pre.dim() != 4 or qstate.dim() != 5:
        raise ValueError("gp_append_step: k_new/v_new [L,R,Hkv,d], q_pre [L,R,Hq,d], qstate [L,M,2,Hq,d]")
    arr = (_KVLayer * L)(*[layer.c() for layer in layers])
    c_ps = ps.c()
    st = load().gp_append_step(arr, L, ctypes.byref(c_ps), _ptr(positions), _ptr(k_new), _ptr(v_new),
                               _ptr(q_pre), q_pre.shape[2], _ptr(slot_ids), _ptr(init), _ptr(qstate),
                               qstate.shape[1], float(beta_s), float(beta_l), _stream(stream))
    _check(st, "gp_append_step")

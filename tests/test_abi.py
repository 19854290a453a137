"""The C-ABI library loads on the host and exports every entry point the header
declares; host-side validation answers without touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2609_03494_amd as gp
from paper_2609_03494_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_03494_amd import build
        build.build()
    return gp.load()


def _declared():
    with open(os.path.join(ROOT, "include", "growpage.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(gp_\w+)\s*\(", text, re.M)))


def test_header_declares_the_four_path_calls():
    names = _declared()
    for n in ("gp_update_summaries", "gp_decode_attention", "gp_boundary_score", "gp_boundary_apply"):
        assert n in names
    assert set(names) == set(_lib.EXPORTS)


def test_every_declared_symbol_is_exported(lib):
    for name in _declared():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in range(6):
        assert gp.status_string(code)


def test_workspace_sizes(lib):
    import torch
    n = gp.gp_workspace_bytes(gp.GP_OP_DECODE, 64, 0, 32, 8, 128, 260, torch.bfloat16)
    assert n > 64 * 8 * 4
    assert gp.gp_workspace_bytes(gp.GP_OP_SCORE, 64, 4, 32, 8, 128, 260, torch.bfloat16) > 0
    assert gp.gp_workspace_bytes(gp.GP_OP_APPLY, 64, 4, 32, 8, 128, 260, torch.bfloat16) > 0
    assert lib.gp_workspace_bytes(0, 4, 0, 32, 8, 96, 10, 16, 1, 1) == 0      # head_dim 96
    assert lib.gp_workspace_bytes(0, 4, 0, 24, 8, 128, 10, 16, 1, 1) == 0     # G = 3
    assert lib.gp_workspace_bytes(0, 4, 0, 32, 8, 128, 10, 32, 1, 1) == 0     # page size 32


def test_host_validation_without_launch(lib):
    fake = 0x1000
    kv = _lib._KVLayer(fake, fake, 100, 8, 16, 128, 1)
    ps = _lib._PageState(fake, fake, fake, fake, fake, fake, 4, 10, 100)
    # null layer -> invalid
    assert lib.gp_decode_attention(None, ctypes.byref(ps), fake, 32, 0.1, fake, fake, 1 << 30, None) == 1
    # head_dim 96 -> unsupported
    bad = _lib._KVLayer(fake, fake, 100, 8, 16, 96, 1)
    assert lib.gp_decode_attention(ctypes.byref(bad), ctypes.byref(ps), fake, 32, 0.1, fake, fake,
                                   1 << 30, None) == 2
    # workspace too small
    assert lib.gp_decode_attention(ctypes.byref(kv), ctypes.byref(ps), fake, 32, 0.1, fake, fake, 16,
                                   None) == 3
    # pool sizes disagree
    ps2 = _lib._PageState(fake, fake, fake, fake, fake, fake, 4, 10, 99)
    assert lib.gp_decode_attention(ctypes.byref(kv), ctypes.byref(ps2), fake, 32, 0.1, fake, fake,
                                   1 << 30, None) == 1
    # staged decode: stages must be GP_DECODE_CHUNKS, GP_DECODE_MERGE or both
    for bad_stages in (0, 4, -1):
        assert lib.gp_decode_attention_stages(ctypes.byref(kv), ctypes.byref(ps), fake, 32, 0.1, fake,
                                              bad_stages, fake, 1 << 30, None) == 1
    # summaries: beta outside [0, 1]
    assert lib.gp_update_summaries(fake, 1, 4, 32, 128, fake, fake, fake, 512, 1.5, 0.9, None) == 1
    # score: max_cand too small for the table width
    p = _lib._Params(0.9, 0.999, 0.99, 0.0, 0.088, 1e6, 4, 0)
    assert lib.gp_boundary_score(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 512, fake, fake, fake,
                                 2, 32, ctypes.byref(p), fake, fake, 16, fake, 1 << 30, None) == 1
    # staged score: the mask must be GP_SCORE_WEIGHTS, GP_SCORE_COUNTS or both
    pv = _lib._Params(0.9, 0.999, 0.99, 0.0, 0.088, 1e6, 4, 0)
    for bad_stages in (0, 4, -1):
        assert lib.gp_boundary_score_stages(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 512, fake, fake, fake,
                                            2, 32, ctypes.byref(pv), fake, fake, 144, fake, 1 << 30, None,
                                            bad_stages) == 1
    # apply: too many layers
    arr = (_lib._KVLayer * 1)(kv)
    assert lib.gp_boundary_apply(arr, 65, ctypes.byref(ps), fake, 2, fake, fake, 144, ctypes.byref(p),
                                 fake, fake, fake, fake, 1 << 30, None) == 2
    # score: unknown demand metric
    pm = _lib._Params(0.9, 0.999, 0.99, 0.0, 0.088, 1e6, 4, 0, 0, 2)
    assert lib.gp_boundary_score(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 512, fake, fake, fake,
                                 2, 32, ctypes.byref(pm), fake, fake, 144, fake, 1 << 30, None) == 1
    # apply: unknown policy, random policy without draws or with a probability
    # outside [0, 1], shrink with a non-finite threshold, unknown layout
    for fields in ((9, 0, 0, 0, 0.7, -0.005, None), (2, 0, 0, 0, 0.7, -0.005, None),
                   (2, 0, 0, 0, 1.5, -0.005, fake), (4, 0, 0, 64, 0.7, float("nan"), None),
                   (0, 0, 0, 0, 0.7, -0.005, None, 2)):
        pa = _lib._Params(0.9, 0.999, 0.99, 0.0, 0.088, 1e6, 4, 0, *fields)
        assert lib.gp_boundary_apply(arr, 1, ctypes.byref(ps), fake, 2, fake, fake, 144, ctypes.byref(pa),
                                     fake, fake, fake, fake, 1 << 30, None) == 1, fields
    # fused step: beta outside [0, 1], null summary pool, then a small workspace
    assert lib.gp_decode_step(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 32, 0.1, fake, fake, fake,
                              fake, 512, 0.9, -0.5, None, None, None, 0, fake, 1 << 30, None) == 1
    assert lib.gp_decode_step(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 32, 0.1, fake, fake, fake,
                              None, 512, 0.9, 0.999, None, None, None, 0, fake, 1 << 30, None) == 1
    assert lib.gp_decode_step(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 32, 0.1, fake, fake, fake,
                              fake, 512, 0.9, 0.999, None, None, None, 0, fake, 16, None) == 3
    # fused step with a token: K without V, or advancing without positions
    assert lib.gp_decode_step(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 32, 0.1, fake, fake, fake,
                              fake, 512, 0.9, 0.999, fake, None, fake, 1, fake, 1 << 30, None) == 1
    assert lib.gp_decode_step(ctypes.byref(kv), ctypes.byref(ps), fake, fake, 32, 0.1, fake, fake, fake,
                              fake, 512, 0.9, 0.999, fake, fake, None, 1, fake, 1 << 30, None) == 1
    # release: null state; append: beta outside [0, 1], too many layers, null summaries
    assert lib.gp_release_held(None, None) == 1
    assert lib.gp_append_step(arr, 1, ctypes.byref(ps), fake, fake, fake, fake, 32, fake, None, fake, 512,
                              1.5, 0.999, None) == 1
    assert lib.gp_append_step(arr, 65, ctypes.byref(ps), fake, fake, fake, fake, 32, fake, None, fake, 512,
                              0.9, 0.999, None) == 2
    assert lib.gp_append_step(arr, 1, ctypes.byref(ps), fake, fake, fake, fake, 32, fake, None, None, 512,
                              0.9, 0.999, None) == 1
    # split apply validates like apply; decide takes the hold flag last
    for name in ("gp_boundary_select", "gp_boundary_compact"):
        assert getattr(lib, name)(arr, 65, ctypes.byref(ps), fake, 2, fake, fake, 144, ctypes.byref(p),
                                  fake, fake, fake, fake, 1 << 30, None) == 2
    assert lib.gp_boundary_decide(arr, 65, ctypes.byref(ps), fake, 2, fake, fake, 144, ctypes.byref(p),
                                  fake, fake, fake, fake, 1 << 30, None, 1) == 2
    # no-allocation decode: null layer; a batch whose partials exceed the 8 MiB
    # static scratch is refused on the host (GP_ERR_SCRATCH) before any device call
    assert lib.gp_decode_attention_noalloc(None, ctypes.byref(ps), fake, 32, 0.1, fake, None) == 1
    big = _lib._PageState(fake, fake, fake, fake, fake, fake, 2048, 8192, 100)
    assert lib.gp_decode_attention_noalloc(ctypes.byref(kv), ctypes.byref(big), fake, 32, 0.1, fake, None) == 5
    # zero requests is a no-op that succeeds
    ps0 = _lib._PageState(fake, fake, fake, fake, fake, fake, 0, 10, 100)
    assert lib.gp_decode_attention(ctypes.byref(kv), ctypes.byref(ps0), fake, 32, 0.1, fake, fake, 0,
                                   None) == 0
    # streaming-read reference: null pointers, sizes not a multiple of 16
    assert lib.gp_stream_read(None, 16, fake, None) == 1
    assert lib.gp_stream_read(fake, 24, fake, None) == 1
    assert lib.gp_stream_read(fake, 0, fake, None) == 0


@pytest.mark.gpu
def test_stream_read_checksum(lib):
    """The streaming-read reference reads every word: its XOR checksum equals
    the host's, for a size with a ragged tail beyond the unrolled loop."""
    import numpy as np
    import torch
    rng = np.random.default_rng(3)
    for n_words in (4, 4 * 1000003, 4 * (1 << 22)):
        host = rng.integers(0, 2**32, size=n_words, dtype=np.uint64).astype(np.uint32)
        src = torch.from_numpy(host.view(np.int32)).cuda()
        out = torch.zeros(1, dtype=torch.int32, device="cuda")
        gp.gp_stream_read(src, out)
        torch.cuda.synchronize()
        assert int(out.cpu().numpy().view(np.uint32)[0]) == int(np.bitwise_xor.reduce(host))

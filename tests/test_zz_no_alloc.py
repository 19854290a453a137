"""gp_decode_attention_noalloc (partials in the library's static scratch, no
workspace) against gp_decode_attention with a workspace, through the C ABI:
two calls in a row, the second on a smaller batch, each bit-identical to the
workspace call on the same inputs; and the size limit."""
import math

import numpy as np
import pytest
import torch

import paper_2609_03494_amd as gp
import workloads as W
from _harness import DeviceCase

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gp.load()


def _say(*a):
    print(*a, flush=True)


def _both(w):
    dc = DeviceCase(w)
    scale = float(np.float32(1.0 / math.sqrt(w.head_dim)))
    ref = torch.full_like(dc.q_post, float("nan"))
    gp.gp_decode_attention(dc.layers[0], dc.ps, dc.q_post, scale, ref, dc.ws_decode)
    got = torch.full_like(dc.q_post, float("nan"))
    gp.gp_decode_attention_noalloc(dc.layers[0], dc.ps, dc.q_post, scale, got)
    torch.cuda.synchronize()
    return got, ref


def test_noalloc_equals_workspace_call_twice_second_smaller():
    # call 1: Qwen3-8B heads, 16 requests of up to 8000 tokens (several chunks
    # each); call 2: 5 short requests (fewer chunks, a smaller partial layout
    # over the same scratch, which still holds call 1's partials)
    big = W.qwen3_8b(seed=51, num_reqs=16, len_lo=500, len_hi=8000, budget_choices=(64, 128, 520),
                     free_pages=16)
    small = W.qwen3_8b(seed=52, num_reqs=5, len_lo=20, len_hi=1500, budget_choices=(100,), free_pages=8)
    need = [gp.gp_workspace_bytes(gp.GP_OP_DECODE, w.num_reqs, 0, w.num_q_heads, w.num_kv_heads,
                                  w.head_dim, w.max_pages, torch.bfloat16) for w in (big, small)]
    assert need[1] < need[0] <= 8 << 20
    for name, w in (("first, larger", big), ("second, smaller", small)):
        _say(f"noalloc decode: {name} batch, {w.num_reqs} requests, {int(w.seq_lens.max())} tokens max")
        got, ref = _both(w)
        assert torch.isfinite(ref.float()).all()
        assert torch.equal(got, ref), name


def test_noalloc_fp32_and_rejects_oversized_batch():
    _say("noalloc decode: tiny fp32, then a batch beyond the scratch")
    w = W.tiny()
    got, ref = _both(w)
    assert torch.equal(got, ref)
    # 2048 requests of up to 8192 pages: the partials would need far more than
    # 8 MiB, so the call is refused on the host, before any launch
    R, Hq, Hkv, d, maxp = 2048, 32, 8, 128, 8192
    assert gp.gp_workspace_bytes(gp.GP_OP_DECODE, R, 0, Hq, Hkv, d, maxp, torch.bfloat16) > 8 << 20
    k = torch.zeros((4, Hkv, 16, d), dtype=torch.bfloat16, device="cuda")
    kv = gp.KVLayer(k, k)
    i32 = lambda *s: torch.zeros(s, dtype=torch.int32, device="cuda")
    ps = gp.PageState(i32(R, maxp), i32(R), i32(R), i32(4), i32(4), i32(1))
    q = torch.zeros((R, Hq, d), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(gp.GrowPageError) as e:
        gp.gp_decode_attention_noalloc(kv, ps, q, 0.088, q.clone())
    assert e.value.status == gp.GP_ERR_SCRATCH

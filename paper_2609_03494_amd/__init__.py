"""GrowPage decode-step hot path on MI355X: a C-ABI HIP library and its binding.

The library (``libgrowpage.so``, header ``include/growpage.h``) runs paged GQA
decode attention, the dual-timescale query summaries, and the capacity-boundary
scoring / compress-vs-grow decision / selection / compaction of GrowPage
(arXiv 2609.03494) as hand-written gfx950 kernels.  PyTorch supplies device
memory and streams.
"""
from ._lib import (  # noqa: F401
    EXPORTS, GP_BF16, GP_COMPRESS, GP_DECODE_CHUNKS, GP_DECODE_MERGE, GP_DECODE_PREFIX, GP_F32, GP_FALLBACK, GP_GROW, GP_NOT_BOUNDARY,
    GP_METRIC_ENTROPY, GP_METRIC_TOP_P, GP_OP_APPLY, GP_OP_DECODE, GP_OP_SCORE, GP_POLICY_FIXED,
    GP_POLICY_GROWPAGE, GP_POLICY_INVERSE, GP_POLICY_RANDOM, GP_POLICY_SHRINK, GP_PREEMPT, GP_SHRINK,
    GP_ERR_SCRATCH, GP_SCORE_COUNTS, GP_SCORE_WEIGHTS, LIB_PATH, PAGE_SIZE,
    GP_LAYOUT_FILL, GP_LAYOUT_SHIFT, GrowPageError, KVLayer, PageState, Params, gp_append_step, gp_boundary_apply, gp_boundary_compact,
    gp_boundary_decide, gp_boundary_score, gp_boundary_select, gp_release_held,
    gp_decode_attention, gp_decode_attention_noalloc, gp_decode_attention_shared, gp_decode_attention_stages, gp_decode_step, gp_stream_read, gp_update_summaries, gp_workspace_bytes, load, status_string,
    workspace,
)

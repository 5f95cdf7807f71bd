"""SparseCoder hot path on MI355X: sliding-window + global sparse attention fused
with learned token pruning (arXiv 2310.07109), as hand-written gfx950 kernels
behind a C ABI (``include/sc.h``, ``libsc.so``).

This package is the thin Python binding: it marshals torch device tensors to
the C entry points of the same names.  torch only allocates device memory and
provides the stream; every step of the path runs in the library's kernels.
There is no fallback: without the built library every call raises.
"""
from ._binding import (SC_BF16, SC_F32, SC_SCORE_FROM_BAND_PROBS, SC_SCORE_FROM_PARTIALS, Desc, ScError,  # noqa
                       lib_path, load, sc_band_probs_size, sc_encoder_attn_stack,
                       sc_encoder_attn_stack_workspace_size, sc_encoder_stack, sc_encoder_stack_workspace_size,
                       sc_ltp_prune_compact, sc_ltp_prune_compact_workspace_size, sc_ltp_score,
                       sc_ltp_score_workspace_size, sc_ltp_soft_backward,
                       sc_ltp_soft_backward_workspace_size, sc_ltp_soft_mask, sc_profile_window_kernel, sc_profile_window_kernel_read,
                       sc_score_partials_size, sc_status_str, sc_topk_prune_compact, sc_window_attention,
                       sc_window_attention_noalloc, sc_window_attention_workspace_size, SC_NOALLOC_SCRATCH_BYTES,
                       SC_ENOSCRATCH, SC_VALID_LEN, SC_VALID_POS_RANGE, SC_VALID_POS_ORDER,
                       SC_VALID_POS_UNUSED_FIRST, debug_lib_path, load_debug, sc_validate_desc)

__all__ = [
    "SC_BF16", "SC_F32", "SC_SCORE_FROM_PARTIALS", "SC_SCORE_FROM_BAND_PROBS", "Desc", "ScError", "load",
    "lib_path", "sc_status_str", "sc_score_partials_size", "sc_band_probs_size",
    "sc_window_attention_workspace_size", "sc_window_attention", "sc_ltp_score_workspace_size", "sc_ltp_score",
    "sc_ltp_prune_compact_workspace_size", "sc_ltp_prune_compact", "sc_topk_prune_compact",
    "sc_ltp_soft_mask", "sc_ltp_soft_backward_workspace_size", "sc_ltp_soft_backward",
    "sc_encoder_attn_stack_workspace_size", "sc_encoder_attn_stack", "sc_encoder_stack_workspace_size",
    "sc_encoder_stack", "sc_profile_window_kernel", "sc_profile_window_kernel_read",
    "sc_window_attention_noalloc", "SC_NOALLOC_SCRATCH_BYTES", "SC_ENOSCRATCH", "SC_VALID_LEN",
    "SC_VALID_POS_RANGE", "SC_VALID_POS_ORDER", "SC_VALID_POS_UNUSED_FIRST", "debug_lib_path", "load_debug",
    "sc_validate_desc",
]

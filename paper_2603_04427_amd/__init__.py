"""Thin-key attention for AMD Instinct MI355X (gfx950).

The computation lives in libtkattn.so (hand-written HIP kernels behind the C
ABI of include/tk_attn.h); ``binding`` exposes its entry points under the same
names, plus prepared (pre-marshalled) calls for timing loops. ``accounting``
holds the byte/FLOP accounting used for roofline figures.
"""
from .binding import (PreparedCall, TkError, prepare_cache_append, prepare_decode, prepare_prefill,  # noqa: F401
                      prepare_prefill_backward, prepare_prefill_lse, prepare_project_heads, tk_attn_decode,
                      tk_attn_decode_noalloc, tk_attn_decode_workspace_bytes, tk_attn_prefill, tk_attn_prefill_backward,
                      tk_attn_prefill_backward_workspace_bytes, tk_attn_prefill_lse, tk_cache_append,
                      tk_project_heads, tk_status_str, tk_version)

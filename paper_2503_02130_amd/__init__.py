"""Forgetting Attention (FoX, arXiv 2503.02130) for AMD Instinct MI355X.

The operator runs entirely in hand-written HIP kernels for gfx950, reached
through the C ABI declared in include/fox.h (libfox.so).  This package holds
the ctypes binding (same entry-point names as the C ABI), the build script and
the seeded input generators used by tests and benchmarks.
"""
from ._lib import (  # noqa: F401
    FoxError, default_scale, load, status_string,
    fox_gate_prefix, fox_attn_fwd, fox_attn_bwd, fox_attn_bwd_workspace_bytes,
    fox_attn_bwd_delta, fox_attn_bwd_dkdv, fox_attn_bwd_dq, fox_dlogf_from_dc,
    fox_dlogit_from_dc, fox_attn_decode, fox_attn_decode_noalloc,
    fox_fixed_gate_init, fox_attn_fwd_fixed_gate, fox_attn_bwd_fixed_gate,
    fox_attn_bwd_fixed_gate_workspace_bytes, fox_attn_decode_fixed_gate,
    fox_attn_decode_workspace_bytes, fox_row_norm_max, fox_attn_decode_skip,
    fox_attn_fwd_skip, fox_attn_bwd_skip, LIB_PATH,
    fox_attn_fwd_fixed_gate_skip, fox_attn_bwd_fixed_gate_skip, fox_attn_decode_fixed_gate_skip,
    fox_pro_prologue, fox_pro_prologue_bwd, fox_pro_prologue_bwd_workspace_bytes,
    fox_pro_output_gate, fox_attn_fwd_pro, fox_attn_bwd_pro, fox_attn_bwd_pro_workspace_bytes,
    fox_attn_bwd_stored, fox_attn_bwd_stored_workspace_bytes, fox_attn_bwd_ds_store_bytes,
    fox_attn_bwd_dkdv_store, fox_attn_bwd_dq_stored, fox_attn_bwd_pro_stored,
    fox_attn_bwd_pro_stored_workspace_bytes, fox_attn_bwd_skip_stored,
    fox_attn_bwd_fixed_gate_stored, fox_attn_bwd_fixed_gate_stored_workspace_bytes,
    fox_attn_bwd_fixed_gate_skip_stored,
    fox_gate_projection, fox_gate_projection_bwd, fox_gate_projection_bwd_workspace_bytes,
    EXPORTED,
)

from .autograd import (  # noqa: E402,F401
    ForgettingAttention, GateProjection, forget_gate_logits, forgetting_attention,
)

__all__ = [
    "ForgettingAttention", "forgetting_attention", "GateProjection", "forget_gate_logits",
    "FoxError", "default_scale", "load", "status_string",
    "fox_gate_prefix", "fox_attn_fwd", "fox_attn_bwd", "fox_attn_bwd_workspace_bytes",
    "fox_attn_bwd_delta", "fox_attn_bwd_dkdv", "fox_attn_bwd_dq", "fox_dlogf_from_dc",
    "fox_dlogit_from_dc", "fox_fixed_gate_init", "fox_attn_fwd_fixed_gate",
    "fox_attn_bwd_fixed_gate", "fox_attn_bwd_fixed_gate_workspace_bytes",
    "fox_attn_decode_fixed_gate",
    "fox_attn_decode", "fox_attn_decode_noalloc", "fox_attn_decode_workspace_bytes",
    "fox_row_norm_max",
    "fox_attn_decode_skip", "fox_attn_fwd_skip", "fox_attn_bwd_skip",
    "fox_attn_fwd_fixed_gate_skip", "fox_attn_bwd_fixed_gate_skip",
    "fox_attn_decode_fixed_gate_skip",
    "fox_pro_prologue", "fox_pro_prologue_bwd", "fox_pro_prologue_bwd_workspace_bytes",
    "fox_pro_output_gate", "fox_attn_fwd_pro", "fox_attn_bwd_pro",
    "fox_attn_bwd_pro_workspace_bytes", "fox_attn_bwd_stored", "fox_attn_bwd_stored_workspace_bytes",
    "fox_attn_bwd_ds_store_bytes", "fox_attn_bwd_dkdv_store", "fox_attn_bwd_dq_stored",
    "fox_attn_bwd_pro_stored", "fox_attn_bwd_pro_stored_workspace_bytes",
    "fox_attn_bwd_skip_stored", "fox_attn_bwd_fixed_gate_stored",
    "fox_attn_bwd_fixed_gate_stored_workspace_bytes", "fox_attn_bwd_fixed_gate_skip_stored",
    "fox_gate_projection", "fox_gate_projection_bwd", "fox_gate_projection_bwd_workspace_bytes",
]

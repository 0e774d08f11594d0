"""fp64 CPU oracle for Forgetting Attention.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.
"""
from .fox_oracle import (  # noqa: F401
    log_sigmoid, prefix_c, gate_prefix, decay_matrix,
    forward_head_from_c, backward_head_from_c, reverse_cumsum,
    forward_from_logf, forward, backward_from_logf, backward, decode,
    gate_backward, backward_logit, gate_projection, gate_projection_backward,
    time_constant, fixed_gate_bias_init, fixed_gate_log_f, forward_fixed_gate,
    backward_fixed_gate,
    rms_norm, rms_norm_backward, token_shift, token_shift_backward,
    pro_prologue, pro_prologue_backward, output_gate, output_gate_backward,
    pro_forward, pro_backward,
)

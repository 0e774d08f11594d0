"""Forgetting Attention as a PyTorch autograd function.

Glue only: the forward runs fox_gate_prefix and fox_attn_fwd, the backward the
staged backward (recomputing, or keeping dS when asked and the dtype is bf16)
and fox_dlogit_from_dc, which returns the gradient of the gate logits through
log f = logsigmoid(logit) and c = cumsum(log f) (Sec. 3).  GateProjection
gives the logits themselves from the layer input, w_f^T x_t + b_f per head,
with fox_gate_projection and fox_gate_projection_bwd.  Every step runs in the
library's kernels.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import _lib as fox


class ForgettingAttention(torch.autograd.Function):
    """o = FoX attention of q, k, v [B,H,L,d] with gate logits [B,H,L] (fp32)."""

    @staticmethod
    def forward(ctx, q, k, v, gate_logit, scale, keep_ds):
        q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
        gate_logit = gate_logit.contiguous()
        c = fox.fox_gate_prefix(gate_logit)
        o, lse = fox.fox_attn_fwd(q, k, v, c, scale)
        ctx.save_for_backward(q, k, v, gate_logit, c, o, lse)
        ctx.scale = scale
        ctx.keep_ds = bool(keep_ds) and q.dtype == torch.bfloat16
        return o

    @staticmethod
    def backward(ctx, d_o):
        q, k, v, gate_logit, c, o, lse = ctx.saved_tensors
        d_o = d_o.to(q.dtype).contiguous()
        s = ctx.scale
        delta = fox.fox_attn_bwd_delta(o, d_o)
        if ctx.keep_ds:
            B, H, L, d = q.shape
            store = torch.empty(fox.fox_attn_bwd_ds_store_bytes(q.dtype, B, H, L, d),
                                dtype=torch.uint8, device=q.device)
            dk, dv, dc_k = fox.fox_attn_bwd_dkdv_store(q, k, v, c, lse, d_o, delta, store, s)
            dq, dc_q = fox.fox_attn_bwd_dq_stored(k, store, s)
        else:
            dk, dv, dc_k = fox.fox_attn_bwd_dkdv(q, k, v, c, lse, d_o, delta, s)
            dq, dc_q = fox.fox_attn_bwd_dq(q, k, v, c, lse, d_o, delta, s)
        d_logit = fox.fox_dlogit_from_dc(dc_q, dc_k, gate_logit)
        return dq, dk, dv, d_logit, None, None


def forgetting_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                         gate_logit: torch.Tensor, scale: Optional[float] = None,
                         keep_ds: bool = False) -> torch.Tensor:
    """Causal Forgetting Attention with autograd support.

    q, k, v: [B, H, L, d] bf16 or fp32 on the GPU (d = 64 or 128); gate_logit:
    [B, H, L] fp32, the forget gate f = sigmoid(gate_logit).  scale defaults to
    1/sqrt(d).  keep_ds (bf16): the backward keeps dS in a temporary workspace of
    about B*H*L^2 bytes instead of recomputing it for dQ (faster at long L).
    """
    s = fox.default_scale(q.shape[-1]) if scale is None else float(scale)
    return ForgettingAttention.apply(q, k, v, gate_logit, s, keep_ds)


class GateProjection(torch.autograd.Function):
    """gate_logit[b, h, t] = w_f[h] . x[b, t] + b_f[h] (Sec. 3, gate definition)."""

    @staticmethod
    def forward(ctx, x, w_f, b_f):
        x, w_f = x.contiguous(), w_f.contiguous()
        b = None if b_f is None else b_f.contiguous()
        logit = fox.fox_gate_projection(x, w_f, b)
        ctx.save_for_backward(x, w_f)
        ctx.has_bias = b_f is not None
        return logit

    @staticmethod
    def backward(ctx, d_logit):
        x, w_f = ctx.saved_tensors
        dx, dw, db = fox.fox_gate_projection_bwd(x, w_f, d_logit.contiguous(),
                                                 want_dx=ctx.needs_input_grad[0],
                                                 want_db=ctx.has_bias)
        return dx, dw, db


def forget_gate_logits(x: torch.Tensor, w_f: torch.Tensor,
                       b_f: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The forget-gate logits [B, H, L] fp32 from the layer input x [B, L, M]
    (bf16 or fp32, M % 8 == 0), w_f [H, M] and b_f [H] fp32 (H <= 64), with
    autograd support; feed them to forgetting_attention."""
    return GateProjection.apply(x, w_f, b_f)

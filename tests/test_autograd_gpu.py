"""forgetting_attention as a torch.autograd function: its gradients are the
library's backward entry points, bit for bit, and match the oracle."""
import os

import pytest
import torch

import oracle
import paper_2503_02130_amd as fox
from paper_2503_02130_amd import inputs

pytestmark = pytest.mark.gpu
torch.set_num_threads(max(1, min(16, len(os.sched_getaffinity(0)))))
DEV = "cuda:0"


def _rel_l2(a, b):
    a, b = a.detach().double().cpu(), b.detach().double().cpu()
    return float(torch.linalg.vector_norm(a - b) / torch.linalg.vector_norm(b))


@pytest.mark.parametrize("dtype,d,L,keep", [("bf16", 128, 333, False), ("bf16", 128, 333, True),
                                            ("bf16", 64, 1000, True), ("f32", 64, 129, False)])
def test_forgetting_attention_autograd(dtype, d, L, keep):
    print(f"autograd dtype={dtype} d={d} L={L} keep_ds={keep}", flush=True)
    x = inputs.attn_inputs(2, 3, L, d, dtype, ("normal", 2.0, 1.5), 50 + L, device=DEV)
    q, k, v = (x[n].clone().requires_grad_() for n in ("q", "k", "v"))
    logit = x["logit"].clone().requires_grad_()
    o = fox.forgetting_attention(q, k, v, logit, keep_ds=keep)
    o.backward(x["do"])
    # the same through the entry points
    s = fox.default_scale(d)
    c = fox.fox_gate_prefix(x["logit"])
    o2, lse = fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s)
    bwd = fox.fox_attn_bwd_stored if keep else fox.fox_attn_bwd
    dq, dk, dv, _ = bwd(x["q"], x["k"], x["v"], c, o2, lse, x["do"], s)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2)
    for name, a, b in (("dq", q.grad, dq), ("dk", k.grad, dk), ("dv", v.grad, dv)):
        assert torch.equal(a, b), name
    xc = {n: t.cpu() for n, t in x.items()}
    ref = oracle.backward_logit(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    lim = 1e-4 if dtype == "f32" else 2e-2
    for name, g, r in zip(("dq", "dk", "dv", "dlogit"), (q.grad, k.grad, v.grad, logit.grad), ref):
        e = _rel_l2(g, r)
        assert e <= lim, f"{name} rel-L2 {e:.3e}"


def test_gate_projection_autograd_chain():
    """Layer input -> gate logits -> Forgetting Attention, all through autograd:
    the projection's gradients equal the entry point's on the same d_logit bit
    for bit, and the chain matches the oracle's."""
    B, H, L, d, M = 2, 3, 200, 64, 96
    print(f"autograd gate projection chain B={B} H={H} L={L} d={d} M={M}", flush=True)
    a = inputs.attn_inputs(B, H, L, d, "bf16", ("normal", 2.0, 1.0), 71, device=DEV)
    p = inputs.projection_inputs(B, L, H, M, "bf16", 72, device=DEV)
    xin = p["x"].clone().requires_grad_()
    w = p["w_f"].clone().requires_grad_()
    b = (p["b_f"] + 2.0).requires_grad_()
    logit = fox.forget_gate_logits(xin, w, b)
    logit.retain_grad()
    o = fox.forgetting_attention(a["q"], a["k"], a["v"], logit)
    o.backward(a["do"])
    torch.cuda.synchronize()
    assert torch.equal(logit.detach(), fox.fox_gate_projection(p["x"], p["w_f"], b.detach()))
    dx, dw, db = fox.fox_gate_projection_bwd(p["x"], p["w_f"], logit.grad)
    torch.cuda.synchronize()
    for name, u, v in (("dx", xin.grad, dx), ("dw", w.grad, dw), ("db", b.grad, db)):
        assert torch.equal(u, v), name
    # the oracle's chain: logits, then the logit gradient of the attention, then the projection
    cpu = lambda t: t.detach().cpu()
    ref_logit = oracle.gate_projection(cpu(p["x"]), cpu(w), cpu(b))
    s = fox.default_scale(d)
    _, _, _, dlogit_ref = oracle.backward_logit(cpu(a["q"]), cpu(a["k"]), cpu(a["v"]), ref_logit,
                                                cpu(a["do"]), s)
    rdx, rdw, rdb = oracle.gate_projection_backward(cpu(p["x"]), cpu(w), dlogit_ref)
    assert _rel_l2(logit, ref_logit) <= 1e-5
    for name, u, r in (("dx", xin.grad, rdx), ("dw", w.grad, rdw), ("db", b.grad, rdb)):
        assert _rel_l2(u, r) <= 2e-2, name

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

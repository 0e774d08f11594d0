"""The training step inside a HIP graph.

Every entry point only enqueues kernels on the caller's stream (no allocation,
no memset, no synchronisation), so a whole step can be captured once and
replayed.  The graph here holds the gate projection from the layer input, the
gate prefix, the forward, the four stages of the backward keeping dS and the
projection's backward; it is replayed several times with eager work
and synchronisations between the replays, and every replay must reproduce the
eager step bit for bit.
"""
import pytest
import torch

import paper_2503_02130_amd as fox
from paper_2503_02130_amd import inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_training_step_replays_in_a_hip_graph():
    B, H, L, d = 2, 3, 777, 128
    print(f"graph step B={B} H={H} L={L} d={d}", flush=True)
    x = inputs.attn_inputs(B, H, L, d, "bf16", ("normal", 2.0, 1.0), 31, device=DEV)
    s = fox.default_scale(d)
    c = torch.empty((B, H, L), device=DEV)
    o, lse = torch.empty_like(x["q"]), torch.empty((B, H, L), device=DEV)
    dq, dk, dv = (torch.empty_like(x["q"]) for _ in range(3))
    delta, dcq, dck, dlf, dlogit = (torch.empty((B, H, L), device=DEV) for _ in range(5))
    store = torch.empty(fox.fox_attn_bwd_ds_store_bytes(torch.bfloat16, B, H, L, d),
                        dtype=torch.uint8, device=DEV)
    M = 96
    pj = inputs.projection_inputs(B, L, H, M, "bf16", 32, device=DEV)
    logit = torch.empty((B, H, L), device=DEV)
    pdx, pdw, pdb = torch.empty_like(pj["x"]), torch.empty((H, M), device=DEV), torch.empty(H, device=DEV)
    pws = torch.empty(fox.fox_gate_projection_bwd_workspace_bytes(torch.bfloat16, B, L, H, M),
                      dtype=torch.uint8, device=DEV)
    outs = (logit, c, o, lse, dq, dk, dv, dlf, dlogit, pdx, pdw, pdb)

    def step():
        fox.fox_gate_projection(pj["x"], pj["w_f"], pj["b_f"], gate_logit=logit)
        fox.fox_gate_prefix(logit, c=c)
        fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s, o=o, lse=lse)
        fox.fox_attn_bwd_delta(o, x["do"], delta=delta)
        fox.fox_attn_bwd_dkdv_store(x["q"], x["k"], x["v"], c, lse, x["do"], delta, store, s,
                                    dk=dk, dv=dv, dc_k=dck)
        fox.fox_attn_bwd_dq_stored(x["k"], store, s, dq=dq, dc_q=dcq)
        fox.fox_dlogit_from_dc(dcq, dck, logit, d_logit=dlogit, d_log_f=dlf)
        fox.fox_gate_projection_bwd(pj["x"], pj["w_f"], dlogit, workspace=pws, dx=pdx, dw=pdw,
                                    db=pdb)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()  # a warm-up on the capture's side stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in outs:
            t.fill_(float("nan"))  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("c", "o", "lse", "dq", "dk", "dv", "dlf", "dlogit"), outs, ref):
            assert torch.equal(a, b), f"replay {rep}: {name}"
        step()  # the eager step again, interleaved with the replays
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(a, b)

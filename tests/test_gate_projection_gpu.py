"""GPU parity of the forget-gate projection (Sec. 3, gate definition) and its
backward against the fp64 oracle, through the C ABI.

Error bars, per element, from the arithmetic: bf16 keeps 8 significant bits,
so hi = RNE(v) is within 2^-8 |v| and the pair hi + lo within 2^-16 |v|; a
product keeps three of its four terms, so it is within 4 * 2^-16 of exact; the fp32 accumulation adds at most
K * 2^-24 relative for K additions in sequence, K counting every product of
the contraction (three split terms per pair of operands) and the final sums.  Both scale with the sum of the
absolute values of the terms, which the oracle gives when fed |x|, |w_f| and
|d_logit|.  A relative L2 bar on top of that catches a dropped token or
contraction step, which the elementwise worst case can be too loose to see.
"""
import math

import pytest
import torch

import oracle
import paper_2503_02130_amd as fox
from paper_2503_02130_amd import inputs

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
U24 = 2.0 ** -24
SPLIT = 4 * 2.0 ** -16


def rel_l2(a, b) -> float:
    a, b = a.double().cpu(), b.double().cpu()
    return float((a - b).norm() / max(b.norm().item(), 1e-300))


def within(got, ref, bound, what, mag=None):
    err = (got.double().cpu() - ref).abs()
    if mag is not None:
        print(f"  {what}: max err/sum|terms| {float((err / mag.clamp_min(1e-300)).max()):.3e}, "
              f"rel-L2 {rel_l2(got, ref):.3e}", flush=True)
    bad = err > bound
    i = int((err / bound).flatten().argmax())
    assert not bool(bad.any()), (f"{what}: {int(bad.sum())} elements beyond the bound; worst at "
                                 f"flat index {i}: err {float(err.flatten()[i]):.3e}, bound "
                                 f"{float(bound.flatten()[i]):.3e}, ref {float(ref.flatten()[i]):.3e}")


def run_case(B, L, H, M, dtype, seed, with_bias=True, want_dx=True, want_db=True):
    print(f"[gate projection] B={B} L={L} H={H} M={M} {dtype} seed={seed}", flush=True)
    cpu = inputs.projection_inputs(B, L, H, M, dtype, seed)
    gpu = {k: v.to(DEV) for k, v in cpu.items()}
    b_f = gpu["b_f"] if with_bias else None
    logit = fox.fox_gate_projection(gpu["x"], gpu["w_f"], b_f)
    dx, dw, db = fox.fox_gate_projection_bwd(gpu["x"], gpu["w_f"], gpu["d_logit"],
                                             want_dx=want_dx, want_db=want_db)
    torch.cuda.synchronize()

    x, w, g = cpu["x"], cpu["w_f"], cpu["d_logit"]
    ref = oracle.gate_projection(x, w, cpu["b_f"] if with_bias else None)
    mag = oracle.gate_projection(x.abs(), w.abs())
    K = 3 * M + 8
    within(logit, ref, (SPLIT + K * U24) * mag + 1e-6 * (1 + ref.abs()), "logit", mag)
    assert rel_l2(logit, ref) <= 1e-5

    rdx, rdw, rdb = oracle.gate_projection_backward(x, w, g)
    mdx, mdw, mdb = oracle.gate_projection_backward(x.abs(), w.abs(), g.abs())
    N = B * L
    within(dw, rdw, (SPLIT + (3 * N + 8 + math.ceil(N / 32)) * U24) * mdw + 1e-30, "dw_f", mdw)
    assert rel_l2(dw, rdw) <= 2e-5
    if want_db:
        within(db, rdb, (N + 8) * U24 * mdb + 1e-30, "db_f", mdb)
        assert rel_l2(db, rdb) <= 1e-5
    else:
        assert db is None
    if want_dx:
        bound = (SPLIT + (3 * 16 * math.ceil(H / 16) + 4) * U24) * mdx + 1e-30
        if dtype == "bf16":
            bound = bound + 2.0 ** -8 * rdx.abs()
        within(dx, rdx, bound, "dx", mdx)
        assert rel_l2(dx, rdx) <= (5e-3 if dtype == "bf16" else 2e-5)
    else:
        assert dx is None
    return logit, dx, dw, db


CASES = [("f32", 1, 1, 1, 8), ("bf16", 1, 1, 1, 8),
         ("f32", 2, 37, 3, 40), ("bf16", 2, 37, 3, 40),
         ("f32", 1, 256, 2, 128), ("bf16", 3, 300, 12, 768),
         ("bf16", 2, 129, 40, 136), ("f32", 1, 65, 64, 264),
         ("bf16", 1, 1000, 16, 2048), ("f32", 3, 33, 32, 16),
         # every 32-token tile crosses batches; the smallest two-head-block case;
         # a long ragged token count with the largest head count and M = 8
         ("bf16", 5, 1, 2, 16), ("f32", 3, 7, 33, 24), ("bf16", 2, 4097, 64, 8)]


@pytest.mark.parametrize("dtype,B,L,H,M", CASES)
def test_gate_projection_small(dtype, B, L, H, M):
    run_case(B, L, H, M, dtype, seed=1000 + 7 * L + M + H)


def test_gate_projection_optional_outputs():
    run_case(2, 70, 5, 48, "bf16", seed=3, with_bias=False, want_dx=False, want_db=False)


def test_gate_projection_is_deterministic():
    a = run_case(2, 600, 16, 256, "bf16", seed=4)
    b = run_case(2, 600, 16, 256, "bf16", seed=4)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("B,L,H,M", [(8, 2048, 12, 768), (2, 16384, 16, 2048)])
def test_gate_projection_workload(B, L, H, M):
    """The model widths of the two training workloads (M = H * head dim)."""
    run_case(B, L, H, M, "bf16", seed=5)

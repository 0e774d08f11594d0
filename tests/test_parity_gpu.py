"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Tolerances (from the operator's specification):
  * fp32: max-abs <= 1e-4 on O (and on LSE);
  * bf16: relative L2 <= 1e-2 on O, <= 2e-2 on dQ, dK, dV and d(log f);
    LSE max-abs <= 1e-2 (bf16 inputs and fp32 accumulation);
  * gate prefix (fp32): log f within 2e-6 absolute, c within a few fp32 ulps of
    the largest |c| of its row times log2(L).
Small shapes cover ragged tails (lengths that are not multiples of any tile),
L = 1, both head dims and both dtypes; the full-size workloads run in the same
launch configuration as the benchmark and are compared on sampled heads / rows
that the oracle computes exactly.
"""
import math
import os

import pytest
import torch

import oracle
import paper_2503_02130_amd as fox
from paper_2503_02130_amd import inputs

pytestmark = pytest.mark.gpu
torch.set_num_threads(max(1, min(16, len(os.sched_getaffinity(0)))))
DEV = "cuda:0"


def rel_l2(a, b) -> float:
    a = a.detach().double().cpu()
    b = b.detach().double().cpu()
    den = float(torch.linalg.vector_norm(b))
    return float(torch.linalg.vector_norm(a - b)) / max(den, 1e-300)


def max_abs(a, b) -> float:
    return float((a.detach().double().cpu() - b.detach().double().cpu()).abs().max())


def gpu_forward(x, s):
    c = fox.fox_gate_prefix(x["logit"])
    o, lse = fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s)
    return c, o, lse


def cpu(x):
    return {k: v.cpu() for k, v in x.items()}


def c_precision(c_abs, L):
    """How far an fp32 prefix value may lie from the exact one: the bound the gate
    prefix test holds c to (4 ulps of the largest |c| per scan level).  A
    difference c_i - c_j of two stored values carries twice that."""
    return 4 * 2.0 ** -23 * c_abs * max(1.0, math.log2(max(L, 2)))


def check_fwd(dtype, o, lse, O, LSE, what="", c_abs=0.0, L=1):
    """fp32: max-abs <= 1e-4 on O and LSE; where the prefix values c reach a
    large |c_abs| the LSE (which includes c_i - c_j) may in addition carry the
    fp32 rounding of the stored c (reading: c is kept in fp32)."""
    if dtype == "f32":
        assert max_abs(o, O) <= 1e-4, f"{what} O max-abs {max_abs(o, O):.3e}"
        tol = 1e-4 + 2 * c_precision(c_abs, L)
        assert max_abs(lse, LSE) <= tol, f"{what} LSE max-abs {max_abs(lse, LSE):.3e} > {tol:.3e}"
    else:
        assert rel_l2(o, O) <= 1e-2, f"{what} O rel-L2 {rel_l2(o, O):.3e}"
        assert max_abs(lse, LSE) <= 1e-2, f"{what} LSE max-abs {max_abs(lse, LSE):.3e}"


def check_grad(dtype, name, g, r, what=""):
    """Relative L2 of one gradient.  Where the exact gradient vanishes
    identically (dQ = dK = d(log f) = 0 at L = 1) a relative error is undefined,
    and the rounding residue is bounded absolutely instead."""
    lim = 1e-4 if dtype == "f32" else 2e-2
    lim_abs = 1e-5 if dtype == "f32" else 1e-3
    r64 = r.detach().double().cpu()
    if float(torch.linalg.vector_norm(r64)) <= 1e-9 * math.sqrt(r64.numel()):
        e = max_abs(g, r64)
        assert e <= lim_abs, f"{what} {name} (exactly zero) max-abs {e:.3e} > {lim_abs}"
        return
    e = rel_l2(g, r)
    assert e <= lim, f"{what} {name} rel-L2 {e:.3e} > {lim}"


def check_bwd(dtype, got, ref, what=""):
    for name, g, r in zip(("dQ", "dK", "dV", "dlogf"), got, ref):
        check_grad(dtype, name, g, r, what)


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# --------------------------------------------------------------------- prelude
# aligned rows of one segment (2048), of several (16384, 65536: log sigmoid
# over all rows first, then the scan in place), and unaligned rows (odd L, 16387)
@pytest.mark.parametrize("L", [1, 2, 3, 17, 2047, 2048, 2049, 16384, 16387, 65536])
def test_gate_prefix(L):
    print(f"gate_prefix L={L}", flush=True)
    g = torch.Generator(device=DEV).manual_seed(L)
    x = torch.randn(3, 2, L, generator=g, device=DEV) * 2.0 + torch.tensor(
        [-2.0, 1.0, 6.0], device=DEV)[:, None, None]
    c, lf = fox.fox_gate_prefix(x, want_log_f=True)
    c_only = fox.fox_gate_prefix(x)  # without the log f output: the same c
    torch.cuda.synchronize()
    assert torch.equal(c, c_only)
    lf_ref, c_ref = oracle.gate_prefix(x.cpu())
    assert max_abs(lf, lf_ref) <= 2e-6
    tol = 4 * 2.0 ** -23 * float(c_ref.abs().max()) * max(1.0, math.log2(L)) + 1e-5
    assert max_abs(c, c_ref) <= tol, (max_abs(c, c_ref), tol)


# ------------------------------------------------------------ small forward
FWD_CASES = ([("f32", 64, L) for L in (1, 3, 64, 65, 200)] +
             [("f32", 128, L) for L in (17, 130)] +
             [("bf16", 64, L) for L in (1, 2, 17, 63, 64, 65, 127, 128, 129, 1000)] +
             [("bf16", 128, L) for L in (1, 31, 129, 333, 1000)])


@pytest.mark.parametrize("dtype,d,L", FWD_CASES)
def test_forward_small(dtype, d, L):
    print(f"forward dtype={dtype} d={d} L={L}", flush=True)
    x = inputs.attn_inputs(2, 3, L, d, dtype, ("normal", 2.0, 1.0), 100 + L, device=DEV, grad=False)
    s = fox.default_scale(d)
    _, o, lse = gpu_forward(x, s)
    torch.cuda.synchronize()
    xc = cpu(x)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    check_fwd(dtype, o, lse, O, LSE, f"L={L}")


GATES = {
    "strong": ("normal", -2.0, 1.0),      # log f ~ -2: very local attention
    "none": ("constant", 30.0),           # log f ~ -1e-13: plain causal softmax attention
    "full": ("constant", -30.0),          # log f ~ -30: every row copies its own value
    "mixed": ("split_heads", (6.0, 1.0), (0.0, 1.4142135623730951)),
}


@pytest.mark.parametrize("gate", sorted(GATES))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_gate_regimes(gate, dtype):
    print(f"forward gate={gate} dtype={dtype}", flush=True)
    x = inputs.attn_inputs(1, 4, 300, 128, dtype, GATES[gate], 7, device=DEV, grad=False)
    s = fox.default_scale(128)
    _, o, lse = gpu_forward(x, s)
    torch.cuda.synchronize()
    xc = cpu(x)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    check_fwd(dtype, o, lse, O, LSE, gate)
    if gate == "full":
        assert rel_l2(o, xc["v"]) <= (1e-6 if dtype == "f32" else 1e-2)


# ------------------------------------------- the forward's rescale path
RESCALE_CASES = [(128, 700, ("constant", 30.0)), (64, 700, ("constant", 30.0)),
                 (128, 2000, ("normal", 6.0, 1.0)), (64, 300, ("normal", 4.0, 1.0))]


@pytest.mark.parametrize("d,L,gate", RESCALE_CASES)
def test_forward_rescale_path(d, L, gate):
    """Rows dominated by a few early keys (inputs.rescale_inputs): scores of
    later-visited tiles exceed the diagonal tile's reference by far more than
    the kernel's 2^8 slack, so the bf16 forward must take its rescale path
    (the online-softmax update of Alg. 1) on many tiles, and on several tiles in
    a row for the same wave.  A host model of the kernel's decision rule checks
    that it does for these exact inputs; O, LSE and the gradients (which read the
    LSE the rescaled rows produce) are compared with the oracle.

    In rows that one key dominates, the exact dS of that key is ~1e-5 while the
    bf16 rounding of the stored O moves dP - Delta by ~1e-2 (Alg. 2 reads O back
    from HBM for Delta), so those rows' gradients are set by that rounding: the
    oracle's backward here takes Delta from its own O rounded to bf16."""
    import fwd_rescale_model
    print(f"forward rescale path d={d} L={L} gate={gate}", flush=True)
    B, H = 2, 2
    x = inputs.rescale_inputs(B, H, L, d, "bf16", gate, 1500 + L, device=DEV)
    s = fox.default_scale(d)
    c, o, lse = gpu_forward(x, s)
    got = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    kept = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    xc = cpu(x)
    cc = c.cpu()
    for b in range(B):
        for h in range(H):
            fired, visited, repeat = fwd_rescale_model.rescale_events(
                xc["q"][b, h], xc["k"][b, h], cc[b, h], s)
            print(f"  head {(b, h)}: rescale path on {fired} of {visited} (wave, tile) pairs, "
                  f"up to {repeat} per wave", flush=True)
            assert fired >= max(8, visited // 4) and repeat >= 2, (fired, visited, repeat)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    check_fwd("bf16", o, lse, O, LSE, f"rescale L={L}")
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s,
                          o_dtype=torch.bfloat16)
    check_bwd("bf16", got, ref, f"rescale L={L}")
    check_bwd("bf16", kept, ref, f"rescale stored L={L}")


# ----------------------------------------------------------- small backward
BWD_CASES = ([("f32", 64, L) for L in (1, 5, 64, 100)] +
             [("f32", 128, L) for L in (33, 130)] +
             [("bf16", 64, L) for L in (1, 2, 17, 63, 64, 65, 127, 128, 129, 700)] +
             [("bf16", 128, L) for L in (1, 31, 129, 333, 700)])


@pytest.mark.parametrize("dtype,d,L", BWD_CASES)
def test_backward_small(dtype, d, L):
    print(f"backward dtype={dtype} d={d} L={L}", flush=True)
    x = inputs.attn_inputs(2, 2, L, d, dtype, ("normal", 2.0, 1.0), 200 + L, device=DEV)
    s = fox.default_scale(d)
    c, o, lse = gpu_forward(x, s)
    got = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    xc = cpu(x)
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    check_bwd(dtype, got, ref, f"L={L}")
    assert float(got[3][..., 0].abs().max()) <= 1e-3 * max(1.0, float(ref[3].abs().max()))


@pytest.mark.parametrize("gate", sorted(GATES))
def test_backward_gate_regimes(gate):
    print(f"backward gate={gate}", flush=True)
    x = inputs.attn_inputs(1, 4, 260, 64, "bf16", GATES[gate], 11, device=DEV)
    s = fox.default_scale(64)
    c, o, lse = gpu_forward(x, s)
    got = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    xc = cpu(x)
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    if gate == "full":
        # dQ = dK = 0 and d(log f) ~ 0 exactly in the limit; compare absolutely
        assert max_abs(got[0], ref[0]) <= 1e-3 and max_abs(got[1], ref[1]) <= 1e-3
        assert rel_l2(got[2], ref[2]) <= 2e-2
        assert max_abs(got[3], ref[3]) <= 1e-3
    else:
        check_bwd("bf16", got, ref, gate)


def test_backward_is_deterministic():
    x = inputs.attn_inputs(2, 2, 777, 128, "bf16", ("normal", 1.0, 1.0), 5, device=DEV)
    s = fox.default_scale(128)
    c, o, lse = gpu_forward(x, s)
    a = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    b = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    for u, w in zip(a, b):
        assert torch.equal(u, w)


# ------------------------------------------------- backward keeping dS
STORED_CASES = ([(2, 2, 64, L) for L in (1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 257, 700)] +
                [(2, 2, 128, L) for L in (1, 31, 129, 333, 700, 1000)] +
                [(1, 3, 128, 513), (3, 1, 64, 1100)])


@pytest.mark.parametrize("B,H,d,L", STORED_CASES)
def test_backward_stored_small(B, H, d, L):
    """fox_attn_bwd_stored against the oracle; its dK/dV pass is the recompute
    path's (bit for bit), and no read touches a stored slot the dK/dV pass did
    not write (the workspace starts as NaN patterns)."""
    print(f"backward stored B={B} H={H} d={d} L={L}", flush=True)
    x = inputs.attn_inputs(B, H, L, d, "bf16", ("normal", 2.0, 1.0), 300 + L, device=DEV)
    s = fox.default_scale(d)
    c, o, lse = gpu_forward(x, s)
    need = fox.fox_attn_bwd_stored_workspace_bytes(torch.bfloat16, B, H, L, d)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
    got = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s, workspace=ws)
    base = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    assert torch.equal(got[1], base[1]) and torch.equal(got[2], base[2])
    for t in got:
        assert bool(torch.isfinite(t).all())
    xc = cpu(x)
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    check_bwd("bf16", got, ref, f"stored L={L}")
    # sum(dc) = d(log f)_1 = 0: dc^q and dc^k are the row and column sums of one matrix
    assert float(got[3][..., 0].abs().max()) <= 1e-3 * max(1.0, float(ref[3].abs().max()))


def test_backward_stored_stages_equal_fused_entry_point():
    """fox_attn_bwd_stored == delta -> dkdv_store -> dq_stored -> d(log f), bit
    for bit; dkdv_store's dK, dV, dc_k equal fox_attn_bwd_dkdv's."""
    for d in (128, 64):
        x = inputs.attn_inputs(2, 3, 333, d, "bf16", ("normal", 1.0, 1.0), 78, device=DEV)
        s = fox.default_scale(d)
        c, o, lse = gpu_forward(x, s)
        ref = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
        delta = fox.fox_attn_bwd_delta(o, x["do"])
        store = torch.empty(fox.fox_attn_bwd_ds_store_bytes(torch.bfloat16, 2, 3, 333, d),
                            dtype=torch.uint8, device=DEV)
        dk, dv, dck = fox.fox_attn_bwd_dkdv_store(x["q"], x["k"], x["v"], c, lse, x["do"], delta,
                                                  store, s)
        dk2, dv2, dck2 = fox.fox_attn_bwd_dkdv(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s)
        dq, dcq = fox.fox_attn_bwd_dq_stored(x["k"], store, s)
        dlf = fox.fox_dlogf_from_dc(dcq, dck)
        torch.cuda.synchronize()
        for a, b in zip(ref, (dq, dk, dv, dlf)):
            assert torch.equal(a, b), d
        for a, b in zip((dk, dv, dck), (dk2, dv2, dck2)):
            assert torch.equal(a, b), d


def test_backward_stored_is_deterministic():
    x = inputs.attn_inputs(2, 2, 777, 128, "bf16", ("normal", 1.0, 1.0), 5, device=DEV)
    s = fox.default_scale(128)
    c, o, lse = gpu_forward(x, s)
    a = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    b = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    for u, w in zip(a, b):
        assert torch.equal(u, w)


# ------------------------------------------------------------------- decode
@pytest.mark.parametrize("dtype,d,T", [("bf16", 128, 1), ("bf16", 128, 2), ("bf16", 128, 100),
                                       ("bf16", 64, 1000), ("bf16", 128, 5000),
                                       ("f32", 64, 77), ("f32", 128, 3000)])
def test_decode_small(dtype, d, T):
    print(f"decode dtype={dtype} d={d} T={T}", flush=True)
    B, H = 3, 2
    y = inputs.decode_inputs(B, H, T, d, dtype, ("normal", 3.0, 1.0), 300 + T, device=DEV)
    cc = torch.full((B, H, T), float("nan"), device=DEV)
    if T > 1:
        cc[..., : T - 1] = fox.fox_gate_prefix(y["cached_logit"])
    o, lse = fox.fox_attn_decode(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"])
    torch.cuda.synchronize()
    yc = cpu(y)
    o_ref, lse_ref, cT_ref = oracle.decode(yc["q"], yc["k_cache"], yc["v_cache"],
                                           yc["cached_logit"], yc["logit_new"], fox.default_scale(d))
    if dtype == "f32":
        assert max_abs(o, o_ref) <= 1e-4 and max_abs(lse, lse_ref) <= 1e-4
    else:
        assert rel_l2(o, o_ref) <= 1e-2 and max_abs(lse, lse_ref) <= 1e-2
    assert max_abs(cc[..., T - 1], cT_ref) <= 1e-5 * max(1.0, float(cT_ref.abs().max())) * 8


def test_decode_equals_last_forward_row():
    T, d = 1500, 128
    x = inputs.attn_inputs(2, 2, T, d, "bf16", ("normal", 3.0, 1.0), 9, device=DEV, grad=False)
    s = fox.default_scale(d)
    c, o, lse = gpu_forward(x, s)
    cc = c.clone()
    cc[..., T - 1] = float("nan")
    od, lsed = fox.fox_attn_decode(x["q"][:, :, T - 1].contiguous(), x["k"], x["v"], cc,
                                   x["logit"][..., T - 1].contiguous(), s)
    torch.cuda.synchronize()
    assert rel_l2(od, o[:, :, T - 1]) <= 1e-2
    assert max_abs(lsed, lse[..., T - 1]) <= 1e-3
    assert max_abs(cc[..., T - 1], c[..., T - 1]) <= 1e-3


# ------------------------------------------------------- full-size workloads
W = inputs.WORKLOADS


def test_workload_fwd_f32_b1_h2_l256_d64():
    w = W["fwd_f32_b1_h2_l256_d64"]
    x = inputs.workload_inputs(w, device=DEV)
    s = fox.default_scale(w.d)
    _, o, lse = gpu_forward(x, s)
    torch.cuda.synchronize()
    xc = cpu(x)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    check_fwd("f32", o, lse, O, LSE, w.name)


def test_workload_fwdbwd_bf16_b8_h12_l2048_d64():
    w = W["fwdbwd_bf16_b8_h12_l2048_d64"]
    x = inputs.workload_inputs(w, device=DEV)
    s = fox.default_scale(w.d)
    c, o, lse = gpu_forward(x, s)
    got = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    kept = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
    torch.cuda.synchronize()
    xc = cpu(x)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    check_fwd("bf16", o, lse, O, LSE, w.name)
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    check_bwd("bf16", [t.cpu() for t in got], ref, w.name)
    check_bwd("bf16", [t.cpu() for t in kept], ref, w.name + " (stored dS)")
    assert torch.equal(kept[1], got[1]) and torch.equal(kept[2], got[2])


def test_workload_fwd_bf16_b1_h16_l65536_d128():
    w = W["fwd_bf16_b1_h16_l65536_d128"]
    x = inputs.workload_inputs(w, device=DEV)
    s = fox.default_scale(w.d)
    c, o, lse = gpu_forward(x, s)
    torch.cuda.synchronize()
    L = w.L
    g = torch.Generator().manual_seed(1)
    rows = sorted(set([0, 1, 63, 64, 127, 128, L - 129, L - 2, L - 1] +
                      torch.randint(0, L, (39,), generator=g).tolist()))
    num = den = 0.0
    for h in range(w.H):                          # both gate groups
        sl = {k: v[:, h:h + 1].cpu() for k, v in x.items()}
        O, LSE = oracle.forward(sl["q"], sl["k"], sl["v"], sl["logit"], s, rows=rows)
        check_fwd("bf16", o[:, h:h + 1, rows], lse[:, h:h + 1, rows], O, LSE, f"head {h}")
        num += float(((o[:, h:h + 1, rows].double().cpu() - O) ** 2).sum())
        den += float((O ** 2).sum())
    # the sampled rows of all heads together
    assert math.sqrt(num / den) <= 1e-2


def test_backward_stages_equal_fused_entry_point():
    """fox_attn_bwd == delta -> dkdv -> dq -> d(log f) stages, bit for bit."""
    for dtype, d in (("bf16", 128), ("bf16", 64), ("f32", 64)):
        x = inputs.attn_inputs(2, 3, 333, d, dtype, ("normal", 1.0, 1.0), 77, device=DEV)
        s = fox.default_scale(d)
        c, o, lse = gpu_forward(x, s)
        ref = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o, lse, x["do"], s)
        delta = fox.fox_attn_bwd_delta(o, x["do"])
        dk, dv, dck = fox.fox_attn_bwd_dkdv(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s)
        dq, dcq = fox.fox_attn_bwd_dq(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s)
        dlf = fox.fox_dlogf_from_dc(dcq, dck)
        torch.cuda.synchronize()
        for a, b in zip(ref, (dq, dk, dv, dlf)):
            assert torch.equal(a, b), dtype


# ------------------------------------------------------------ gate backward
@pytest.mark.parametrize("dtype,d,L", [("f32", 64, 100), ("bf16", 64, 1), ("bf16", 64, 129),
                                       ("bf16", 128, 700), ("bf16", 128, 4100)])
def test_gate_logit_gradient(dtype, d, L):
    """d(logit) = d(log f) * sigmoid(-logit), fused into the reverse scan, against
    the oracle; its d(log f) output equals fox_dlogf_from_dc bit for bit."""
    print(f"gate logit gradient dtype={dtype} d={d} L={L}", flush=True)
    x = inputs.attn_inputs(2, 2, L, d, dtype, ("normal", 2.0, 1.5), 300 + L, device=DEV)
    s = fox.default_scale(d)
    c, o, lse = gpu_forward(x, s)
    delta = fox.fox_attn_bwd_delta(o, x["do"])
    _, _, dck = fox.fox_attn_bwd_dkdv(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s)
    _, dcq = fox.fox_attn_bwd_dq(x["q"], x["k"], x["v"], c, lse, x["do"], delta, s)
    dlf_ref_gpu = fox.fox_dlogf_from_dc(dcq, dck)
    dx, dlf = fox.fox_dlogit_from_dc(dcq, dck, x["logit"], d_log_f=torch.empty_like(dcq))
    dx_only = fox.fox_dlogit_from_dc(dcq, dck, x["logit"])
    torch.cuda.synchronize()
    assert torch.equal(dlf, dlf_ref_gpu)
    assert torch.equal(dx, dx_only)
    xc = cpu(x)
    ref = oracle.backward_logit(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)[3]
    check_grad(dtype, "dlogit", dx, ref, f"L={L}")
    assert float(dx[..., 0].abs().max()) <= 1e-3 * max(1.0, float(ref.abs().max()))


# ------------------------------------------------------------- fixed gates
FIXED_CASES = [("f32", 64, 100, 2.0, 128.0), ("bf16", 64, 129, 2.0, 128.0),
               ("bf16", 128, 700, 2.0, 64.0), ("bf16", 128, 3000, 8.0, 4096.0)]


@pytest.mark.parametrize("dtype,d,L,tmin,tmax", FIXED_CASES)
def test_fixed_gate_forward_backward(dtype, d, L, tmin, tmax):
    """Fixed gates f = sigmoid(b) (ALiBi form) with the paper's initialisation:
    O, LSE, dQ, dK, dV and d b against the oracle."""
    print(f"fixed gate dtype={dtype} d={d} L={L} T=({tmin},{tmax})", flush=True)
    B, H = 2, 4
    x = inputs.attn_inputs(B, H, L, d, dtype, ("normal", 2.0, 1.0), 400 + L, device=DEV)
    b = fox.fox_fixed_gate_init(H, tmin, tmax).to(DEV)
    s = fox.default_scale(d)
    o, lse = fox.fox_attn_fwd_fixed_gate(x["q"], x["k"], x["v"], b, s)
    dq, dk, dv, db = fox.fox_attn_bwd_fixed_gate(x["q"], x["k"], x["v"], b, o, lse, x["do"], s)
    torch.cuda.synchronize()
    xc = cpu(x)
    bc = b.cpu()
    O, LSE = oracle.forward_fixed_gate(xc["q"], xc["k"], xc["v"], bc, s)
    check_fwd(dtype, o, lse, O, LSE, f"fixed L={L}")
    ref = oracle.backward_fixed_gate(xc["q"], xc["k"], xc["v"], bc, xc["do"], s)
    for name, g, r in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref[:3]):
        check_grad(dtype, name, g, r, f"fixed L={L}")
    # d b sums d(log f) over B * L positions: compare against its own scale
    tol = 1e-4 if dtype == "f32" else 2e-2
    err = max_abs(db, ref[3]) / max(1e-6, float(ref[3].abs().max()))
    assert err <= tol, f"fixed L={L} d_bias rel error {err:.3e}"
    if dtype == "bf16":
        # keeping dS: dK, dV bit for bit, the rest against the oracle (NaN-filled workspace)
        need = fox.fox_attn_bwd_fixed_gate_stored_workspace_bytes(torch.bfloat16, B, H, L, d)
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
        sq, sk, sv, sb = fox.fox_attn_bwd_fixed_gate_stored(x["q"], x["k"], x["v"], b, o, lse,
                                                            x["do"], s, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(sk, dk) and torch.equal(sv, dv)
        check_grad(dtype, "dQ", sq, ref[0], f"fixed stored L={L}")
        err = max_abs(sb, ref[3]) / max(1e-6, float(ref[3].abs().max()))
        assert err <= tol, f"fixed stored L={L} d_bias rel error {err:.3e}"
    # the same gates through the data-dependent path (constant logits = b)
    logit = b[None, :, None].expand(B, H, L).contiguous()
    c = fox.fox_gate_prefix(logit)
    o2, _ = fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s)
    torch.cuda.synchronize()
    assert rel_l2(o2, o.double()) <= (1e-5 if dtype == "f32" else 1e-2)


@pytest.mark.parametrize("dtype,d,T", [("f32", 64, 77), ("bf16", 128, 1), ("bf16", 128, 5000)])
def test_fixed_gate_decode(dtype, d, T):
    """Fixed-gate decode equals the last row of the fixed-gate oracle forward."""
    print(f"fixed gate decode dtype={dtype} d={d} T={T}", flush=True)
    B, H = 3, 4
    x = inputs.attn_inputs(B, H, T, d, dtype, ("normal", 2.0, 1.0), 500 + T, device=DEV)
    b = fox.fox_fixed_gate_init(H, 2.0, 256.0).to(DEV)
    s = fox.default_scale(d)
    q_last = x["q"][:, :, T - 1].contiguous()
    o, lse = fox.fox_attn_decode_fixed_gate(q_last, x["k"], x["v"], b, s)
    torch.cuda.synchronize()
    xc = cpu(x)
    O, LSE = oracle.forward_fixed_gate(xc["q"], xc["k"], xc["v"], b.cpu(), s, rows=[T - 1])
    check_fwd(dtype, o, lse, O[:, :, 0], LSE[:, :, 0], f"fixed decode T={T}")


# ------------------------------------------------------ gate-aware skipping
@pytest.mark.parametrize("dtype,d,L", [("bf16", 128, 1), ("bf16", 64, 3000), ("f32", 128, 1000)])
def test_row_norm_max(dtype, d, L):
    x = inputs.attn_inputs(2, 3, L, d, dtype, ("normal", 0.0, 1.0), 600 + L, device=DEV)["k"]
    got = fox.fox_row_norm_max(x)
    torch.cuda.synchronize()
    ref = torch.linalg.vector_norm(x.double().cpu(), dim=-1).amax(dim=-1)
    g = got.double().cpu()
    assert torch.all(g >= ref) and torch.all(g <= ref * (1 + 2e-3))


DECODE_SKIP_CASES = [
    # (dtype, d, B, H, T, gate (kind, mean, std)): strong gates skip almost all
    # splits, weak gates none, the workload's N(3, 1) the distant past only
    ("bf16", 128, 2, 4, 20000, ("normal", 3.0, 1.0)),
    ("bf16", 128, 2, 2, 9000, ("normal", -2.0, 1.0)),
    ("bf16", 64, 3, 2, 5000, ("normal", 12.0, 1.0)),
    ("f32", 64, 2, 2, 7777, ("normal", 1.0, 1.0)),
    ("bf16", 128, 1, 1, 1, ("normal", 3.0, 1.0)),
]


@pytest.mark.parametrize("dtype,d,B,H,T,gate", DECODE_SKIP_CASES)
def test_decode_skip_is_bitwise_dense(dtype, d, B, H, T, gate):
    """Skipping only drops splits whose merge weight is an exact zero, so o, lse
    and the appended c_T equal the dense decode's bit for bit."""
    print(f"decode skip dtype={dtype} d={d} B={B} H={H} T={T} gate={gate}", flush=True)
    y = inputs.decode_inputs(B, H, T, d, dtype, gate, 700 + T, device=DEV)
    cc = torch.zeros((B, H, T), device=DEV)
    if T > 1:
        cc[..., : T - 1] = fox.fox_gate_prefix(y["cached_logit"])
    cc2 = cc.clone()
    kn = fox.fox_row_norm_max(y["k_cache"])
    o1, l1 = fox.fox_attn_decode(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"])
    o2, l2 = fox.fox_attn_decode_skip(y["q"], y["k_cache"], y["v_cache"], cc2, y["logit_new"], kn)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2) and torch.equal(cc, cc2)
    # the skipping decode on its own against the oracle
    yc = cpu(y)
    o_ref, lse_ref, cT_ref = oracle.decode(yc["q"], yc["k_cache"], yc["v_cache"],
                                           yc["cached_logit"], yc["logit_new"],
                                           fox.default_scale(d))
    check_fwd(dtype, o2, l2, o_ref, lse_ref, f"decode skip T={T}",
              c_abs=float(cT_ref.abs().max()), L=T)
    assert max_abs(cc2[..., T - 1], cT_ref) <= 1e-5 * max(1.0, float(cT_ref.abs().max())) * 8


SKIP_CASES = [
    ("bf16", 128, 2, 3, 3000, ("normal", 1.0, 1.0)),
    ("bf16", 64, 2, 2, 4100, ("normal", -3.0, 1.0)),
    ("bf16", 128, 1, 4, 2500, ("head_mean_uniform", 0.0, 6.0, 1.0)),
    ("bf16", 64, 1, 2, 1000, ("normal", 8.0, 1.0)),
    ("bf16", 128, 1, 1, 1, ("normal", 1.0, 1.0)),
    ("f32", 64, 1, 2, 300, ("normal", -2.0, 1.0)),
    # B*H a multiple of 8: the skipping backward runs on its work plan
    ("bf16", 128, 2, 4, 2000, ("head_mean_uniform", 0.0, 6.0, 1.0)),
    ("bf16", 64, 1, 16, 1000, ("normal", -1.0, 1.0)),
]


@pytest.mark.parametrize("dtype,d,B,H,L,gate", SKIP_CASES)
def test_fwd_bwd_skip_is_bitwise_dense(dtype, d, B, H, L, gate):
    """Exact gate-aware skipping drops only tile pairs whose contributions are
    fp32 zeros: O, LSE, dQ, dK, dV, d(log f) equal the dense results bit for bit."""
    print(f"fwd/bwd skip dtype={dtype} d={d} B={B} H={H} L={L} gate={gate}", flush=True)
    x = inputs.attn_inputs(B, H, L, d, dtype, gate, 800 + L, device=DEV)
    s = fox.default_scale(d)
    c = fox.fox_gate_prefix(x["logit"])
    qn, kn = fox.fox_row_norm_max(x["q"]), fox.fox_row_norm_max(x["k"])
    o1, l1 = fox.fox_attn_fwd(x["q"], x["k"], x["v"], c, s)
    o2, l2 = fox.fox_attn_fwd_skip(x["q"], x["k"], x["v"], c, qn, kn, s)
    g1 = fox.fox_attn_bwd(x["q"], x["k"], x["v"], c, o1, l1, x["do"], s)
    g2 = fox.fox_attn_bwd_skip(x["q"], x["k"], x["v"], c, o1, l1, x["do"], qn, kn, s)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for name, a, b in zip(("dq", "dk", "dv", "dlogf"), g1, g2):
        assert torch.equal(a, b), name
    g4 = None
    if dtype == "bf16":
        # keeping dS: the skipping dQ pass reads only the slots the skipping dK/dV
        # pass wrote (the workspace starts as NaN patterns)
        need = fox.fox_attn_bwd_stored_workspace_bytes(torch.bfloat16, B, H, L, d)
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
        g3 = fox.fox_attn_bwd_stored(x["q"], x["k"], x["v"], c, o1, l1, x["do"], s)
        g4 = fox.fox_attn_bwd_skip_stored(x["q"], x["k"], x["v"], c, o1, l1, x["do"], qn, kn, s,
                                          workspace=ws)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv", "dlogf"), g3, g4):
            assert torch.equal(a, b), f"stored {name}"
    # the skipping outputs on their own against the oracle
    xc = cpu(x)
    O, LSE = oracle.forward(xc["q"], xc["k"], xc["v"], xc["logit"], s)
    c_abs = float(oracle.prefix_c(oracle.log_sigmoid(xc["logit"])).abs().max())
    check_fwd(dtype, o2, l2, O, LSE, f"skip L={L}", c_abs=c_abs, L=L)
    ref = oracle.backward(xc["q"], xc["k"], xc["v"], xc["logit"], xc["do"], s)
    check_bwd(dtype, [t.cpu() for t in g2], ref, f"skip L={L}")
    if g4 is not None:
        check_bwd(dtype, [t.cpu() for t in g4], ref, f"skip stored L={L}")


FIXED_SKIP_CASES = [("bf16", 128, 2, 4, 3000, 2.0, 64.0), ("bf16", 64, 1, 3, 4100, 8.0, 4096.0),
                    ("bf16", 128, 1, 2, 1, 2.0, 4.0), ("f32", 64, 1, 2, 300, 2.0, 16.0)]


@pytest.mark.parametrize("dtype,d,B,H,L,tmin,tmax", FIXED_SKIP_CASES)
def test_fixed_gate_skip_is_bitwise_dense(dtype, d, B, H, L, tmin, tmax):
    """Fixed gates with exact skipping: O, LSE, dQ, dK, dV, d b and one decode step
    (the last row against the whole sequence as cache) equal the fixed-gate entry
    points without skipping bit for bit."""
    print(f"fixed skip dtype={dtype} d={d} B={B} H={H} L={L} T=({tmin},{tmax})", flush=True)
    x = inputs.attn_inputs(B, H, L, d, dtype, ("normal", 0.0, 1.0), 1300 + L, device=DEV)
    s = fox.default_scale(d)
    b = fox.fox_fixed_gate_init(H, tmin, tmax).to(DEV)
    qn, kn = fox.fox_row_norm_max(x["q"]), fox.fox_row_norm_max(x["k"])
    o1, l1 = fox.fox_attn_fwd_fixed_gate(x["q"], x["k"], x["v"], b, s)
    o2, l2 = fox.fox_attn_fwd_fixed_gate_skip(x["q"], x["k"], x["v"], b, qn, kn, s)
    g1 = fox.fox_attn_bwd_fixed_gate(x["q"], x["k"], x["v"], b, o1, l1, x["do"], s)
    g2 = fox.fox_attn_bwd_fixed_gate_skip(x["q"], x["k"], x["v"], b, o1, l1, x["do"], qn, kn, s)
    if dtype == "bf16":
        need = fox.fox_attn_bwd_fixed_gate_stored_workspace_bytes(torch.bfloat16, B, H, L, d)
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
        g3 = fox.fox_attn_bwd_fixed_gate_stored(x["q"], x["k"], x["v"], b, o1, l1, x["do"], s)
        g4 = fox.fox_attn_bwd_fixed_gate_skip_stored(x["q"], x["k"], x["v"], b, o1, l1, x["do"],
                                                     qn, kn, s, workspace=ws)
    qd = x["q"][:, :, -1].contiguous()
    d1 = fox.fox_attn_decode_fixed_gate(qd, x["k"], x["v"], b, s)
    d2 = fox.fox_attn_decode_fixed_gate_skip(qd, x["k"], x["v"], b, kn, s)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for name, a, c in zip(("dq", "dk", "dv", "db"), g1, g2):
        assert torch.equal(a, c), name
    assert torch.equal(d1[0], d2[0]) and torch.equal(d1[1], d2[1])
    if dtype == "bf16":
        for name, a, c in zip(("dq", "dk", "dv", "db"), g3, g4):
            assert torch.equal(a, c), f"stored {name}"
        assert torch.equal(g3[1], g1[1]) and torch.equal(g3[2], g1[2])
    # the skipping outputs on their own against the oracle
    xc = cpu(x)
    bc = b.cpu()
    O, LSE = oracle.forward_fixed_gate(xc["q"], xc["k"], xc["v"], bc, s)
    check_fwd(dtype, o2, l2, O, LSE, f"fixed skip L={L}")
    check_fwd(dtype, d2[0], d2[1], O[:, :, -1], LSE[:, :, -1], f"fixed skip decode L={L}")
    ref = oracle.backward_fixed_gate(xc["q"], xc["k"], xc["v"], bc, xc["do"], s)
    tol = 1e-4 if dtype == "f32" else 2e-2
    for tag, grads in (("", g2),) + ((("stored ", g4),) if dtype == "bf16" else ()):
        for name, g_, r in zip(("dQ", "dK", "dV"), grads[:3], ref[:3]):
            check_grad(dtype, name, g_, r, f"fixed skip {tag}L={L}")
        err = max_abs(grads[3], ref[3]) / max(1e-6, float(ref[3].abs().max()))
        assert err <= tol, f"fixed skip {tag}L={L} d_bias rel error {err:.3e}"


# ------------------------------------------------------------ FoX (Pro) layer
PRO_EPS = 1e-6
PRO_GATE = ("normal", 2.0, 1.0)


def check_out(dtype, name, g, r, what=""):
    """Forward outputs: fp32 max-abs <= 1e-4, bf16 relative L2 <= 1e-2."""
    if dtype == "f32":
        e = max_abs(g, r)
        assert e <= 1e-4, f"{what} {name} max-abs {e:.3e}"
    else:
        e = rel_l2(g, r)
        assert e <= 1e-2, f"{what} {name} rel-L2 {e:.3e}"


PRO_CASES = [("f32", 64, 1), ("f32", 128, 300), ("bf16", 64, 2), ("bf16", 128, 257),
             ("bf16", 64, 1000), ("bf16", 128, 513)]


@pytest.mark.parametrize("dtype,d,L", PRO_CASES)
def test_pro_prologue_forward_backward(dtype, d, L):
    print(f"pro prologue dtype={dtype} d={d} L={L}", flush=True)
    x = inputs.pro_inputs(2, 3, L, d, dtype, PRO_GATE, 700 + L, device=DEV)
    args = (x["q_raw"], x["k_raw"], x["v_raw"], x["k_shift"], x["v_shift"], x["wq"], x["wk"])
    q, k, v = fox.fox_pro_prologue(*args, eps=PRO_EPS)
    grads = fox.fox_pro_prologue_bwd(*args, x["dq"], x["dk"], x["dv"], eps=PRO_EPS)
    torch.cuda.synchronize()
    xc = cpu(x)
    cargs = (xc["q_raw"], xc["k_raw"], xc["v_raw"], xc["k_shift"], xc["v_shift"], xc["wq"],
             xc["wk"], PRO_EPS)
    for name, g, r in zip("qkv", (q, k, v), oracle.pro_prologue(*cargs)):
        check_out(dtype, name, g, r, f"L={L}")
    ref = oracle.pro_prologue_backward(*cargs, xc["dq"], xc["dk"], xc["dv"])
    names = ("dq_raw", "dk_raw", "dv_raw", "dk_shift", "dv_shift", "dwq", "dwk")
    for name, g, r in zip(names, grads, ref):
        if L == 1 and name == "dk_shift":
            # one token: k = RMSNorm((1 - a) k~_1) depends on a only through
            # eps, so the exact gradient is a small difference of large terms
            # (eps / mean square); bound the fp32 cancellation absolutely
            assert max_abs(g, r) <= (2e-5 if dtype == "f32" else 1e-4), max_abs(g, r)
            continue
        check_grad(dtype, name, g, r, f"L={L}")


@pytest.mark.parametrize("dtype,d,L", [("f32", 64, 100), ("f32", 128, 257), ("bf16", 64, 1),
                                       ("bf16", 128, 333), ("bf16", 64, 1000)])
def test_pro_attention_forward_backward(dtype, d, L):
    """Attention with the output norm and gate (fused into the bf16 forward's
    epilogue; its backward fused with Delta) against the oracle's chain."""
    print(f"pro attention dtype={dtype} d={d} L={L}", flush=True)
    x = inputs.pro_inputs(2, 3, L, d, dtype, PRO_GATE, 800 + L, device=DEV)
    q, k, v = x["q_raw"], x["k_raw"], x["v_raw"]  # any q, k, v will do here
    s = fox.default_scale(d)
    c = fox.fox_gate_prefix(x["logit"])
    y, o, lse = fox.fox_attn_fwd_pro(q, k, v, c, x["g"], x["wo"], s, eps=PRO_EPS)
    grads = fox.fox_attn_bwd_pro(q, k, v, c, o, lse, x["g"], x["wo"], x["dy"], s, eps=PRO_EPS)
    y_sep = fox.fox_pro_output_gate(o, x["g"], x["wo"], eps=PRO_EPS)
    torch.cuda.synchronize()
    xc = cpu(x)
    Y, O, LSE = oracle.pro_forward(xc["q_raw"], xc["k_raw"], xc["v_raw"], xc["logit"], xc["g"],
                                   xc["wo"], PRO_EPS, s)
    check_fwd(dtype, o, lse, O, LSE, f"L={L}")
    check_out(dtype, "y", y, Y, f"L={L}")
    # the fused epilogue and the standalone kernel normalise the same stored O
    assert rel_l2(y, y_sep) <= (1e-6 if dtype == "f32" else 4e-3), rel_l2(y, y_sep)
    ref = oracle.pro_backward(xc["q_raw"], xc["k_raw"], xc["v_raw"], xc["logit"], xc["g"],
                              xc["wo"], PRO_EPS, s, xc["dy"])
    for name, g, r in zip(("dQ", "dK", "dV", "dlogf", "dg", "dwo"), grads, ref):
        check_grad(dtype, name, g, r, f"L={L}")
    if dtype == "bf16":
        # the same backward keeping dS: dK, dV, dg, dwo bit for bit, dQ and
        # d(log f) to rounding; the workspace starts as NaN patterns
        need = fox.fox_attn_bwd_pro_stored_workspace_bytes(torch.bfloat16, 2, 3, L, d)
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device=DEV)
        kept = fox.fox_attn_bwd_pro_stored(q, k, v, c, o, lse, x["g"], x["wo"], x["dy"], s,
                                           eps=PRO_EPS, workspace=ws)
        torch.cuda.synchronize()
        for i in (1, 2, 4, 5):
            assert torch.equal(kept[i], grads[i]), i
        for name, g, r in zip(("dQ", "dK", "dV", "dlogf", "dg", "dwo"), kept, ref):
            check_grad(dtype, name, g, r, f"stored L={L}")


def test_pro_layer_chain_bf16():
    """Prologue -> attention with output norm and gate -> backward -> prologue
    backward, against the oracle's chain (every gradient of the Pro layer)."""
    B, H, L, d = 2, 4, 700, 128
    x = inputs.pro_inputs(B, H, L, d, "bf16", ("head_mean_uniform", 0.0, 6.0, 1.0), 901,
                          device=DEV)
    s = fox.default_scale(d)
    pargs = (x["q_raw"], x["k_raw"], x["v_raw"], x["k_shift"], x["v_shift"], x["wq"], x["wk"])
    q, k, v = fox.fox_pro_prologue(*pargs, eps=PRO_EPS)
    c = fox.fox_gate_prefix(x["logit"])
    y, o, lse = fox.fox_attn_fwd_pro(q, k, v, c, x["g"], x["wo"], s, eps=PRO_EPS)
    dq, dk, dv, dlf, dg, dwo = fox.fox_attn_bwd_pro(q, k, v, c, o, lse, x["g"], x["wo"], x["dy"],
                                                    s, eps=PRO_EPS)
    pg = fox.fox_pro_prologue_bwd(*pargs, dq, dk, dv, eps=PRO_EPS)
    torch.cuda.synchronize()
    xc = cpu(x)
    cq, ck, cv = oracle.pro_prologue(xc["q_raw"], xc["k_raw"], xc["v_raw"], xc["k_shift"],
                                     xc["v_shift"], xc["wq"], xc["wk"], PRO_EPS)
    Y, _, _ = oracle.pro_forward(cq, ck, cv, xc["logit"], xc["g"], xc["wo"], PRO_EPS, s)
    check_out("bf16", "y", y, Y)
    rq, rk, rv, rlf, rg, rwo = oracle.pro_backward(cq, ck, cv, xc["logit"], xc["g"], xc["wo"],
                                                   PRO_EPS, s, xc["dy"])
    rp = oracle.pro_prologue_backward(xc["q_raw"], xc["k_raw"], xc["v_raw"], xc["k_shift"],
                                      xc["v_shift"], xc["wq"], xc["wk"], PRO_EPS, rq, rk, rv)
    got = (dlf, dg, dwo) + tuple(pg)
    ref = (rlf, rg, rwo) + tuple(rp)
    names = ("dlogf", "dg", "dwo", "dq_raw", "dk_raw", "dv_raw", "dk_shift", "dv_shift", "dwq",
             "dwk")
    for name, g, r in zip(names, got, ref):
        check_grad("bf16", name, g, r, "chain")


def test_workload_pro_bf16_b2_h16_l16384_d128():
    """The FoX (Pro) layer at the benchmark's shape and launch configuration.  The
    prologue and the output norm/gate are row-local, so the oracle checks them on
    whole heads: the prologue forward and backward on the slices of head 15 (its
    weight gradients sum over both batch rows), y on sampled query rows (oracle
    attention rows, then the output norm and gate), the norm/gate backward (dg,
    dw_o) on every row of head 15 from the stored O; the attention backward that
    follows it equals fox_attn_bwd fed the oracle's dO."""
    w = W["fwdbwd_bf16_b2_h16_l16384_d128"]
    B, H, L, d = w.B, w.H, w.L, w.d
    x = inputs.pro_inputs(B, H, L, d, w.dtype, w.gate, w.seed + 1, device=DEV)
    s = fox.default_scale(d)
    pargs = (x["q_raw"], x["k_raw"], x["v_raw"], x["k_shift"], x["v_shift"], x["wq"], x["wk"])
    q, k, v = fox.fox_pro_prologue(*pargs, eps=PRO_EPS)
    c = fox.fox_gate_prefix(x["logit"])
    y, o, lse = fox.fox_attn_fwd_pro(q, k, v, c, x["g"], x["wo"], s, eps=PRO_EPS)
    dq, dk, dv, dlf, dg, dwo = fox.fox_attn_bwd_pro(q, k, v, c, o, lse, x["g"], x["wo"], x["dy"],
                                                    s, eps=PRO_EPS)
    pg = fox.fox_pro_prologue_bwd(*pargs, dq, dk, dv, eps=PRO_EPS)
    torch.cuda.synchronize()
    h = 15
    print(f"pro workload: oracle on head {h}", flush=True)
    sl = {n: t[:, h:h + 1].cpu() for n, t in x.items() if t.dim() >= 3}
    wsl = {n: x[n][h:h + 1].cpu() for n in ("wq", "wk", "wo")}
    # prologue forward and backward (both batch rows of head h)
    ref = oracle.pro_prologue(sl["q_raw"], sl["k_raw"], sl["v_raw"], sl["k_shift"],
                              sl["v_shift"], wsl["wq"], wsl["wk"], PRO_EPS)
    for name, g_, r in zip("qkv", (q, k, v), ref):
        check_out("bf16", name, g_[:, h:h + 1], r, "pro workload")
    gsl = [t[:, h:h + 1].cpu() for t in (dq, dk, dv)]
    pref = oracle.pro_prologue_backward(sl["q_raw"], sl["k_raw"], sl["v_raw"], sl["k_shift"],
                                        sl["v_shift"], wsl["wq"], wsl["wk"], PRO_EPS, *gsl)
    got = [t[:, h:h + 1] for t in pg[:5]] + [pg[5][h:h + 1], pg[6][h:h + 1]]
    for name, g_, r in zip(("dq_raw", "dk_raw", "dv_raw", "dk_shift", "dv_shift", "dwq", "dwk"),
                           got, pref):
        check_grad("bf16", name, g_, r, "pro workload")
    del ref, pref
    # y on sampled rows of (b, h) = (1, h): oracle attention rows, then the norm and gate
    rows = torch.tensor([0, 1, 63, 64, 4095, 8191, 12000, L - 2, L - 1])
    qs = [t[1, h].cpu() for t in (q, k, v)]
    O_rows, _ = oracle.forward_head_from_c(*qs, oracle.prefix_c(oracle.log_sigmoid(
        x["logit"][1, h].cpu())), s, rows=rows)
    Y_rows = oracle.output_gate(O_rows[None, None], x["g"][1, h, rows].cpu()[None, None],
                                wsl["wo"], PRO_EPS)[0, 0]
    check_out("bf16", "y rows", y[1, h, rows], Y_rows, "pro workload")
    # the norm/gate backward from the stored O (every row of head h)
    dO_h, dg_h, dwo_h = oracle.output_gate_backward(o[:, h:h + 1].cpu(), sl["g"], wsl["wo"],
                                                    PRO_EPS, sl["dy"])
    check_grad("bf16", "dg", dg[:, h:h + 1], dg_h, "pro workload")
    check_grad("bf16", "dwo", dwo[h:h + 1], dwo_h, "pro workload")
    del dO_h, dg_h
    # the attention backward behind it: fox_attn_bwd with the oracle's dO (all heads)
    dO_ref = oracle.output_gate_backward(o.cpu(), x["g"].cpu(), x["wo"].cpu(), PRO_EPS,
                                         x["dy"].cpu())[0].to(torch.bfloat16).to(DEV)
    ref2 = fox.fox_attn_bwd(q, k, v, c, o, lse, dO_ref, s)
    torch.cuda.synchronize()
    for name, g_, r in zip(("dq", "dk", "dv", "dlogf"), (dq, dk, dv, dlf), ref2):
        e = rel_l2(g_, r)
        assert e <= 1e-2, f"pro workload {name} vs fox_attn_bwd with the oracle's dO: {e:.3e}"

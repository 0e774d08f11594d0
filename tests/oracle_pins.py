"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

Every function takes the oracle module (`ora`) as an argument and raises
AssertionError when a pin fails, so that the same pins can be run both on the
real oracle (tests/test_oracle_pins.py) and on deliberately broken copies of it
(tests/test_oracle_mutants.py), which shows that a plausible mistake anywhere
in the oracle is caught by at least one pin.

The pins, with what in the paper fixes them:
  P1  log f = 0 turns Forgetting Attention into standard causal softmax
      attention (Eq. attn-softmax vs Eq. fot-weight)  -> torch SDPA (fp64) and
      its autograd gradients.
  P2  log f -> -inf (here -1e4): every off-diagonal weight vanishes, so
      o_i = v_i, LSE_i = s q_i.k_i, dQ = dK = 0, dV = dO.
  P3  a constant, head-specific gate f = exp(-m) is ALiBi with slope m
      (Sec. 3, "Connection to ALiBi") -> SDPA with the additive mask -m(i-j).
  P4  D_ii = 0, D_ij = D_ik + D_kj, D <= 0, D monotone in j; c_i - c_j equals
      the direct sum of log f over (j, i]  (Eq. fot-weight).
  P5  attention rows are probability vectors with a zero upper triangle.
  P6  first row: o_1 = v_1, LSE_1 = s q_1.k_1; L = 1 gives O = V.
  P7  O is invariant to log f_1 and to c + const; d(log f)_1 = 0; sum dc = 0;
      rowsum(dS) = 0 (softmax shift invariance).
  P8  product form prod f_l exp(s q.k) (left side of Eq. fot-weight, gates as
      sigmoid values) equals the logit-bias form (right side).
  P9  gradients equal central finite differences and torch autograd of an
      independently written forward.
  P10 rectangle identity: d(log f)_l = sum_{r>=l} sum_{j<l} dS_rj, since log f_l
      sits inside D_rj exactly when j < l <= r.
  P11 decode equals the last row of the full forward.
  P12 closed forms with q = 0: LSE_i = log i for log f = 0, and the geometric
      series log((1 - e^{-m i}) / (1 - e^{-m})) for constant log f = -m.
  P13 L = 2 written out by hand.
  P14 gate-logit gradient: central finite differences through the logits, the
      zero gradient of the first gate, and the sigmoid-derivative closed form.
  P15 fixed gates: the appendix's initialisation example (golden file), the
      equivalence with ALiBi at slopes 1/T_h, and d b by finite differences.
  P16 RMSNorm (Pro layer): unit weight and eps = 0 give rows of mean square
      exactly 1 and invariance to scaling each row; eps > 0 gives mean square
      ms / (ms + eps); each head uses its own weight row.
  P17 token shift (Eq. shift-linear): logit -> -inf is the identity, +inf the
      shift by one step with a zero first row, 0 the average of neighbours; the
      Pro prologue reduces to these with QK-norm applied.
  P18 Pro gradients: central finite differences of the prologue and of the
      output norm and gate, and torch autograd of an independently written
      Pro layer (prologue, attention, epilogue) against the oracle's chain.
  P19 output gate: g -> +inf leaves RMSNorm(o); g = 0 halves it; d g vanishes
      where the gate saturates.
"""
from __future__ import annotations

import math
import os

import torch
import torch.nn.functional as Fnn

F64 = torch.float64


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(shape, generator=g, dtype=F64) * scale


def _close(a, b, tol, what):
    a, b = torch.as_tensor(a, dtype=F64), torch.as_tensor(b, dtype=F64)
    err = (a - b).abs().max().item() if a.numel() else 0.0
    assert err <= tol, f"{what}: max-abs error {err:.3e} > {tol:.1e}"


def _sdpa_with_grads(q, k, v, dO, scale, mask=None):
    q, k, v = (t.clone().requires_grad_(True) for t in (q, k, v))
    if mask is None:
        O = Fnn.scaled_dot_product_attention(q, k, v, is_causal=True, scale=scale)
    else:
        O = Fnn.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
    gq, gk, gv = torch.autograd.grad((O * dO).sum(), (q, k, v))
    return O.detach(), gq, gk, gv


# --------------------------------------------------------------------------- P1
def pin_p1_zero_forgetting_is_softmax_attention(ora, B=2, H=3, L=37, d=16, seed=1):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    s = 1.0 / math.sqrt(d)
    lf = torch.zeros(B, H, L, dtype=F64)
    O, _ = ora.forward_from_logf(q, k, v, lf, s)
    dQ, dK, dV, _ = ora.backward_from_logf(q, k, v, lf, dO, s)
    Oref, gq, gk, gv = _sdpa_with_grads(q, k, v, dO, s)
    _close(O, Oref, 1e-12, "P1 O")
    _close(dQ, gq, 1e-12, "P1 dQ")
    _close(dK, gk, 1e-12, "P1 dK")
    _close(dV, gv, 1e-12, "P1 dV")


# --------------------------------------------------------------------------- P2
def pin_p2_full_forgetting(ora, B=1, H=2, L=19, d=8, seed=2):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    s = 0.37
    lf = torch.full((B, H, L), -1.0e4, dtype=F64)
    O, LSE = ora.forward_from_logf(q, k, v, lf, s)
    _close(O, v, 1e-12, "P2 O = V")
    _close(LSE, s * (q * k).sum(-1), 1e-12, "P2 LSE = s q.k")
    dQ, dK, dV, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    _close(dQ, torch.zeros_like(dQ), 1e-12, "P2 dQ = 0")
    _close(dK, torch.zeros_like(dK), 1e-12, "P2 dK = 0")
    _close(dV, dO, 1e-12, "P2 dV = dO")
    _close(dlf, torch.zeros_like(dlf), 1e-12, "P2 dlogf = 0")


# --------------------------------------------------------------------------- P3
def pin_p3_constant_gate_is_alibi(ora, B=1, H=4, L=29, d=8, seed=3):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    s = 1.0 / math.sqrt(d)
    m = torch.tensor([0.05, 0.3, 1.0, 2.5], dtype=F64)[:H]
    lf = (-m)[None, :, None].expand(B, H, L).clone()
    i = torch.arange(L, dtype=F64)
    dist = i[:, None] - i[None, :]
    mask = -m[:, None, None] * dist[None]
    mask = mask.masked_fill(dist[None] < 0, -math.inf)[None].expand(B, H, L, L)
    O, _ = ora.forward_from_logf(q, k, v, lf, s)
    dQ, dK, dV, _ = ora.backward_from_logf(q, k, v, lf, dO, s)
    Oref, gq, gk, gv = _sdpa_with_grads(q, k, v, dO, s, mask)
    _close(O, Oref, 1e-12, "P3 O")
    _close(dQ, gq, 1e-12, "P3 dQ")
    _close(dK, gk, 1e-12, "P3 dK")
    _close(dV, gv, 1e-12, "P3 dV")


# --------------------------------------------------------------------------- P4
def pin_p4_decay_matrix(ora, L=23, seed=4):
    x = _rand((L,), seed) * 2 + 1
    lf = ora.log_sigmoid(x)
    c = ora.prefix_c(lf)
    D = ora.decay_matrix(c)
    for i in range(L):
        for j in range(L):
            if j > i:
                assert D[i, j] == -math.inf, "P4 upper triangle must be -inf"
            else:
                direct = sum(float(lf[l]) for l in range(j + 1, i + 1))
                assert abs(D[i, j] - direct) <= 1e-12, f"P4 D[{i},{j}] != direct sum"
    assert torch.all(torch.diagonal(D) == 0), "P4 D_ii = 0"
    tri = torch.tril(torch.ones(L, L, dtype=torch.bool))
    assert torch.all(D[tri] <= 0), "P4 D <= 0"
    for i in range(L):       # monotone non-decreasing in j on the causal part
        row = D[i, : i + 1]
        assert torch.all(row[1:] >= row[:-1] - 1e-12), "P4 monotone in j"
    for (i, kk, j) in [(20, 10, 3), (5, 5, 0), (22, 1, 1)]:
        assert abs(D[i, j] - (D[i, kk] + D[kk, j])) < 1e-12, "P4 telescoping"
    # the gate values themselves: log sigmoid(x) = log(1 / (1 + exp(-x)))
    _close(lf, torch.log(1.0 / (1.0 + torch.exp(-x))), 1e-14, "P4 log sigmoid")
    _close(ora.log_sigmoid(torch.tensor([0.0, -800.0, 800.0], dtype=F64)),
           torch.tensor([-math.log(2.0), -800.0, 0.0], dtype=F64), 1e-14, "P4 log sigmoid limits")


# --------------------------------------------------------------------------- P5
def pin_p5_attention_rows(ora, L=31, d=8, seed=5):
    q, k, v = (_rand((L, d), seed + i) for i in range(3))
    c = ora.prefix_c(ora.log_sigmoid(_rand((L,), seed + 9)))
    _, _, A = ora.forward_head_from_c(q, k, v, c, 0.5, return_A=True)
    assert torch.all(A >= 0), "P5 A >= 0"
    _close(A.sum(1), torch.ones(L, dtype=F64), 1e-13, "P5 rows sum to 1")
    assert torch.all(torch.triu(A, 1) == 0), "P5 strict upper triangle is 0"


# --------------------------------------------------------------------------- P6
def pin_p6_first_row(ora, L=17, d=8, seed=6):
    q, k, v = (_rand((1, 1, L, d), seed + i) for i in range(3))
    x = _rand((1, 1, L), seed + 7)
    s = 0.21
    O, LSE = ora.forward(q, k, v, x, s)
    _close(O[0, 0, 0], v[0, 0, 0], 1e-14, "P6 o_1 = v_1")
    _close(LSE[0, 0, 0], s * (q[0, 0, 0] * k[0, 0, 0]).sum(), 1e-14, "P6 LSE_1")
    O1, _ = ora.forward(q[:, :, :1], k[:, :, :1], v[:, :, :1], x[:, :, :1], s)
    _close(O1, v[:, :, :1], 1e-14, "P6 L = 1")


# --------------------------------------------------------------------------- P7
def pin_p7_invariances(ora, B=1, H=2, L=27, d=8, seed=7):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    lf = ora.log_sigmoid(_rand((B, H, L), seed + 5) + 1)
    s = 0.33
    O, LSE = ora.forward_from_logf(q, k, v, lf, s)
    lf2 = lf.clone()
    lf2[..., 0] = -7.5
    O2, LSE2 = ora.forward_from_logf(q, k, v, lf2, s)
    _close(O, O2, 1e-13, "P7 O invariant to log f_1")
    _close(LSE, LSE2, 1e-12, "P7 LSE invariant to log f_1")
    c = ora.prefix_c(lf[0, 0])
    Oa, La = ora.forward_head_from_c(q[0, 0], k[0, 0], v[0, 0], c, s)
    Ob, Lb = ora.forward_head_from_c(q[0, 0], k[0, 0], v[0, 0], c + 123.25, s)
    _close(Oa, Ob, 1e-12, "P7 O invariant to c + const")
    _close(La, Lb, 1e-10, "P7 LSE invariant to c + const")
    _, _, _, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    _close(dlf[..., 0], torch.zeros(B, H, dtype=F64), 1e-12, "P7 d(log f)_1 = 0")
    _, _, _, dc, dS = ora.backward_head_from_c(q[0, 0], k[0, 0], v[0, 0], c, dO[0, 0], s,
                                              return_dS=True)
    _close(dc.sum(), 0.0, 1e-12, "P7 sum dc = 0")
    _close(dS.sum(1), torch.zeros(L, dtype=F64), 1e-12, "P7 rowsum dS = 0")


# --------------------------------------------------------------------------- P8
def pin_p8_product_form(ora, L=12, d=4, seed=8):
    q, k, v = (_rand((L, d), seed + i) for i in range(3))
    x = _rand((L,), seed + 3) * 1.5 + 0.5
    s = 0.6
    f = [1.0 / (1.0 + math.exp(-float(t))) for t in x]          # sigmoid gate values
    O_ref = torch.zeros(L, d, dtype=F64)
    for i in range(L):
        num = torch.zeros(d, dtype=F64)
        den = 0.0
        for j in range(i + 1):
            F = 1.0
            for l in range(j + 1, i + 1):
                F *= f[l]
            w = F * math.exp(s * float(q[i] @ k[j]))
            num += w * v[j]
            den += w
        O_ref[i] = num / den
    O, _ = ora.forward(q[None, None], k[None, None], v[None, None], x[None, None], s)
    _close(O[0, 0], O_ref, 1e-12, "P8 product form = logit-bias form")


# --------------------------------------------------------------------------- P9
def _objective(ora, q, k, v, lf, dO, s):
    O, _ = ora.forward_from_logf(q, k, v, lf, s)
    return float((O * dO).sum())


def pin_p9_finite_differences(ora, B=1, H=2, L=6, d=3, seed=9):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    lf = ora.log_sigmoid(_rand((B, H, L), seed + 5) + 0.5)
    s = 0.7
    dQ, dK, dV, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    eps = 1e-6
    for name, t, g in (("dQ", q, dQ), ("dK", k, dK), ("dV", v, dV), ("dlogf", lf, dlf)):
        flat = t.view(-1)
        gflat = g.reshape(-1)
        for idx in range(flat.numel()):
            old = float(flat[idx])
            flat[idx] = old + eps
            fp = _objective(ora, q, k, v, lf, dO, s)
            flat[idx] = old - eps
            fm = _objective(ora, q, k, v, lf, dO, s)
            flat[idx] = old
            fd = (fp - fm) / (2 * eps)
            assert abs(fd - float(gflat[idx])) <= 1e-7 * max(1.0, abs(fd)), \
                f"P9 {name}[{idx}]: finite difference {fd:.9f} vs oracle {float(gflat[idx]):.9f}"


def _autograd_forward(q, k, v, lf, s):
    """An independent autograd construction of the forward (matrix form)."""
    L = q.shape[-2]
    c = torch.cumsum(lf, dim=-1)
    D = c[..., :, None] - c[..., None, :]
    upper = torch.ones(L, L, dtype=torch.bool).triu(1)
    S = s * torch.matmul(q, k.transpose(-1, -2)) + D.masked_fill(upper, -math.inf)
    return torch.matmul(torch.softmax(S, dim=-1), v)


def pin_p9_autograd(ora, B=2, H=2, L=33, d=8, seed=19):
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    lf = ora.log_sigmoid(_rand((B, H, L), seed + 5) * 2 + 1)
    s = 0.35
    leaves = [t.clone().requires_grad_(True) for t in (q, k, v, lf)]
    O = _autograd_forward(*leaves, s)
    gq, gk, gv, glf = torch.autograd.grad((O * dO).sum(), leaves)
    dQ, dK, dV, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    _close(dQ, gq, 1e-12, "P9 autograd dQ")
    _close(dK, gk, 1e-12, "P9 autograd dK")
    _close(dV, gv, 1e-12, "P9 autograd dV")
    _close(dlf, glf, 1e-12, "P9 autograd dlogf")


# --------------------------------------------------------------------------- P10
def pin_p10_rectangle_identity(ora, L=21, d=6, seed=10):
    q, k, v, dO = (_rand((L, d), seed + i) for i in range(4))
    lf = ora.log_sigmoid(_rand((L,), seed + 5) + 1)
    c = ora.prefix_c(lf)
    _, _, _, dc, dS = ora.backward_head_from_c(q, k, v, c, dO, 0.4, return_dS=True)
    dlf = ora.reverse_cumsum(dc)
    rect = torch.tensor([float(dS[l:, :l].sum()) for l in range(L)], dtype=F64)
    _close(dlf, rect, 1e-12, "P10 rectangle identity")


# --------------------------------------------------------------------------- P11
def pin_p11_decode_is_last_row(ora, B=2, H=2, T=40, d=8, seed=11):
    q, k, v = (_rand((B, H, T, d), seed + i) for i in range(3))
    x = _rand((B, H, T), seed + 4) + 2
    s = 1.0 / math.sqrt(d)
    O, LSE = ora.forward(q, k, v, x, s)
    o, lse, cT = ora.decode(q[:, :, T - 1], k, v, x[..., : T - 1], x[..., T - 1], s)
    _close(o, O[:, :, T - 1], 1e-12, "P11 decode o")
    _close(lse, LSE[:, :, T - 1], 1e-12, "P11 decode lse")
    _close(cT, ora.log_sigmoid(x).sum(-1), 1e-12, "P11 c_T")


# --------------------------------------------------------------------------- P12
def pin_p12_zero_query_closed_forms(ora, L=50, d=4, seed=12):
    k, v = (_rand((1, 1, L, d), seed + i) for i in range(2))
    q = torch.zeros(1, 1, L, d, dtype=F64)
    i = torch.arange(1, L + 1, dtype=F64)
    _, LSE = ora.forward_from_logf(q, k, v, torch.zeros(1, 1, L, dtype=F64), 0.5)
    _close(LSE[0, 0], torch.log(i), 1e-13, "P12 LSE = log i")
    m = 0.3
    O, LSE = ora.forward_from_logf(q, k, v, torch.full((1, 1, L), -m, dtype=F64), 0.5)
    geo = torch.log((1 - torch.exp(-m * i)) / (1 - math.exp(-m)))
    _close(LSE[0, 0], geo, 1e-12, "P12 geometric LSE")
    w = torch.exp(-m * (i[:, None] - i[None, :])).tril()       # F_ij = e^{-m(i-j)}
    _close(O[0, 0], (w @ v[0, 0]) / w.sum(1, keepdim=True), 1e-12, "P12 O weights")


# --------------------------------------------------------------------------- P13
def pin_p13_two_tokens(ora):
    q = torch.tensor([[[[0.5, -1.0], [2.0, 0.25]]]], dtype=F64)
    k = torch.tensor([[[[1.0, 0.5], [-0.5, 1.5]]]], dtype=F64)
    v = torch.tensor([[[[3.0, -2.0], [1.0, 4.0]]]], dtype=F64)
    x = torch.tensor([[[0.7, -0.4]]], dtype=F64)
    s = 0.8
    O, LSE = ora.forward(q, k, v, x, s)
    lf2 = -math.log1p(math.exp(0.4))                   # log sigmoid(-0.4)
    a = s * (2.0 * 1.0 + 0.25 * 0.5) + lf2             # row 2, key 1: s q2.k1 + D_21
    b = s * (2.0 * -0.5 + 0.25 * 1.5)                  # row 2, key 2: D_22 = 0
    lse2 = math.log(math.exp(a) + math.exp(b))
    o2 = (math.exp(a) * v[0, 0, 0] + math.exp(b) * v[0, 0, 1]) / (math.exp(a) + math.exp(b))
    _close(LSE[0, 0, 0], s * (0.5 * 1.0 - 1.0 * 0.5), 1e-14, "P13 LSE_1")
    _close(LSE[0, 0, 1], lse2, 1e-14, "P13 LSE_2")
    _close(O[0, 0, 1], o2, 1e-14, "P13 o_2")


# --------------------------------------------------------------------------- P14
def _objective_logit(ora, q, k, v, x, dO, s):
    O, _ = ora.forward(q, k, v, x, s)
    return float((O * dO).sum())


def pin_p14_gate_logit_gradient(ora, B=1, H=2, L=7, d=3, seed=14):
    """d(logit) equals central finite differences of sum(O o dO) taken through
    the gate logits themselves (f = sigmoid(x), Sec. 3), and the gate factor
    d log f / dx is 1 - f (closed form of the sigmoid's derivative)."""
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    x = _rand((B, H, L), seed + 5) * 2 + 1
    s = 0.6
    _, _, _, dx = ora.backward_logit(q, k, v, x, dO, s)
    eps = 1e-6
    flat = x.view(-1)
    for idx in range(flat.numel()):
        old = float(flat[idx])
        flat[idx] = old + eps
        fp = _objective_logit(ora, q, k, v, x, dO, s)
        flat[idx] = old - eps
        fm = _objective_logit(ora, q, k, v, x, dO, s)
        flat[idx] = old
        fd = (fp - fm) / (2 * eps)
        got = float(dx.reshape(-1)[idx])
        assert abs(fd - got) <= 1e-7 * max(1.0, abs(fd)), \
            f"P14 dlogit[{idx}]: finite difference {fd:.9f} vs oracle {got:.9f}"
    # the first gate never enters O: its logit gradient is zero
    assert float(dx[..., 0].abs().max()) <= 1e-12
    # gate factor: 1 - f with f = exp(log sigmoid(x)); 1/2 at x = 0
    xs = torch.tensor([-30.0, -3.0, -0.5, 0.0, 0.5, 3.0, 30.0], dtype=torch.float64)
    factor = ora.gate_backward(xs, torch.ones_like(xs))
    _close(factor, 1.0 - torch.exp(ora.log_sigmoid(xs)), 1e-15, "P14 gate factor 1 - f")
    assert abs(float(factor[3]) - 0.5) <= 1e-15


# --------------------------------------------------------------------------- P15
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read_golden(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].split()
        if line:
            vals[line[0]] = [float(x) for x in line[1:]]
    return vals


def pin_p15_fixed_gate_init_worked_example(ora):
    """The appendix's worked example: H = 4, (T_min, T_max) = (2, 128) gives time
    constants (2, 8, 32, 128); and sigmoid(b)^T(b) = 1/e by definition of T."""
    g = _read_golden("fixed_gate_init.txt")
    b = ora.fixed_gate_bias_init(int(g["H"][0]), g["T_min"][0], g["T_max"][0])
    _close(ora.time_constant(b), torch.tensor(g["T"], dtype=F64), 1e-11, "P15 T(b_init)")
    _close(torch.sigmoid(b) ** ora.time_constant(b), torch.full_like(b, math.exp(-1.0)), 1e-14,
           "P15 sigmoid(b)^T(b) = 1/e")
    assert torch.all(b[1:] > b[:-1]), "P15 longer time constants need larger biases"


def pin_p15_fixed_gate_is_alibi_with_init_slopes(ora, B=1, H=4, L=26, d=8, seed=15):
    """A fixed gate initialised with (T_min, T_max) is ALiBi with slopes 1/T_h,
    ranging from 1/T_max to 1/T_min (Sec. 3 and the appendix)."""
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    s = 1.0 / math.sqrt(d)
    b = ora.fixed_gate_bias_init(H, 2.0, 128.0)
    slopes = torch.tensor([1 / 2, 1 / 8, 1 / 32, 1 / 128], dtype=F64)
    i = torch.arange(L, dtype=F64)
    dist = i[:, None] - i[None, :]
    mask = -slopes[:, None, None] * dist[None]
    mask = mask.masked_fill(dist[None] < 0, -math.inf)[None].expand(B, H, L, L)
    O, _ = ora.forward_fixed_gate(q, k, v, b, s)
    Oref, _, _, _ = _sdpa_with_grads(q, k, v, dO, s, mask)
    _close(O, Oref, 1e-11, "P15 fixed gate = ALiBi(1/T_h)")


def _objective_bias(ora, q, k, v, b, dO, s):
    O, _ = ora.forward_fixed_gate(q, k, v, b, s)
    return float((O * dO).sum())


def pin_p15_fixed_gate_bias_gradient(ora, B=2, H=3, L=9, d=3, seed=25):
    """d b^(h) equals central finite differences of sum(O o dO) in b^(h)."""
    q, k, v, dO = (_rand((B, H, L, d), seed + i) for i in range(4))
    b = _rand((H,), seed + 5) + 1.0
    s = 0.5
    _, _, _, db = ora.backward_fixed_gate(q, k, v, b, dO, s)
    eps = 1e-6
    for h in range(H):
        old = float(b[h])
        b[h] = old + eps
        fp = _objective_bias(ora, q, k, v, b, dO, s)
        b[h] = old - eps
        fm = _objective_bias(ora, q, k, v, b, dO, s)
        b[h] = old
        fd = (fp - fm) / (2 * eps)
        assert abs(fd - float(db[h])) <= 1e-7 * max(1.0, abs(fd)), \
            f"P15 db[{h}]: finite difference {fd:.9f} vs oracle {float(db[h]):.9f}"


# --------------------------------------------------------------------------- P16
def pin_p16_rms_norm(ora, H=3, L=11, d=7, seed=16):
    """Unit weight, eps = 0: every row has mean square 1 and is scale invariant;
    with eps the mean square is ms / (ms + eps); per-head weights scale per head."""
    x = _rand((2, H, L, d), seed)
    ones = torch.ones(H, d, dtype=F64)
    y, r = ora.rms_norm(x, ones, 0.0)
    _close((y * y).mean(-1), torch.ones(2, H, L, dtype=F64), 1e-12, "P16 unit mean square")
    lam = torch.rand(2, H, L, 1, generator=torch.Generator().manual_seed(seed), dtype=F64) * 5 + 0.1
    y2, _ = ora.rms_norm(x * lam, ones, 0.0)
    _close(y2, y, 1e-12, "P16 scale invariance")
    ms = (x * x).mean(-1)
    eps = 0.37
    y3, _ = ora.rms_norm(x, ones, eps)
    _close((y3 * y3).mean(-1), ms / (ms + eps), 1e-12, "P16 mean square with eps")
    w = _rand((H, d), seed + 1)
    y4, _ = ora.rms_norm(x, w, 0.0)
    for h in range(H):
        _close(y4[:, h], y[:, h] * w[h], 1e-12, f"P16 head {h} weight")


# --------------------------------------------------------------------------- P17
def pin_p17_token_shift_limits(ora, B=2, H=2, L=9, d=5, seed=17):
    """Shift logits at -inf, +inf and 0 give the identity, the one-step shift with
    a zero first row, and the average with the previous row (zero before t = 1)."""
    x = _rand((B, H, L, d), seed)
    big = torch.full((B, H, L), 1e4, dtype=F64)
    _close(ora.token_shift(x, -big), x, 0.0, "P17 identity")
    sh = ora.token_shift(x, big)
    _close(sh[..., 0, :], torch.zeros(B, H, d, dtype=F64), 0.0, "P17 first row")
    _close(sh[..., 1:, :], x[..., :-1, :], 0.0, "P17 shift")
    av = ora.token_shift(x, torch.zeros(B, H, L, dtype=F64))
    _close(av[..., 1:, :], 0.5 * (x[..., 1:, :] + x[..., :-1, :]), 1e-15, "P17 average")
    _close(av[..., 0, :], 0.5 * x[..., 0, :], 1e-15, "P17 average, first row")
    # the prologue with saturated shifts: plain QK-norm, and keys taken from t - 1
    qr, kr, vr = x, _rand((B, H, L, d), seed + 1), _rand((B, H, L, d), seed + 2)
    wq, wk = _rand((H, d), seed + 3), _rand((H, d), seed + 4)
    q, k, v = ora.pro_prologue(qr, kr, vr, -big, big, wq, wk, 1e-6)
    n = lambda t, w: t / torch.sqrt((t * t).mean(-1, keepdim=True) + 1e-6) * w[None, :, None, :]
    _close(q, n(qr, wq), 1e-12, "P17 prologue q")
    _close(k, n(kr, wk), 1e-12, "P17 prologue k without shift")
    _close(v[..., 1:, :], vr[..., :-1, :], 0.0, "P17 prologue v shifted")


# --------------------------------------------------------------------------- P18
def _fd_check(f, x, grad, eps, tol, what, n_probe=12, seed=0):
    """Central finite differences of the scalar f at n_probe entries of x."""
    g = torch.Generator().manual_seed(seed)
    flat = x.view(-1)
    idx = torch.randperm(flat.numel(), generator=g)[:n_probe]
    for i in idx.tolist():
        old = float(flat[i])
        flat[i] = old + eps
        fp = f()
        flat[i] = old - eps
        fm = f()
        flat[i] = old
        fd = (fp - fm) / (2 * eps)
        an = float(grad.reshape(-1)[i])
        assert abs(fd - an) <= tol * max(1.0, abs(fd)), f"{what}[{i}]: fd {fd:.9f} vs oracle {an:.9f}"


def pin_p18_pro_finite_differences(ora, B=1, H=2, L=5, d=3, seed=18):
    """Prologue and output-gate gradients against central finite differences."""
    t = [_rand((B, H, L, d), seed + i) for i in range(3)]
    ka, va = _rand((B, H, L), seed + 3), _rand((B, H, L), seed + 4)
    wq, wk = _rand((H, d), seed + 5), _rand((H, d), seed + 6)
    dq, dk, dv = (_rand((B, H, L, d), seed + 7 + i) for i in range(3))
    eps = 0.05
    grads = ora.pro_prologue_backward(t[0], t[1], t[2], ka, va, wq, wk, eps, dq, dk, dv)

    def obj():
        q, k, v = ora.pro_prologue(t[0], t[1], t[2], ka, va, wq, wk, eps)
        return float((q * dq).sum() + (k * dk).sum() + (v * dv).sum())
    for x, g, name in zip((t[0], t[1], t[2], ka, va, wq, wk), grads,
                          ("dq_raw", "dk_raw", "dv_raw", "dk_shift", "dv_shift", "dwq", "dwk")):
        _fd_check(obj, x, g, 1e-6, 1e-6, f"P18 {name}")
    o, gl = _rand((B, H, L, d), seed + 10), _rand((B, H, L, d), seed + 11)
    wo, dy = _rand((H, d), seed + 12), _rand((B, H, L, d), seed + 13)
    do, dg, dw = ora.output_gate_backward(o, gl, wo, eps, dy)
    obj2 = lambda: float((ora.output_gate(o, gl, wo, eps) * dy).sum())
    for x, g, name in ((o, do, "do"), (gl, dg, "dg"), (wo, dw, "dwo")):
        _fd_check(obj2, x, g, 1e-6, 1e-6, f"P18 {name}")


def _autograd_pro_layer(qr, kr, vr, ka, va, wq, wk, lf, gl, wo, eps, s):
    """The Pro layer written directly with differentiable torch ops."""
    def norm(x, w):
        return x * torch.rsqrt(x.pow(2).mean(-1, keepdim=True) + eps) * w[None, :, None, :]

    def shift(x, logit):
        a = torch.sigmoid(logit)[..., None]
        prev = Fnn.pad(x, (0, 0, 1, 0))[..., :-1, :]
        return a * prev + (1 - a) * x
    q, k, v = norm(qr, wq), norm(shift(kr, ka), wk), shift(vr, va)
    L = q.shape[-2]
    c = torch.cumsum(lf, -1)
    Dm = (c[..., :, None] - c[..., None, :]).masked_fill(
        torch.ones(L, L, dtype=torch.bool).triu(1), -math.inf)
    O = torch.softmax(s * q @ k.transpose(-1, -2) + Dm, -1) @ v
    return norm(O, wo) * torch.sigmoid(gl)


def pin_p18_pro_autograd(ora, B=2, H=2, L=13, d=6, seed=28):
    """torch autograd of an independently written Pro layer equals the oracle's
    prologue -> attention -> epilogue forward and hand-derived backward chain."""
    leaves = [_rand((B, H, L, d), seed), _rand((B, H, L, d), seed + 1), _rand((B, H, L, d), seed + 2),
              _rand((B, H, L), seed + 3), _rand((B, H, L), seed + 4), _rand((H, d), seed + 5),
              _rand((H, d), seed + 6), -torch.rand(B, H, L, generator=torch.Generator().manual_seed(seed),
                                                   dtype=F64), _rand((B, H, L, d), seed + 7),
              _rand((H, d), seed + 8)]
    eps, s = 1e-3, 0.4
    dy = _rand((B, H, L, d), seed + 9)
    lv = [x.clone().requires_grad_(True) for x in leaves]
    y = _autograd_pro_layer(*lv, eps, s)
    ag = torch.autograd.grad((y * dy).sum(), lv)
    qr, kr, vr, ka, va, wq, wk, lf, gl, wo = leaves
    q, k, v = ora.pro_prologue(qr, kr, vr, ka, va, wq, wk, eps)
    O, _ = ora.forward_from_logf(q, k, v, lf, s)
    _close(ora.output_gate(O, gl, wo, eps), y.detach(), 1e-12, "P18 Pro forward")
    dO, dg, dwo = ora.output_gate_backward(O, gl, wo, eps, dy)
    dq, dk, dv, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    pg = ora.pro_prologue_backward(qr, kr, vr, ka, va, wq, wk, eps, dq, dk, dv)
    mine = list(pg[:5]) + [pg[5], pg[6], dlf, dg, dwo]
    names = ("dq_raw", "dk_raw", "dv_raw", "dk_shift", "dv_shift", "dwq", "dwk", "dlogf", "dg", "dwo")
    for a, b, name in zip(ag, mine, names):
        _close(b, a, 1e-10, f"P18 autograd {name}")


# --------------------------------------------------------------------------- P19
def pin_p19_output_gate_limits(ora, B=1, H=3, L=6, d=5, seed=29):
    """Saturated gate: y = RMSNorm(o) and d g = 0; zero logit: y = RMSNorm(o) / 2."""
    o, dy = _rand((B, H, L, d), seed), _rand((B, H, L, d), seed + 1)
    wo = _rand((H, d), seed + 2)
    n, _ = ora.rms_norm(o, wo, 1e-6)
    big = torch.full((B, H, L, d), 1e4, dtype=F64)
    _close(ora.output_gate(o, big, wo, 1e-6), n, 1e-12, "P19 open gate")
    _close(ora.output_gate(o, 0 * big, wo, 1e-6), 0.5 * n, 1e-12, "P19 half gate")
    _, dg, _ = ora.output_gate_backward(o, big, wo, 1e-6, dy)
    _close(dg, torch.zeros_like(dg), 0.0, "P19 saturated gate gradient")
    do, _, _ = ora.output_gate_backward(o, -big, wo, 1e-6, dy)
    _close(do, torch.zeros_like(do), 0.0, "P19 closed gate passes no gradient to o")


def pin_p20_gate_projection(ora, B=2, L=3, M=5, H=2, seed=20):
    """The gate logits against explicit loops over the definition, and the
    special case w_f^(h) = unit vector m_h: logit^(h)_t = x_t[m_h] + b^(h)."""
    x, w, b = _rand((B, L, M), seed), _rand((H, M), seed + 1), _rand((H,), seed + 2)
    got = ora.gate_projection(x, w, b)
    assert tuple(got.shape) == (B, H, L)
    for bb in range(B):
        for h in range(H):
            for t in range(L):
                ref = sum(float(x[bb, t, m]) * float(w[h, m]) for m in range(M)) + float(b[h])
                assert abs(float(got[bb, h, t]) - ref) <= 1e-12 * max(1.0, abs(ref)), (bb, h, t)
    e = torch.zeros((H, M), dtype=torch.float64)
    picks = [3, 1]
    for h, m in enumerate(picks):
        e[h, m] = 1.0
    got = ora.gate_projection(x, e, b)
    for h, m in enumerate(picks):
        _close(got[:, h, :], x[:, :, m] + b[h], 1e-15, "unit-vector projection")
    _close(ora.gate_projection(x, w), ora.gate_projection(x, w, b) - b[None, :, None], 1e-14,
           "bias-free projection")


def pin_p21_gate_projection_backward(ora, B=2, L=4, M=6, H=3, seed=21):
    """dx, dw_f, db_f against explicit loops and against central finite
    differences of sum(logit * d_logit)."""
    x, w, b = _rand((B, L, M), seed), _rand((H, M), seed + 1), _rand((H,), seed + 2)
    g = _rand((B, H, L), seed + 3)
    dx, dw, db = ora.gate_projection_backward(x, w, g)
    for bb in range(B):
        for t in range(L):
            for m in range(M):
                ref = sum(float(g[bb, h, t]) * float(w[h, m]) for h in range(H))
                assert abs(float(dx[bb, t, m]) - ref) <= 1e-12, ("dx", bb, t, m)
    for h in range(H):
        for m in range(M):
            ref = sum(float(g[bb, h, t]) * float(x[bb, t, m]) for bb in range(B) for t in range(L))
            assert abs(float(dw[h, m]) - ref) <= 1e-12, ("dw", h, m)
        ref = sum(float(g[bb, h, t]) for bb in range(B) for t in range(L))
        assert abs(float(db[h]) - ref) <= 1e-12, ("db", h)
    f = lambda: float((ora.gate_projection(x, w, b) * g).sum())
    _fd_check(f, x, dx, 1e-4, 1e-7, "dx")
    _fd_check(f, w, dw, 1e-4, 1e-7, "dw")
    _fd_check(f, b, db, 1e-4, 1e-7, "db")


# --------------------------------------------------------------------------- P22
def pin_p22_delta_from_stored_o(ora):
    """Alg. 2 reads O back from HBM for Delta = rowsum(dO o O).  With O stored in
    bf16, L = 2 written out by hand: q = 0 and log f = 0 give A_21 = A_22 = 1/2;
    v = (1, 2^-8) makes o_2 = 1/2 + 2^-9, a tie that bf16 (round to nearest even)
    sends to 1/2; dO = (1, g) with g = 1 + 2^-9 (not a bf16 value, so a rounded
    dO would show).  Then Delta_2 = g/2, dS_21 = g/4, dS_22 = g (2^-9 - 1/4),
    dS_1 = 0, dQ_2 = s g (k_1/4 + k_2 (2^-9 - 1/4)), dc = (-g/4, g/4) and
    d(log f) = (0, g/4); dV = A^T dO = (1 + g/2, g/2).  With the exact O every
    2^-9 term changes (Delta_2 = g (1/2 + 2^-9))."""
    g = 1.0 + 2.0 ** -9
    q = torch.zeros(1, 1, 2, 1, dtype=F64)
    k = torch.tensor([[[[1.0], [3.0]]]], dtype=F64)
    v = torch.tensor([[[[1.0], [2.0 ** -8]]]], dtype=F64)
    dO = torch.tensor([[[[1.0], [g]]]], dtype=F64)
    lf = torch.zeros(1, 1, 2, dtype=F64)
    s = 0.75
    dQ, dK, dV, dlf = ora.backward_from_logf(q, k, v, lf, dO, s, o_dtype=torch.bfloat16)
    _close(dQ[0, 0, 1, 0], s * g * (1.0 / 4 + 3.0 * (2.0 ** -9 - 1.0 / 4)), 1e-15, "P22 dQ_2")
    _close(dQ[0, 0, 0, 0], 0.0, 1e-15, "P22 dQ_1")
    _close(dK[0, 0], torch.zeros(2, 1, dtype=F64), 1e-15, "P22 dK (q = 0)")
    _close(dV[0, 0, :, 0], torch.tensor([1.0 + g / 2, g / 2], dtype=F64), 1e-15, "P22 dV")
    _close(dlf[0, 0], torch.tensor([0.0, g / 4], dtype=F64), 1e-15, "P22 d(log f)")
    # the exact O: Delta_2 = g (1/2 + 2^-9), dS_21 = g (1/4 - 2^-10), dS_22 = g (2^-10 - 1/4)
    dQ, _, _, dlf = ora.backward_from_logf(q, k, v, lf, dO, s)
    _close(dQ[0, 0, 1, 0], s * g * ((1.0 / 4 - 2.0 ** -10) + 3.0 * (2.0 ** -10 - 1.0 / 4)), 1e-15,
           "P22 dQ_2 (exact O)")
    _close(dlf[0, 0], torch.tensor([0.0, g * (1.0 / 4 - 2.0 ** -10)], dtype=F64), 1e-15,
           "P22 d(log f) (exact O)")


ALL_PINS = [
    pin_p22_delta_from_stored_o,
    pin_p1_zero_forgetting_is_softmax_attention,
    pin_p2_full_forgetting,
    pin_p3_constant_gate_is_alibi,
    pin_p4_decay_matrix,
    pin_p5_attention_rows,
    pin_p6_first_row,
    pin_p7_invariances,
    pin_p8_product_form,
    pin_p9_finite_differences,
    pin_p9_autograd,
    pin_p10_rectangle_identity,
    pin_p11_decode_is_last_row,
    pin_p12_zero_query_closed_forms,
    pin_p13_two_tokens,
    pin_p14_gate_logit_gradient,
    pin_p15_fixed_gate_init_worked_example,
    pin_p15_fixed_gate_is_alibi_with_init_slopes,
    pin_p15_fixed_gate_bias_gradient,
    pin_p16_rms_norm,
    pin_p17_token_shift_limits,
    pin_p18_pro_finite_differences,
    pin_p18_pro_autograd,
    pin_p19_output_gate_limits,
    pin_p20_gate_projection,
    pin_p21_gate_projection_backward,
]

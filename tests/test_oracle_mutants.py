"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that
the pins catch every one of them."""
import importlib.util
import math
import os

import pytest
import torch

import oracle_pins

ORACLE_FILE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "oracle", "fox_oracle.py")


def _fresh_oracle(tag):
    spec = importlib.util.spec_from_file_location(f"fox_oracle_mutant_{tag}", ORACLE_FILE)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _m_scale_on_D(m):
    """The 1/sqrt(d)-like factor applied to D as well as to q.k."""
    orig = m.decay_matrix
    m.decay_matrix = lambda c, rows=None: orig(m._f64(c) * 0.5, rows)


def _m_exclusive_c(m):
    m.prefix_c = lambda lf: torch.cumsum(m._f64(lf), -1) - m._f64(lf)


def _m_no_mask(m):
    def dm(c, rows=None):
        c = m._f64(c)
        L = c.shape[-1]
        r = torch.arange(L) if rows is None else torch.as_tensor(rows)
        return c[r][:, None] - c[None, :]
    m.decay_matrix = dm


def _m_flipped_D(m):
    orig = m.decay_matrix
    m.decay_matrix = lambda c, rows=None: orig(-m._f64(c), rows)


def _m_logsigmoid_max(m):
    m.log_sigmoid = lambda x: torch.maximum(m._f64(x), torch.zeros_like(m._f64(x))) - \
        torch.log1p(torch.exp(-m._f64(x).abs()))


def _patch_backward(m, variant):
    def bwd(q, k, v, c, dO, scale, return_dS=False, o_dtype=None):
        q, k, v, c, dO = (m._f64(t) for t in (q, k, v, c, dO))
        O, _, A = m.forward_head_from_c(q, k, v, c, scale, return_A=True)
        dV = A @ dO if variant == "dV_untransposed" else A.T @ dO
        dA = dO @ v.T
        if o_dtype is not None:
            if variant == "delta_rounds_dO":
                dO = dO.to(o_dtype).to(torch.float64)
            else:
                O = O.to(o_dtype).to(torch.float64)
        delta = (dO * O).sum(1, keepdim=True)
        if variant == "delta_from_dA":
            delta = dA.sum(1, keepdim=True)
        dS = A * (dA - delta)
        dQ = scale * (dS @ k)
        dK = scale * (dS @ q) if variant == "dK_untransposed" else scale * (dS.T @ q)
        if variant == "dK_no_scale":
            dK = dS.T @ q
        dc = dS.sum(1) - dS.sum(0)
        if variant == "dc_sign":
            dc = -dc
        if return_dS:
            return dQ, dK, dV, dc, dS
        return dQ, dK, dV, dc
    m.backward_head_from_c = bwd


def _m_forward_cumsum(m):
    m.reverse_cumsum = lambda x: torch.cumsum(m._f64(x), -1)


def _m_lse_no_max(m):
    """LSE = log(l), forgetting to add back the row max m."""
    def fwd(q, k, v, c, scale, rows=None, return_A=False):
        q, k, v, c = (m._f64(t) for t in (q, k, v, c))
        r = torch.arange(q.shape[0]) if rows is None else torch.as_tensor(rows)
        S = scale * (q[r] @ k.T) + m.decay_matrix(c, r)
        mx = S.max(1, keepdim=True).values
        E = torch.exp(S - mx)
        l = E.sum(1, keepdim=True)
        A = E / l
        LSE = torch.log(l).squeeze(1)
        return (A @ v, LSE, A) if return_A else (A @ v, LSE)
    m.forward_head_from_c = fwd


def _m_decode_sign(m):
    def dec(q, k_cache, v_cache, cached_logit, logit_new, scale, heads=None):
        B, H, d = q.shape
        T = k_cache.shape[2]
        lf = torch.cat([m.log_sigmoid(cached_logit), m.log_sigmoid(logit_new)[..., None]], -1)
        c = m.prefix_c(lf)
        o = torch.zeros(B, H, d, dtype=torch.float64)
        lse = torch.zeros(B, H, dtype=torch.float64)
        for b in range(B):
            for h in range(H):
                s = scale * (m._f64(k_cache[b, h]) @ m._f64(q[b, h])) - (c[b, h, T - 1] - c[b, h])
                e = torch.exp(s - s.max())
                o[b, h] = (e @ m._f64(v_cache[b, h])) / e.sum()
                lse[b, h] = s.max() + torch.log(e.sum())
        return o, lse, c[..., T - 1]
    m.decode = dec


def _m_scale_twice(m):
    orig = m.forward_head_from_c
    m.forward_head_from_c = lambda q, k, v, c, scale, rows=None, return_A=False: \
        orig(q, k, v, c, scale * scale, rows, return_A)


def _m_gate_factor_sign(m):
    """sigmoid(x) instead of sigmoid(-x) as the gate's derivative factor."""
    m.gate_backward = lambda logit, dlf: m._f64(dlf) * torch.sigmoid(m._f64(logit))


def _m_init_linear_spacing(m):
    """Time constants spaced linearly instead of logarithmically."""
    def init(H, t_min, t_max):
        T = torch.linspace(t_min, t_max, H, dtype=torch.float64)
        return -1.0 / T - torch.log(-torch.expm1(-1.0 / T))
    m.fixed_gate_bias_init = init


def _m_fixed_db_no_gate_factor(m):
    """d b summed without the sigmoid(-b) factor."""
    def bwd(q, k, v, bias, dO, scale):
        B, H, L, _ = q.shape
        dQ, dK, dV, dlf = m.backward_from_logf(q, k, v, m.fixed_gate_log_f(bias, B, L), dO, scale)
        return dQ, dK, dV, dlf.sum(dim=(0, 2))
    m.backward_fixed_gate = bwd


def _m_rms_sum_not_mean(m):
    """RMSNorm divides by the root of the sum of squares instead of the mean."""
    def rn(x, weight, eps):
        x = m._f64(x)
        r = 1.0 / torch.sqrt((x * x).sum(dim=-1) + eps)
        return x * r[..., None] * m._head_weight(weight, x.dim()), r
    m.rms_norm = rn


def _m_rms_bwd_no_projection(m):
    """RMSNorm backward without the component along n."""
    def rb(x, weight, eps, dy):
        x, dy = m._f64(x), m._f64(dy)
        _, r = m.rms_norm(x, weight, eps)
        n = x * r[..., None]
        dx = r[..., None] * dy * m._head_weight(weight, x.dim())
        dw = (dy * n).sum(dim=-2)
        return dx, (dw.sum(dim=0) if dw.dim() == 3 else dw)
    m.rms_norm_backward = rb


def _m_shift_from_next(m):
    """The token shift mixes with the next token instead of the previous one."""
    def ts(x, logit):
        x = m._f64(x)
        a = torch.sigmoid(m._f64(logit))[..., None]
        nxt = torch.zeros_like(x)
        nxt[..., :-1, :] = x[..., 1:, :]
        return a * nxt + (1.0 - a) * x
    m.token_shift = ts


def _m_shift_bwd_no_next_term(m):
    """Token-shift backward forgetting that x_t also feeds output t + 1."""
    orig = m.token_shift_backward
    def tb(x, logit, dy):
        dx, dl = orig(x, logit, dy)
        a = torch.sigmoid(m._f64(logit))
        return (1.0 - a)[..., None] * m._f64(dy), dl
    m.token_shift_backward = tb


def _m_shift_logit_sign(m):
    orig = m.token_shift_backward
    def tb(x, logit, dy):
        dx, dl = orig(x, logit, dy)
        return dx, -dl
    m.token_shift_backward = tb


def _m_gate_bwd_no_derivative(m):
    """Output-gate backward using sigmoid(g) in place of its derivative."""
    def ob(o, g, w, eps, dy):
        dy = m._f64(dy)
        sg = torch.sigmoid(m._f64(g))
        u, _ = m.rms_norm(o, w, eps)
        do, dw = m.rms_norm_backward(o, w, eps, dy * sg)
        return do, dy * u * sg, dw
    m.output_gate_backward = ob


def _m_head_weight_first_row(m):
    """Every head normalised with head 0's weight row."""
    def hw(weight, ndim):
        w = m._f64(weight)
        w = w[:1].expand_as(w)
        return w.reshape((1,) * (ndim - 3) + (w.shape[0], 1, w.shape[1]))
    m._head_weight = hw


def _m_projection_heads_swapped(m):
    """The gate projection pairing head h with weight row H-1-h."""
    orig = m.gate_projection
    def gp(x, w_f, b_f=None):
        return orig(x, m._f64(w_f).flip(0), b_f)
    m.gate_projection = gp


def _m_projection_dx_one_head(m):
    """dx taking only the first head's contribution."""
    orig = m.gate_projection_backward
    def gb(x, w_f, d_logit):
        dx, dw, db = orig(x, w_f, d_logit)
        g, w = m._f64(d_logit), m._f64(w_f)
        return g[:, 0, :, None] * w[0][None, None, :], dw, db
    m.gate_projection_backward = gb


def _m_projection_no_bias(m):
    """The gate projection dropping the bias."""
    orig = m.gate_projection
    m.gate_projection = lambda x, w_f, b_f=None: orig(x, w_f, None)


def _m_projection_dw_mean(m):
    """dw_f averaged over tokens instead of summed."""
    orig = m.gate_projection_backward
    def gb(x, w_f, d_logit):
        dx, dw, db = orig(x, w_f, d_logit)
        n = m._f64(x).shape[0] * m._f64(x).shape[1]
        return dx, dw / n, db
    m.gate_projection_backward = gb


MUTANTS = {
    "decay_scaled": _m_scale_on_D,
    "exclusive_prefix": _m_exclusive_c,
    "no_causal_mask": _m_no_mask,
    "decay_sign": _m_flipped_D,
    "logsigmoid_max": _m_logsigmoid_max,
    "dV_untransposed": lambda m: _patch_backward(m, "dV_untransposed"),
    "dK_untransposed": lambda m: _patch_backward(m, "dK_untransposed"),
    "dK_no_scale": lambda m: _patch_backward(m, "dK_no_scale"),
    "delta_from_dA": lambda m: _patch_backward(m, "delta_from_dA"),
    "dc_sign": lambda m: _patch_backward(m, "dc_sign"),
    "delta_rounds_dO": lambda m: _patch_backward(m, "delta_rounds_dO"),
    "forward_cumsum_for_dlogf": _m_forward_cumsum,
    "lse_without_max": _m_lse_no_max,
    "decode_bias_sign": _m_decode_sign,
    "scale_squared": _m_scale_twice,
    "gate_factor_sign": _m_gate_factor_sign,
    "init_linear_spacing": _m_init_linear_spacing,
    "fixed_db_no_gate_factor": _m_fixed_db_no_gate_factor,
    "rms_sum_not_mean": _m_rms_sum_not_mean,
    "rms_bwd_no_projection": _m_rms_bwd_no_projection,
    "shift_from_next": _m_shift_from_next,
    "shift_bwd_no_next_term": _m_shift_bwd_no_next_term,
    "shift_logit_sign": _m_shift_logit_sign,
    "gate_bwd_no_derivative": _m_gate_bwd_no_derivative,
    "head_weight_first_row": _m_head_weight_first_row,
    "projection_heads_swapped": _m_projection_heads_swapped,
    "projection_dx_one_head": _m_projection_dx_one_head,
    "projection_no_bias": _m_projection_no_bias,
    "projection_dw_mean": _m_projection_dw_mean,
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    m = _fresh_oracle(name)
    MUTANTS[name](m)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(m)
        except (AssertionError, RuntimeError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passes every pin"

"""Forgetting Attention -- plain fp64 CPU oracle.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP library.

Everything is computed in float64 on the host with torch CPU ops, fully
materialising the L x L decay matrix D, the logit matrix S and the attention
matrix A for each (batch, head) slice, exactly as the method is defined in the
paper (Forgetting Transformer, arXiv 2503.02130):

  * forget gate                f_t = sigmoid(logit_t), one scalar per head and
                               time step                      (Sec. 3, gate def.)
  * prefix vector              c_i = sum_{l<=i} log f_l       (Sec. 3, "Hardware-
                                                               aware implementation")
  * decay matrix               D_ij = sum_{l=j+1}^{i} log f_l = c_i - c_j for
                               j <= i, -inf above the diagonal (Eq. fot-weight,
                                                               Eq. fot-matrix, log 0 = -inf)
  * output                     O = softmax(s * Q K^T + D) V, the 1/sqrt(d)
                               scale s multiplying q.k only   (Eq. fot-matrix and
                                                               the footnote of Eq. attn-softmax)
  * logsumexp                  LSE_i = m_i + log l_i, natural log (Alg. 1, epilogue)
  * backward                   dV = A^T dO, dA = dO V^T, Delta_i = rowsum(dO o O),
                               dS = A o (dA - Delta), dQ = s dS K, dK = s dS^T Q,
                               dc = rowsum(dS) - colsum(dS)    (Alg. 2)
  * d(log f)                   chain rule through c = cumsum(log f):
                               d(log f)_l = sum_{i >= l} dc_i  (reverse cumsum)
  * d(logit)                   through f = sigmoid(logit): d(logit) =
                               d(log f) * sigmoid(-logit)      (Sec. 3, gate def.)
  * gate projection            logit_t^(h) = w_f^(h) . x_t + b_f^(h) for the layer
                               input x_t, one weight vector and bias per head
                                                              (Sec. 3, gate def.)
  * fixed gates                f_t^(h) = sigmoid(b^(h)) for all t (ALiBi with slope
                               -log sigmoid(b^(h)), Sec. 3); b^(h) initialised so that
                               T(b) = -1/log sigmoid(b) is log-spaced in [T_min, T_max]
                                                              (appendix, gate init.)
  * decode                     the forward's last row for a sequence whose last
                               key/value is the new token, c_T = c_{T-1} +
                               log sigmoid(x_new), c_0 = 0    (Eq. fot-weight at i = T)
  * FoX (Pro) prologue         q = RMSNorm(q~), k = RMSNorm(a k~_{t-1} + (1-a) k~_t),
                               v = b v~_{t-1} + (1-b) v~_t with a, b sigmoids of
                               the shift logits      (Eq. shift-linear; appendix,
                                                      FoX (Pro) layer computation)
  * FoX (Pro) epilogue         y = RMSNorm(o) o sigmoid(g)   (same appendix)

Readings of the paper this oracle takes (where it is silent or garbled):
  * the scale multiplies q.k only; D is unscaled; dQ, dK carry s, dc does not;
  * c is the inclusive prefix sum; O does not depend on log f_1;
  * Alg. 1's rescale of O by diag(exp(m_old - m_new))^{-1} is read as a
    multiplication by exp(m_old - m_new) (the FlashAttention-2 rescale); the
    oracle needs no online softmax, so it simply uses the plain softmax;
  * Alg. 2's rowsum(dO o O) "in R^d" is one value per row (R^N);
  * Delta uses the exact O by default; with o_dtype, the O that Alg. 2 reads
    back from HBM, i.e. O rounded to the dtype it was stored in;
  * decode: the query at position T attends to keys 1..T including itself.
  * Pro layer: RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w with per-head
    weights and eps an argument; the token shift of t = 1 mixes with zero.

All functions accept any-dtype torch tensors (or numpy arrays) and return fp64
torch tensors.  Every pin of this module lives in tests/test_oracle_*.py.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import torch

F64 = torch.float64


def _f64(x) -> torch.Tensor:
    if not isinstance(x, torch.Tensor):
        x = torch.as_tensor(x)
    return x.detach().to(device="cpu", dtype=F64)


# ---------------------------------------------------------------------------
# Gate prelude (Sec. 3: f_t = sigmoid(w_f^T x_t + b_f); c_i = sum_{l<=i} log f_l)
# ---------------------------------------------------------------------------
def log_sigmoid(x) -> torch.Tensor:
    """log sigmoid(x) = -log(1 + exp(-x)), written in the overflow-free form
    min(x, 0) - log1p(exp(-|x|)).  The forget gate value is f = sigmoid(x)."""
    x = _f64(x)
    return torch.minimum(x, torch.zeros_like(x)) - torch.log1p(torch.exp(-x.abs()))


def prefix_c(log_f) -> torch.Tensor:
    """Inclusive prefix sum over the last (time) axis: c_i = sum_{l<=i} log f_l."""
    return torch.cumsum(_f64(log_f), dim=-1)


def gate_prefix(logit):
    """Returns (log f, c) for gate logits of shape [..., L]."""
    lf = log_sigmoid(logit)
    return lf, prefix_c(lf)


# ---------------------------------------------------------------------------
# One (batch, head) slice, materialised
# ---------------------------------------------------------------------------
def decay_matrix(c: torch.Tensor, rows: Optional[torch.Tensor] = None) -> torch.Tensor:
    """D_ij = c_i - c_j for j <= i, -inf for j > i (Eq. fot-weight / fot-matrix).

    `rows` selects query rows (0-based); by default all L rows."""
    c = _f64(c)
    L = c.shape[-1]
    r = torch.arange(L) if rows is None else torch.as_tensor(rows, dtype=torch.long)
    D = c[r][:, None] - c[None, :]
    above = torch.arange(L)[None, :] > r[:, None]
    return D.masked_fill(above, -math.inf)


def forward_head_from_c(q, k, v, c, scale: float, rows=None, return_A: bool = False):
    """O, LSE for one head given c.  q, k, v: [L, d]; c: [L].

    S = s * Q K^T + D;  A = softmax_row(S);  O = A V;  LSE = m + log sum exp(S - m).
    Rows are independent, so `rows` evaluates only the selected query rows."""
    q, k, v, c = _f64(q), _f64(k), _f64(v), _f64(c)
    r = torch.arange(q.shape[0]) if rows is None else torch.as_tensor(rows, dtype=torch.long)
    S = scale * (q[r] @ k.T) + decay_matrix(c, r)
    m = S.max(dim=1, keepdim=True).values
    E = torch.exp(S - m)
    l = E.sum(dim=1, keepdim=True)
    A = E / l
    O = A @ v
    LSE = (m + torch.log(l)).squeeze(1)
    if return_A:
        return O, LSE, A
    return O, LSE


def backward_head_from_c(q, k, v, c, dO, scale: float, return_dS: bool = False,
                         o_dtype=None):
    """Gradients of sum(O * dO) for one head, by Alg. 2's formulas on full matrices.

    Returns dQ, dK, dV [L, d] and dc [L] (= dc^q + dc^k, Alg. 2's last steps).
    Alg. 2 reads O back from HBM for Delta; o_dtype (e.g. torch.bfloat16) is the
    dtype O was stored in there, and Delta then uses O rounded to it (round to
    nearest even); None uses the exact O."""
    q, k, v, c, dO = _f64(q), _f64(k), _f64(v), _f64(c), _f64(dO)
    O, _, A = forward_head_from_c(q, k, v, c, scale, return_A=True)
    dV = A.T @ dO
    dA = dO @ v.T
    O_read = O if o_dtype is None else O.to(o_dtype).to(F64)
    delta = (dO * O_read).sum(dim=1, keepdim=True)     # rowsum(dO o O), one per row
    dS = A * (dA - delta)                               # masked entries: A = 0 there
    dQ = scale * (dS @ k)
    dK = scale * (dS.T @ q)
    dc_q = dS.sum(dim=1)                                # += rowsum(dS)
    dc_k = -dS.sum(dim=0)                               # -= colsum(dS)
    dc = dc_q + dc_k
    if return_dS:
        return dQ, dK, dV, dc, dS
    return dQ, dK, dV, dc


def reverse_cumsum(x) -> torch.Tensor:
    """y_l = sum_{i >= l} x_i over the last axis (chain rule through a cumsum)."""
    x = _f64(x)
    return torch.flip(torch.cumsum(torch.flip(x, dims=[-1]), dim=-1), dims=[-1])


# ---------------------------------------------------------------------------
# Batched entry points: q, k, v, dO [B, H, L, d]; logit / log f [B, H, L]
# ---------------------------------------------------------------------------
def _heads(B: int, H: int, heads: Optional[Sequence] = None):
    if heads is None:
        return [(b, h) for b in range(B) for h in range(H)]
    return list(heads)


def forward_from_logf(q, k, v, log_f, scale: float, heads=None, rows=None):
    """Forward with log f given directly.  Returns O [B,H,L',d], LSE [B,H,L'] in
    fp64, with L' = len(rows) when rows are selected; heads not in `heads` are NaN."""
    B, H, L, d = q.shape
    c = prefix_c(log_f)
    nr = L if rows is None else len(rows)
    O = torch.full((B, H, nr, d), math.nan, dtype=F64)
    LSE = torch.full((B, H, nr), math.nan, dtype=F64)
    for b, h in _heads(B, H, heads):
        O[b, h], LSE[b, h] = forward_head_from_c(q[b, h], k[b, h], v[b, h], c[b, h], scale, rows)
    return O, LSE


def forward(q, k, v, logit, scale: float, heads=None, rows=None):
    """O, LSE for gate logits (the operator's real input)."""
    return forward_from_logf(q, k, v, log_sigmoid(logit), scale, heads, rows)


def backward_from_logf(q, k, v, log_f, dO, scale: float, heads=None, o_dtype=None):
    """dQ, dK, dV [B,H,L,d] and d(log f) [B,H,L], fp64 (NaN outside `heads`);
    o_dtype as for backward_head_from_c."""
    B, H, L, d = q.shape
    c = prefix_c(log_f)
    dQ = torch.full((B, H, L, d), math.nan, dtype=F64)
    dK = dQ.clone()
    dV = dQ.clone()
    dlogf = torch.full((B, H, L), math.nan, dtype=F64)
    kw = {} if o_dtype is None else {"o_dtype": o_dtype}
    for b, h in _heads(B, H, heads):
        gq, gk, gv, dc = backward_head_from_c(q[b, h], k[b, h], v[b, h], c[b, h], dO[b, h], scale,
                                              **kw)
        dQ[b, h], dK[b, h], dV[b, h] = gq, gk, gv
        dlogf[b, h] = reverse_cumsum(dc)
    return dQ, dK, dV, dlogf


def backward(q, k, v, logit, dO, scale: float, heads=None, o_dtype=None):
    return backward_from_logf(q, k, v, log_sigmoid(logit), dO, scale, heads, o_dtype)


def gate_backward(logit, d_log_f) -> torch.Tensor:
    """d(logit) from d(log f) through the forget gate f = sigmoid(logit) (Sec. 3):
    d log sigmoid(x) / dx = 1 - sigmoid(x) = sigmoid(-x), elementwise."""
    return _f64(d_log_f) * torch.sigmoid(-_f64(logit))


def backward_logit(q, k, v, logit, dO, scale: float, heads=None):
    """dQ, dK, dV and the gradient with respect to the gate logits."""
    dQ, dK, dV, dlf = backward(q, k, v, logit, dO, scale, heads)
    return dQ, dK, dV, gate_backward(logit, dlf)


# ---------------------------------------------------------------------------
# Gate projection (Sec. 3, gate definition): the logits are an affine function
# of the layer input, one weight vector and one bias per head.
# ---------------------------------------------------------------------------
def gate_projection(x, w_f, b_f=None) -> torch.Tensor:
    """logit[b, h, t] = sum_m x[b, t, m] w_f[h, m] + b_f[h] for x [B, L, M],
    w_f [H, M], b_f [H] (None: no bias); [B, H, L]."""
    x64, w64 = _f64(x), _f64(w_f)
    logit = torch.matmul(x64, w64.T).transpose(1, 2)
    if b_f is not None:
        logit = logit + _f64(b_f)[None, :, None]
    return logit.contiguous()


def gate_projection_backward(x, w_f, d_logit):
    """Gradients of sum(logit * d_logit): dx [B, L, M] = sum_h d_logit[b, h, t]
    w_f[h]; dw_f [H, M] = sum_{b, t} d_logit[b, h, t] x[b, t]; db_f [H] =
    sum_{b, t} d_logit[b, h, t]."""
    x64, w64, g = _f64(x), _f64(w_f), _f64(d_logit)
    B, L, M = x64.shape
    H = w64.shape[0]
    dx = torch.matmul(g.transpose(1, 2), w64)
    dw = torch.matmul(g.permute(1, 0, 2).reshape(H, B * L), x64.reshape(B * L, M))
    db = g.sum(dim=(0, 2))
    return dx, dw, db


# ---------------------------------------------------------------------------
# Data-independent / fixed forget gates (Sec. 3 "Connection to ALiBi"; Sec. 5
# ablations; appendix "Data-independent forget gate initialization")
# ---------------------------------------------------------------------------
def time_constant(b) -> torch.Tensor:
    """T(b) = 1 / (-log sigmoid(b)): the steps a gate sigmoid(b) needs to decay by 1/e."""
    return -1.0 / log_sigmoid(b)


def fixed_gate_bias_init(H: int, t_min: float, t_max: float) -> torch.Tensor:
    """b^(h), h = 1..H, with T(b^(h)) log-spaced from T_min to T_max.  Inverting
    T: sigmoid(b) = exp(-1/T), so b = log(e^{-1/T} / (1 - e^{-1/T})).  For H = 1
    the spacing is undefined; the single head takes T_min."""
    h = torch.arange(H, dtype=F64)
    frac = h / (H - 1) if H > 1 else torch.zeros(1, dtype=F64)
    T = torch.exp(math.log(t_min) + (math.log(t_max) - math.log(t_min)) * frac)
    return -1.0 / T - torch.log(-torch.expm1(-1.0 / T))


def fixed_gate_log_f(bias, B: int, L: int) -> torch.Tensor:
    """log f_t^(h) = log sigmoid(b^(h)) for every batch row and time step: [B,H,L]."""
    lf = log_sigmoid(bias)
    return lf[None, :, None].expand(B, lf.shape[0], L).clone()


def forward_fixed_gate(q, k, v, bias, scale: float, heads=None, rows=None):
    B, H, L, _ = q.shape
    return forward_from_logf(q, k, v, fixed_gate_log_f(bias, B, L), scale, heads, rows)


def backward_fixed_gate(q, k, v, bias, dO, scale: float):
    """dQ, dK, dV and d b^(h) [H]: every log f_t^(h) is log sigmoid(b^(h)), so
    d b^(h) = sigmoid(-b^(h)) * sum over batch and time of d(log f)."""
    B, H, L, _ = q.shape
    dQ, dK, dV, dlf = backward_from_logf(q, k, v, fixed_gate_log_f(bias, B, L), dO, scale)
    db = torch.sigmoid(-_f64(bias)) * dlf.sum(dim=(0, 2))
    return dQ, dK, dV, db


def decode(q, k_cache, v_cache, cached_logit, logit_new, scale: float, heads=None):
    """One decode step (Eq. fot-weight at i = T).

    q [B,H,d]; k_cache, v_cache [B,H,T,d] whose slot T-1 holds the new token;
    cached_logit [B,H,T-1] are the gate logits of tokens 1..T-1 (c_1..c_{T-1});
    logit_new [B,H] is the new token's gate logit, so c_T = c_{T-1} +
    log sigmoid(logit_new), with c_0 = 0.  Returns o [B,H,d], lse [B,H], and
    c_T [B,H] (the value the step appends to the prefix cache)."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    lf = torch.cat([log_sigmoid(cached_logit), log_sigmoid(logit_new)[..., None]], dim=-1)
    assert lf.shape[-1] == T
    c = prefix_c(lf)
    o = torch.full((B, H, d), math.nan, dtype=F64)
    lse = torch.full((B, H), math.nan, dtype=F64)
    for b, h in _heads(B, H, heads):
        kc, vc = _f64(k_cache[b, h]), _f64(v_cache[b, h])   # one slice at a time
        s = scale * (kc @ _f64(q[b, h])) + (c[b, h, T - 1] - c[b, h])
        m = s.max()
        e = torch.exp(s - m)
        o[b, h] = (e @ vc) / e.sum()
        lse[b, h] = m + torch.log(e.sum())
    return o, lse, c[..., T - 1]


# ---------------------------------------------------------------------------
# FoX (Pro) prologue and epilogue (Sec. 3 "Architecture design", Eq. shift-linear;
# appendix "Detailed FoX (Pro) layer computation").  Per head h and time t, from
# the raw projections q~ = W_q x, k~ = W_k x, v~ = W_v x (already split into heads):
#   q_t = RMSNorm_q(q~_t)
#   k_t = RMSNorm_k(a_t k~_{t-1} + (1 - a_t) k~_t),   a_t = sigmoid(w_k^T x_t)
#   v_t = b_t v~_{t-1} + (1 - b_t) v~_t,              b_t = sigmoid(w_v^T x_t)
# then, after the attention, y_t = RMSNorm_o(o_t) o sigmoid(W_g x_t).  The
# output projection W_o and the sum over heads are plain matrix products and
# not part of this module.
# Readings: RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w with a per-head weight
# w^(h) in R^d (the paper gives no eps; it is an argument); the shift of the
# first token mixes with a zero vector (k~_0 = v~_0 = 0); the shift logits
# w_k^T x_t, w_v^T x_t and the gate logits W_g x_t are the inputs, and their
# gradients are returned.
# ---------------------------------------------------------------------------
def _head_weight(weight, ndim):
    """[H, d] per-head weights broadcast against [B, H, L, d] (or [H, L, d])."""
    w = _f64(weight)
    return w.reshape((1,) * (ndim - 3) + (w.shape[0], 1, w.shape[1]))


def rms_norm(x, weight, eps: float):
    """RMSNorm over the head dimension with per-head weights: x [.., H, L, d],
    weight [H, d].  Returns (y, r) with r = 1 / sqrt(mean(x^2) + eps) [.., H, L]."""
    x = _f64(x)
    r = 1.0 / torch.sqrt((x * x).mean(dim=-1) + eps)
    return x * r[..., None] * _head_weight(weight, x.dim()), r


def rms_norm_backward(x, weight, eps: float, dy):
    """Gradients of sum(RMSNorm(x) o dy): with n = x r and dn = dy o w,
    dx = r (dn - n mean(dn o n)) (the mean over the head dimension), and
    dw^(h) = sum over batch and time of dy o n."""
    x, dy = _f64(x), _f64(dy)
    _, r = rms_norm(x, weight, eps)
    n = x * r[..., None]
    dn = dy * _head_weight(weight, x.dim())
    dx = r[..., None] * (dn - n * (dn * n).mean(dim=-1, keepdim=True))
    dw = (dy * n).sum(dim=-2)                    # over time
    if dw.dim() == 3:
        dw = dw.sum(dim=0)                       # over batch
    return dx, dw


def token_shift(x, shift_logit):
    """Eq. shift-linear's mix: a_t x_{t-1} + (1 - a_t) x_t with a_t = sigmoid(logit_t)
    and x_0 = 0.  x [.., L, d], shift_logit [.., L]."""
    x = _f64(x)
    a = torch.sigmoid(_f64(shift_logit))[..., None]
    prev = torch.zeros_like(x)
    prev[..., 1:, :] = x[..., :-1, :]
    return a * prev + (1.0 - a) * x


def token_shift_backward(x, shift_logit, dy):
    """Gradients of sum(token_shift(x) o dy): x_t enters output t with weight
    (1 - a_t) and output t + 1 with weight a_{t+1}; d logit_t = a_t (1 - a_t)
    (x_{t-1} - x_t) . dy_t."""
    x, dy = _f64(x), _f64(dy)
    a = torch.sigmoid(_f64(shift_logit))
    dx = (1.0 - a)[..., None] * dy
    dx[..., :-1, :] += a[..., 1:, None] * dy[..., 1:, :]
    prev = torch.zeros_like(x)
    prev[..., 1:, :] = x[..., :-1, :]
    dlogit = a * (1.0 - a) * ((prev - x) * dy).sum(dim=-1)
    return dx, dlogit


def pro_prologue(q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                 k_norm_weight, eps: float):
    """q, k, v of a FoX (Pro) layer from the raw projections [B,H,L,d], the shift
    logits [B,H,L] and the QK-norm weights [H,d]."""
    q, _ = rms_norm(q_raw, q_norm_weight, eps)
    k, _ = rms_norm(token_shift(k_raw, k_shift_logit), k_norm_weight, eps)
    v = token_shift(v_raw, v_shift_logit)
    return q, k, v


def pro_prologue_backward(q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                          k_norm_weight, eps: float, dq, dk, dv):
    """Gradients of sum(q o dq + k o dk + v o dv) with respect to the raw
    projections, the shift logits and the QK-norm weights:
    (dq_raw, dk_raw, dv_raw, dk_shift_logit, dv_shift_logit, dq_norm_weight,
    dk_norm_weight)."""
    dq_raw, dwq = rms_norm_backward(q_raw, q_norm_weight, eps, dq)
    k_mix = token_shift(k_raw, k_shift_logit)
    dk_mix, dwk = rms_norm_backward(k_mix, k_norm_weight, eps, dk)
    dk_raw, dka = token_shift_backward(k_raw, k_shift_logit, dk_mix)
    dv_raw, dva = token_shift_backward(v_raw, v_shift_logit, dv)
    return dq_raw, dk_raw, dv_raw, dka, dva, dwq, dwk


def output_gate(o, g_logit, o_norm_weight, eps: float):
    """y = RMSNorm_o(o) o sigmoid(g): o, g_logit [B,H,L,d]; o_norm_weight [H,d]."""
    n, _ = rms_norm(o, o_norm_weight, eps)
    return n * torch.sigmoid(_f64(g_logit))


def output_gate_backward(o, g_logit, o_norm_weight, eps: float, dy):
    """Gradients of sum(y o dy): (do, dg_logit, do_norm_weight).  With
    u = RMSNorm_o(o) and sg = sigmoid(g): du = dy o sg, dg = dy o u o sg (1 - sg)."""
    dy = _f64(dy)
    sg = torch.sigmoid(_f64(g_logit))
    u, _ = rms_norm(o, o_norm_weight, eps)
    do, dw = rms_norm_backward(o, o_norm_weight, eps, dy * sg)
    dg = dy * u * sg * (1.0 - sg)
    return do, dg, dw


def pro_forward(q, k, v, logit, g_logit, o_norm_weight, eps: float, scale: float):
    """Attention followed by the output norm and gate: (y, O, LSE)."""
    O, LSE = forward(q, k, v, logit, scale)
    return output_gate(O, g_logit, o_norm_weight, eps), O, LSE


def pro_backward(q, k, v, logit, g_logit, o_norm_weight, eps: float, scale: float, dy):
    """Gradients of sum(y o dy) for pro_forward:
    (dQ, dK, dV, d(log f), dg_logit, do_norm_weight)."""
    O, _ = forward(q, k, v, logit, scale)
    dO, dg, dw = output_gate_backward(O, g_logit, o_norm_weight, eps, dy)
    dQ, dK, dV, dlf = backward(q, k, v, logit, dO, scale)
    return dQ, dK, dV, dlf, dg, dw

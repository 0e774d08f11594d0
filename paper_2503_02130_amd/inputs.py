"""Seeded synthetic inputs for Forgetting Attention workloads.

This module only draws random numbers; it holds none of the method's
arithmetic, so that the HIP path and the fp64 oracle can be fed the very same
tensors.  Shapes and distributions follow the paper's workloads:

  * q, k, v and the upstream gradient dO are i.i.d. N(0, 1), drawn in fp32 and
    rounded to the working dtype (bf16 rounding is round-to-nearest-even);
  * forget-gate logits are fp32.  Their distributions stand in for the strong-
    and weak-decay heads the paper visualises (Sec. 4.2, Fig. 3 and the
    appendix visualisations): a single N(mean, std) for every head, a per-head
    mean drawn uniformly from an interval, or a split of the heads into two
    groups with different distributions;
  * head dims 64 and 128 (model configuration table), sequence lengths 2048
    (SlimPajama experiments), 16384 (LongCrawl64 training context) and 65536
    (length-extrapolation evaluation).

The datasets the paper trains on are not available; these N(0, 1) stand-ins
have the same shapes.  Normal distributions are written N(mean, std).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, Tuple

import torch

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str                 # "fwd", "fwdbwd" or "decode"
    dtype: str                # "f32" or "bf16"
    B: int
    H: int
    L: int                    # sequence length; for decode the cache length T
    d: int
    gate: Tuple               # see gate_logits()
    seed: int
    note: str = ""


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("fwd_f32_b1_h2_l256_d64", "fwd", "f32", 1, 2, 256, 64,
             ("normal", 2.0, 1.0), 20250303,
             "small fp32 forward, logits N(2,1)"),
    Workload("fwdbwd_bf16_b8_h12_l2048_d64", "fwdbwd", "bf16", 8, 12, 2048, 64,
             ("normal", 2.0, 1.0), 20250304,
             "125M-model head shape at a 2k context, logits N(2,1)"),
    Workload("fwdbwd_bf16_b2_h16_l16384_d128", "fwdbwd", "bf16", 2, 16, 16384, 128,
             ("head_mean_uniform", 0.0, 6.0, 1.0), 20250305,
             "long-context training shape, per-head logit mean U[0,6], std 1"),
    Workload("fwd_bf16_b1_h16_l65536_d128", "fwd", "bf16", 1, 16, 65536, 128,
             ("split_heads", (6.0, 1.0), (0.0, math.sqrt(2.0))), 20250306,
             "length-extrapolation prefill; heads 0-7 logits N(6,1), heads 8-15 N(0, var 2)"),
    Workload("decode_bf16_b64_h16_t32768_d128", "decode", "bf16", 64, 16, 32768, 128,
             ("normal", 3.0, 1.0), 20250307,
             "one new token per sequence against 32768 cached keys (the new one included)"),
]}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFFFFFFFFFF)
    return g


def randn(shape, dtype: str, g: torch.Generator, device, chunk_dim0: bool = False) -> torch.Tensor:
    """N(0,1) in fp32, rounded to `dtype`.  With chunk_dim0 the draw is done one
    leading index at a time (bounded fp32 scratch for very large tensors)."""
    dt = DTYPES[dtype]
    if not chunk_dim0:
        return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(dt)
    out = torch.empty(shape, device=device, dtype=dt)
    for i in range(shape[0]):
        out[i] = torch.randn(shape[1:], generator=g, device=device, dtype=torch.float32).to(dt)
    return out


def gate_logits(spec: Tuple, B: int, H: int, L: int, g: torch.Generator, device) -> torch.Tensor:
    """fp32 gate logits [B, H, L].

    ("normal", mean, std)                 every element N(mean, std)
    ("head_mean_uniform", lo, hi, std)    mean_h ~ U[lo, hi] once per head (shared
                                          over the batch), elements N(mean_h, std)
    ("split_heads", (m0, s0), (m1, s1))   heads [0, H/2) N(m0, s0), the rest N(m1, s1)
    """
    z = torch.randn((B, H, L), generator=g, device=device, dtype=torch.float32)
    kind = spec[0]
    if kind == "normal":
        return z * spec[2] + spec[1]
    if kind == "head_mean_uniform":
        lo, hi, std = spec[1], spec[2], spec[3]
        mu = torch.rand((H,), generator=g, device=device, dtype=torch.float32) * (hi - lo) + lo
        return z * std + mu[None, :, None]
    if kind == "split_heads":
        (m0, s0), (m1, s1) = spec[1], spec[2]
        mean = torch.full((H,), m1, device=device, dtype=torch.float32)
        std = torch.full((H,), s1, device=device, dtype=torch.float32)
        mean[: H // 2] = m0
        std[: H // 2] = s0
        return z * std[None, :, None] + mean[None, :, None]
    if kind == "constant":
        return torch.full((B, H, L), float(spec[1]), device=device, dtype=torch.float32)
    raise ValueError(f"unknown gate spec {spec!r}")


def attn_inputs(B: int, H: int, L: int, d: int, dtype: str, gate: Tuple, seed: int,
                device="cpu", grad: bool = True) -> Dict[str, torch.Tensor]:
    """q, k, v [B,H,L,d] (dtype), logit [B,H,L] fp32 and, with grad, dO [B,H,L,d]."""
    g = _gen(seed, device)
    big = B * H * L * d > (1 << 26)
    out = {
        "q": randn((B, H, L, d), dtype, g, device, big),
        "k": randn((B, H, L, d), dtype, g, device, big),
        "v": randn((B, H, L, d), dtype, g, device, big),
        "logit": gate_logits(gate, B, H, L, g, device),
    }
    if grad:
        out["do"] = randn((B, H, L, d), dtype, g, device, big)
    return out


def pro_inputs(B: int, H: int, L: int, d: int, dtype: str, gate: Tuple, seed: int,
               device="cpu") -> Dict[str, torch.Tensor]:
    """Inputs of a FoX (Pro) layer around the attention: raw projections q_raw,
    k_raw, v_raw and the output-gate logits g [B,H,L,d] N(0,1) (dtype); the token
    shift logits k_shift, v_shift [B,H,L] fp32 N(0, 2) (mix weights spread over
    (0, 1)); per-head norm weights wq, wk, wo [H,d] fp32 1 + N(0, 0.1^2); the
    forget-gate logits [B,H,L] by `gate`; upstream gradients dq, dk, dv, dy
    [B,H,L,d] N(0,1) (dtype)."""
    g = _gen(seed, device)
    f32 = dict(generator=g, device=device, dtype=torch.float32)
    out = {name: randn((B, H, L, d), dtype, g, device) for name in ("q_raw", "k_raw", "v_raw")}
    out["k_shift"] = torch.randn((B, H, L), **f32) * 2.0
    out["v_shift"] = torch.randn((B, H, L), **f32) * 2.0
    for name in ("wq", "wk", "wo"):
        out[name] = 1.0 + 0.1 * torch.randn((H, d), **f32)
    out["logit"] = gate_logits(gate, B, H, L, g, device)
    for name in ("g", "dq", "dk", "dv", "dy"):
        out[name] = randn((B, H, L, d), dtype, g, device)
    return out


def decode_inputs(B: int, H: int, T: int, d: int, dtype: str, gate: Tuple, seed: int,
                  device="cpu") -> Dict[str, torch.Tensor]:
    """One decode step: q [B,H,d]; k_cache, v_cache [B,H,T,d] whose slot T-1 is
    the new token; cached_logit [B,H,T-1] for tokens 1..T-1 and logit_new [B,H]."""
    g = _gen(seed, device)
    logits = gate_logits(gate, B, H, T, g, device)
    return {
        "q": randn((B, H, d), dtype, g, device),
        "k_cache": randn((B, H, T, d), dtype, g, device, True),
        "v_cache": randn((B, H, T, d), dtype, g, device, True),
        "cached_logit": logits[..., : T - 1].contiguous(),
        "logit_new": logits[..., T - 1].contiguous(),
    }


def projection_inputs(B: int, L: int, H: int, M: int, dtype: str, seed: int,
                      device="cpu") -> Dict[str, torch.Tensor]:
    """The forget-gate projection's operands: the layer input x [B,L,M] ~ N(0, 1)
    in `dtype`; w_f [H,M] ~ N(0, 0.02) (the paper's weight initialisation) and
    b_f [H] ~ N(0, 1) in fp32; an upstream d_logit [B,H,L] ~ N(0, 1) in fp32."""
    g = _gen(seed, device)
    return {
        "x": randn((B, L, M), dtype, g, device, True),
        "w_f": 0.02 * torch.randn((H, M), generator=g, device=device, dtype=torch.float32),
        "b_f": torch.randn((H,), generator=g, device=device, dtype=torch.float32),
        "d_logit": torch.randn((B, H, L), generator=g, device=device, dtype=torch.float32),
    }


def rescale_inputs(B: int, H: int, L: int, d: int, dtype: str, gate: Tuple, seed: int,
                   device="cpu") -> Dict[str, torch.Tensor]:
    """Inputs whose softmax rows are dominated by a few early keys: the shape of
    attention-sink rows.  Per (b, h) a random unit direction u; every query is
    sqrt(d) u plus N(0, 0.3^2) noise, so that s q.k_j is about u.k_j for the
    N(0, 1) keys; a key in each of up to five early 64-key tiles (0, 3, .., 12) is
    a multiple of u whose score is 12 nats for the latest and 7 nats more for each
    earlier one;
    the key at every 64-key tile start is -3 sqrt(d) u + noise, so the first query
    of a tile sees its own key at a very low score.  With the 1/sqrt(d) scale
    these give scores far above each query's nearby ones.  dO ~ N(0, 1)."""
    g = _gen(seed, device)
    f32 = dict(generator=g, device=device, dtype=torch.float32)
    u = torch.randn((B, H, 1, d), **f32)
    u = u / torch.linalg.vector_norm(u, dim=-1, keepdim=True)
    sd = math.sqrt(d)
    q = sd * u + 0.3 * torch.randn((B, H, L, d), **f32)
    k = torch.randn((B, H, L, d), **f32)
    n_tiles = (L + 63) // 64
    planted = [t for t in range(0, min(n_tiles - 1, 15), 3)]  # tiles 0, 3, .., 12
    for rank, t in enumerate(reversed(planted)):             # later tile, lower score
        k[:, :, 64 * t + 17] = (12.0 + 7.0 * rank) * u[:, :, 0]
    for t in range(1, n_tiles):
        k[:, :, 64 * t] = -3.0 * sd * u[:, :, 0] + 0.3 * torch.randn((B, H, d), **f32)
    dt = DTYPES[dtype]
    return {
        "q": q.to(dt),
        "k": k.to(dt),
        "v": randn((B, H, L, d), dtype, g, device),
        "logit": gate_logits(gate, B, H, L, g, device),
        "do": randn((B, H, L, d), dtype, g, device),
    }


def workload_inputs(w: Workload, device="cpu", seed: int = None) -> Dict[str, torch.Tensor]:
    s = w.seed if seed is None else seed
    if w.kind == "decode":
        return decode_inputs(w.B, w.H, w.L, w.d, w.dtype, w.gate, s, device)
    return attn_inputs(w.B, w.H, w.L, w.d, w.dtype, w.gate, s, device, grad=(w.kind == "fwdbwd"))

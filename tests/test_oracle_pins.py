"""The fp64 oracle against the paper's closed forms, invariants and brute force."""
import math

import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle)


@settings(max_examples=40, deadline=None)
@given(L=st.integers(1, 64), d=st.integers(1, 8), mean=st.floats(-3, 8), std=st.floats(0.0, 3.0),
       seed=st.integers(0, 2**31 - 1))
def test_properties_random_shapes(L, d, mean, std, seed):
    """P4-P7 as properties over random lengths, head dims and gate distributions."""
    g = torch.Generator().manual_seed(seed)
    q, k, v, dO = (torch.randn(1, 1, L, d, generator=g, dtype=torch.float64) for _ in range(4))
    x = torch.randn(1, 1, L, generator=g, dtype=torch.float64) * std + mean
    s = 1.0 / math.sqrt(d)
    lf = oracle.log_sigmoid(x)
    assert torch.all(lf < 0) or torch.all(lf <= 0)
    c = oracle.prefix_c(lf)[0, 0]
    O, LSE, A = oracle.forward_head_from_c(q[0, 0], k[0, 0], v[0, 0], c, s, return_A=True)
    assert torch.allclose(A.sum(1), torch.ones(L, dtype=torch.float64), atol=1e-12)
    assert torch.all(torch.triu(A, 1) == 0)
    assert torch.allclose(O[0], v[0, 0, 0], atol=1e-12)
    # every output row is a convex combination of value rows
    vmin, vmax = v[0, 0].min(0).values, v[0, 0].max(0).values
    assert torch.all(O >= vmin - 1e-12) and torch.all(O <= vmax + 1e-12)
    _, _, _, dc, dS = oracle.backward_head_from_c(q[0, 0], k[0, 0], v[0, 0], c, dO[0, 0], s,
                                                  return_dS=True)
    assert abs(float(dc.sum())) < 1e-9
    assert torch.allclose(dS.sum(1), torch.zeros(L, dtype=torch.float64), atol=1e-10)
    dlf = oracle.reverse_cumsum(dc)
    assert abs(float(dlf[0])) < 1e-9


def test_decode_uses_new_gate_only_through_c_T():
    """c_T = c_{T-1} + log sigmoid(x_new), and c_0 = 0 for T = 1."""
    g = torch.Generator().manual_seed(3)
    q = torch.randn(1, 1, 4, generator=g, dtype=torch.float64)
    kc, vc = (torch.randn(1, 1, 1, 4, generator=g, dtype=torch.float64) for _ in range(2))
    o, lse, cT = oracle.decode(q, kc, vc, torch.zeros(1, 1, 0), torch.tensor([[0.0]]), 0.5)
    assert torch.allclose(o[0, 0], vc[0, 0, 0])
    assert abs(float(cT) + math.log(2.0)) < 1e-15

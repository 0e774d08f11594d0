"""The throughput metric counts causal FLOPs the way the paper's FLOP table does.

The table gives forward FLOPs/token = 2N + 2 n_layer d_model L (fixture
tests/golden/flops_per_token.txt); the attention part 2 n_layer d_model L is
QK^T and PV at 2 FLOPs per multiply-add over the L/2 keys an average causal
query sees.  bench.py's 4d FLOPs per causal pair must reproduce it.
"""
import os

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "flops_per_token.txt")


def _fixture():
    vals = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        k, v = line.split(None, 1)
        vals[k] = v.strip()
    return vals


def test_forward_flops_per_token_match_the_paper():
    g = _fixture()
    n_layer, d_model, L = int(g["n_layer"]), int(g["d_model"]), int(g["context_length"])
    N = float(g["params"])
    d = 64                                   # FoX head dim in the 760M configuration
    H = d_model // d
    attn_per_token = bench.fwd_flops(1, H, L, d) / L * n_layer
    # causal pairs L(L+1)/2 vs the table's L^2/2: equal up to 1/L
    assert abs(attn_per_token / (2 * n_layer * d_model * L) - 1) < 2.0 / L
    total = 2 * N + attn_per_token
    # the table prints three significant figures (2.726e9 appears as 2.72e9)
    assert abs(total - float(g["flops_per_token"])) < 0.01e9


def test_backward_is_two_and_a_half_forwards():
    # dV, dP, dQ, dK plus the recomputed QK^T: five products against two
    assert bench.bwd_flops(2, 16, 16384, 128) == 2.5 * bench.fwd_flops(2, 16, 16384, 128)


def test_decode_bytes():
    # K and V in bf16 plus the fp32 prefix value, per cached key
    assert bench.decode_bytes(64, 16, 32768, 128) == 64 * 16 * 32768 * (2 * 128 * 2 + 4)

"""fox_attn_decode_noalloc (the decode step without a workspace, for callers that
cannot allocate) against fox_attn_decode through the C ABI: bit for bit, on
calls in a row whose shapes shrink (the scratch array keeps the previous call's
partials; nothing of them may leak into a smaller call)."""
import pytest
import torch

import paper_2503_02130_amd as fox
from paper_2503_02130_amd import inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _decode_pair(B, H, T, d, dtype, seed):
    y = inputs.decode_inputs(B, H, T, d, dtype, ("normal", 3.0, 1.0), seed, device=DEV)
    cc = torch.full((B, H, T), float("nan"), device=DEV)
    if T > 1:
        cc[..., : T - 1] = fox.fox_gate_prefix(y["cached_logit"])
    cc2 = cc.clone()
    o_ref, lse_ref = fox.fox_attn_decode(y["q"], y["k_cache"], y["v_cache"], cc, y["logit_new"])
    o, lse = torch.empty_like(o_ref), torch.empty_like(lse_ref)
    torch.cuda.synchronize()
    alloc0 = torch.cuda.memory_allocated()
    free0 = torch.cuda.mem_get_info()[0]
    fox.fox_attn_decode_noalloc(y["q"], y["k_cache"], y["v_cache"], cc2, y["logit_new"], o=o,
                                lse=lse)
    torch.cuda.synchronize()
    # nothing allocated: neither through torch nor on the device
    assert torch.cuda.memory_allocated() == alloc0
    assert torch.cuda.mem_get_info()[0] == free0
    assert torch.equal(o, o_ref), (B, H, T, d, dtype)
    assert torch.equal(lse, lse_ref), (B, H, T, d, dtype)
    assert torch.equal(cc2, cc), (B, H, T, d, dtype)


def test_decode_noalloc_equals_decode_on_shrinking_calls():
    # the decode workload's shape (16.25 MiB of partials), then smaller ones
    cases = [(64, 16, 32768, 128, "bf16", 1), (4, 8, 5000, 128, "bf16", 2),
             (2, 3, 700, 64, "bf16", 3), (1, 2, 77, 64, "f32", 4), (1, 1, 1, 128, "bf16", 5)]
    for B, H, T, d, dtype, seed in cases:
        print(f"noalloc decode B={B} H={H} T={T} d={d} {dtype}", flush=True)
        _decode_pair(B, H, T, d, dtype, seed)
        torch.cuda.empty_cache()

"""A host model of when the bf16 forward kernel takes its rescale path.

The kernel (fwd_bf16_kernel) gives each wave 32 queries of a 128-query block
and visits 64-key tiles from the wave's diagonal tile backwards.  The diagonal
tile fixes the per-query reference m (its maximum of u = log2(e) (s q.k + c_q0
- c_j), c_q0 the prefix value at the block's first query; keys after the query
masked).  Every earlier tile is exponentiated against m without a maximum
search; a lane (one query, the 32 keys of its half of the tile: key % 8 in
4h .. 4h + 3) sums its bf16-rounded exp2(u - m).  If any valid lane's sum
exceeds 2^8, the whole wave takes the slow path for that tile: tile maximum,
m += max(tile max - m, 0), O and l rescaled, exponentiate again.  This is the
online-softmax rescale of Alg. 1 (the FlashAttention-2 update), taken lazily.

This module restates that decision rule in fp32 torch on the CPU (the sums
differ from the kernel's only in summation order, which matters only for sums
within rounding of 2^8).  It models the kernel, not the method: the oracle does
not use it.  It serves the GPU test that must drive the kernel through the slow
path, and measures how often the path runs on a workload.
"""
import math

import torch

LOG2E = 1.4426950408889634
BLOCK = 128        # queries per workgroup
WAVE = 32          # queries per wave
TILE = 64          # keys per tile
SLACK_SUM = 256.0  # 2^8


def rescale_events(q, k, c, scale):
    """For one (batch, head) slice: q, k [L, d] (the values the kernel reads,
    e.g. bf16), c [L] fp32 prefix values.  Returns (fired, visited, repeat): the
    number of (wave, earlier tile) pairs that take the slow path, of all (wave,
    earlier tile) pairs, and the largest number of slow-path tiles of one wave
    (above 1: the wave's maximum rose again after a rescale)."""
    q = q.float()
    k = k.float()
    c = c.float()
    L = q.shape[0]
    n_waves = (L + WAVE - 1) // WAVE
    fired = 0
    visited = 0
    repeat = 0
    chunk = 32 * WAVE  # rows per pass
    for r0 in range(0, n_waves * WAVE, chunk):
        r1 = min(r0 + chunk, n_waves * WAVE)
        rows = torch.arange(r0, r1)
        valid = rows < L
        rows_c = rows.clamp(max=L - 1)
        q0 = (rows // BLOCK) * BLOCK
        kmax = int(min(L, ((r1 - 1) // TILE + 1) * TILE))
        qk = torch.zeros(r1 - r0, kmax)
        qk[valid] = q[rows_c[valid]] @ k[:kmax].T
        u = LOG2E * (scale * qk + (c[q0.clamp(max=L - 1)][:, None] - c[None, :kmax]))
        keys = torch.arange(kmax)
        wave_first = (rows // WAVE) * WAVE
        t_diag = wave_first // TILE
        # the diagonal tile: keys 64 t_diag .. the query itself
        in_diag = (keys[None, :] >= (t_diag * TILE)[:, None]) & (keys[None, :] <= rows[:, None])
        m = torch.where(in_diag, u, torch.tensor(-math.inf)).amax(dim=1)
        # per-wave sweep over earlier tiles, diagonal backwards
        nw = (r1 - r0) // WAVE
        t_d = t_diag.view(nw, WAVE)[:, 0]
        valid_w = valid.view(nw, WAVE)
        m = m.view(nw, WAVE).clone()
        u = u.view(nw, WAVE, kmax)
        half = ((torch.arange(TILE) % 8) // 4)           # the lane half holding each key
        per_wave = torch.zeros(nw, dtype=torch.long)
        for j in range(int(t_d.max()) - 1, -1, -1):
            act = t_d > j
            if not bool(act.any()):
                continue
            ut = u[:, :, j * TILE:(j + 1) * TILE][act]     # [w, 32, 64]
            ma = m[act]
            p = torch.exp2(ut - ma[:, :, None]).to(torch.bfloat16).float()
            s0 = p[:, :, half == 0].sum(-1)
            s1 = p[:, :, half == 1].sum(-1)
            over = ((s0 > SLACK_SUM) | (s1 > SLACK_SUM)) & valid_w[act]
            fire = over.any(dim=1)                       # the wave-wide test
            visited += int(act.sum())
            fired += int(fire.sum())
            per_wave[act] += fire.long()
            if bool(fire.any()):
                tmax = ut.amax(dim=-1)
                shift = torch.clamp(tmax - ma, min=0.0)
                ma = torch.where(fire[:, None], ma + shift, ma)
                m[act] = ma
        repeat = max(repeat, int(per_wave.max()))
    return fired, visited, repeat

"""Host-side models of the kernels' LDS and workspace addressing (no GPU).

The MFMA kernels rely on index arithmetic that no GPU test can check directly:
that their swizzled LDS tiles are read without bank conflicts, that each DMA
load fills every tile position exactly once, and, for the backward keeping dS
(the dQ half of Alg. 2 reading the dS its dK/dV half stored), that every store
lands inside its slot run once and every read names a chunk that was written,
also when gate-aware skipping cuts the stored tiles of each key block.  The
scans' 16-byte accesses and the Delta kernel's row mapping are modelled too.

Each model restates the kernel's formula in Python.  The constants are read
from the kernel sources, and the formulas the models restate are matched
against the source text, so a change to the kernels that the models do not
follow fails here.
"""
import os
import random
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2503_02130_amd", "csrc")


def _src(name):
    with open(os.path.join(CSRC, name)) as f:
        return f.read()


BWD = _src("attn_bwd.hip")
DEV = _src("fox_device.h")


def _const(text, name):
    m = re.search(r"constexpr int %s = ([^;]+);" % name, text)
    assert m, f"{name} not found"
    return m.group(1).strip()


SLOT_BYTES = int(_const(BWD, "kDsSlotBytes"))           # one (key block, query tile) pair
CHUNK_LDS = int(_const(BWD, "kDsChunkLds"))             # LDS bytes per 1 KB stored chunk
KEYS_PER_BLOCK = 128                                    # dK/dV workgroup: 4 pairs x 32 keys
QUERY_TILE = 64
DQ_WAVES = int(_const(BWD, "kDsWaves"))
DQ_BM = 32 * DQ_WAVES                                   # queries per dQ-pass workgroup


def test_model_matches_the_kernel_source():
    """The formulas restated below, as the kernels write them."""
    assert SLOT_BYTES == 16384 and CHUNK_LDS == 1152 and DQ_WAVES == 8
    assert "return (L + 63) / 64;" in BWD and "return (L + 127) / 128;" in BWD
    assert "return nk * nq - nk * (nk - 1);" in BWD
    assert re.search(r"return \(size_t\)nb \* \(size_t\)ds_query_tiles\(L\) - "
                     r"\(size_t\)nb \* \(size_t\)\(nb - 1\) \+\s*\(size_t\)\(qt - 2 \* nb\);", BWD)
    assert "return slot ^ ((slot >> 5) << 2);" in BWD
    assert "(r2 | (r1 << 1) | (r0 << 2) | ((r3 ^ r1 ^ r0) << 3))" in DEV
    assert "(r2 | ((r0 ^ r3) << 1) | (r1 << 2))" in DEV
    assert re.search(r"DOFF = \(B == 2 \? 0 : B \* \(int\)sizeof\(sm\.ds\[0\]\)\) \+ "
                     r"\(S / 2\) \* 4 \* kDsChunkLds \+\s*\(S % 2\) \* 256;", BWD)
    assert "bf16x8 ds[3][kDsTiles][kDsStageLds / 16];" in BWD
    assert "ds_addr + 2 * (uint32_t)sizeof(sm.ds[0])" in BWD


# ----------------------------------------------------------- swizzled tiles
def swz_chunk(D, r, c):
    r0, r1, r2, r3 = r & 1, (r >> 1) & 1, (r >> 2) & 1, (r >> 3) & 1
    if D == 128:
        f = r2 | (r1 << 1) | (r0 << 2) | ((r3 ^ r1 ^ r0) << 3)
    else:
        f = r2 | ((r0 ^ r3) << 1) | (r1 << 2)
    return c ^ f


def _max_way(addrs, nbytes, bank_bytes):
    """Largest number of distinct 4-byte words one bank serves for one access:
    `addrs` are byte addresses of `nbytes`-byte accesses served together."""
    nbanks = bank_bytes // 4
    banks = {}
    for a in addrs:
        for w in range(0, nbytes, 4):
            banks.setdefault(((a + w) // 4) % nbanks, set()).add(a + w)
    return max(len(v) for v in banks.values())


@pytest.mark.parametrize("D", [64, 128])
def test_swizzle_is_a_permutation_of_each_row(D):
    cpr = D // 8
    for r in range(64):
        assert sorted(swz_chunk(D, r, c) for c in range(cpr)) == list(range(cpr))


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("bank_bytes", [128, 256])
def test_plain_operand_reads_are_conflict_free(D, bank_bytes):
    """16-byte reads of one logical chunk by consecutive rows (the lanes of one
    LDS cycle: 8 rows at 128 B per cycle, 16 rows at 256 B) hit distinct banks."""
    rows_per_cycle = bank_bytes // 16
    for r0 in range(0, 64, rows_per_cycle):
        for c in range(D // 8):
            addrs = [r * D * 2 + swz_chunk(D, r, c) * 16 for r in range(r0, r0 + rows_per_cycle)]
            assert _max_way(addrs, 16, bank_bytes) == 1, (r0, c)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("bank_bytes", [128, 256])
def test_transposing_reads_are_conflict_free(D, bank_bytes):
    """ds_read_b64_tr_b16 from a swizzled tile (tile_tr_offsets): each group of
    16 lanes reads a 4 x 16 block, 4 rows (aligned to 4) by 2 logical chunks;
    the lanes served in one cycle (16 at 128 B, 32 at 256 B) hit distinct banks."""
    lanes_per_cycle = bank_bytes // 8
    for chunk16 in range(4):                      # 16-row chunk of a 64-row tile
        for k2 in range(2):
            for db in range(D // 32):
                addrs = []
                for lane in range(64):
                    g16, j16 = lane >> 4, lane & 15
                    r = 16 * chunk16 + 8 * k2 + 4 * (g16 >> 1) + (j16 >> 2)
                    e = db * 32 + 16 * (g16 & 1) + 4 * (j16 & 3)
                    addrs.append(r * D * 2 + swz_chunk(D, r, e >> 3) * 16 + (e & 7) * 2)
                for g0 in range(0, 64, lanes_per_cycle):
                    assert _max_way(addrs[g0:g0 + lanes_per_cycle], 8, bank_bytes) == 1


@pytest.mark.parametrize("D,nwaves,rows", [(128, 4, 64), (64, 4, 64), (128, 8, 64),
                                            (64, 8, 64), (128, 8, 128), (64, 4, 128)])
def test_tile_dma_fills_every_position_once(D, nwaves, rows):
    """tile_dma_offset: load i of wave w fills LDS slots [(i*nwaves + w)*64, +64)
    from global chunk offsets dma_off(w, lane) + i * stride.  Every (row, chunk)
    of the tile is fetched exactly once, into its swizzled position."""
    cpr = D // 8
    stride = nwaves * 64 * 16
    n_loads = rows * D * 2 // 1024 // nwaves
    seen = {}
    for w in range(nwaves):
        for lane in range(64):
            slot = w * 64 + lane
            r = slot // cpr
            off0 = r * D * 2 + swz_chunk(D, r, slot % cpr) * 16
            for i in range(n_loads):
                lds_slot = (i * nwaves + w) * 64 + lane
                g = off0 + i * stride
                row, chunk = g // (D * 2), (g % (D * 2)) // 16
                assert row < rows
                # the LDS slot holds logical chunk `chunk` of row `row` at its swizzled place
                assert lds_slot == row * cpr + swz_chunk(D, row, chunk)
                assert (row, chunk) not in seen
                seen[(row, chunk)] = lds_slot
    assert len(seen) == rows * cpr


# ----------------------------------------------------- stored dS: the slots
def qtiles(L):
    return (L + 63) // 64


def kblocks(L):
    return (L + 127) // 128


def slots_per_head(L):
    nq, nk = qtiles(L), kblocks(L)
    return nk * nq - nk * (nk - 1)


def slot(L, nb, qt):
    return nb * qtiles(L) - nb * (nb - 1) + (qt - 2 * nb)


def _stores(BH, L, cuts=None):
    """The chunks the dK/dV pass with the dS store writes: key block nb stores
    query tiles 2 nb .. cut(nb) - 1 (cut = all tiles without skipping); in tile
    qt, the G wave of pair p (keys 128 nb + 32 p ..) writes only when qt is on or
    below its diagonal tile, four 1 KB chunks (32-query half qb, 16-query chunk
    c).  Returns {byte offset of the chunk: (bh, nb, qt, pair, qb, c)}."""
    T = slots_per_head(L)
    total = BH * T * SLOT_BYTES
    n_qt = qtiles(L)
    written = {}
    for bh in range(BH):
        for nb in range(kblocks(L)):
            t_first = 2 * nb
            cut = n_qt if cuts is None else cuts[bh][nb]
            base = (bh * T + slot(L, nb, t_first)) * SLOT_BYTES
            run = (n_qt - t_first) * SLOT_BYTES        # the block's slot run
            for pair in range(4):
                t_diag = (nb * KEYS_PER_BLOCK + pair * 32) // QUERY_TILE
                for qt in range(t_first, cut):
                    if qt < t_diag:
                        continue
                    for qb in range(2):
                        for c in range(2):
                            soff = (qt - t_first) * SLOT_BYTES + pair * 4096 + (2 * qb + c) * 1024
                            assert soff + 1024 <= run, (L, nb, qt)
                            a = base + soff
                            assert a + 1024 <= total
                            assert a not in written, "two stores to one chunk"
                            written[a] = (bh, nb, qt, pair, qb, c)
    return written


def _first_block(cut, qt0):
    """The dQ pass's binary search: the first key block whose stored tiles reach qt0."""
    lo, hi = 0, qt0 // 2
    while lo < hi:
        mid = (lo + hi) >> 1
        if cut[mid] > qt0:
            hi = mid
        else:
            lo = mid + 1
    return lo


def _check_reads(BH, L, written, cuts=None):
    """The dQ pass: a workgroup owns four 64-query tiles (qt0 ..); stage j (64 keys,
    half of key block j // 2) reads, for its tiles t_lo .. t_hi - 1, the stage's
    half of each slot, one 1 KB chunk per wave.  Every read must name a written
    chunk of the right (head, block, tile), and every tile that needs the stage
    (on or below the diagonal, stored) must be inside the range read."""
    T = slots_per_head(L)
    n_qt = qtiles(L)
    for bh in range(BH):
        cut = [n_qt] * kblocks(L) if cuts is None else cuts[bh]
        for mblk in range((L + DQ_BM - 1) // DQ_BM):
            q0 = mblk * DQ_BM
            qt0 = q0 // 64
            n_st = (min(L, q0 + DQ_BM) + 63) // 64
            j_first = 2 * _first_block(cut, qt0) if cuts is not None else 0
            for j in range(0, j_first):                 # skipped stages hold exact zeros only
                for t in range(DQ_BM // 64):
                    qt = qt0 + t
                    assert not (j <= qt < min(n_qt, cut[j >> 1])), (L, bh, mblk, j)
            for j in range(j_first, n_st):
                nb = j >> 1
                t_lo, t_hi = max(0, j - qt0), min(min(DQ_BM // 64, n_qt - qt0), cut[nb] - qt0)
                if t_lo < t_hi:
                    assert qt0 + t_lo >= 2 * nb
                rbase = (bh * T + slot(L, nb, qt0 + t_lo)) * SLOT_BYTES
                for t in range(t_lo, t_hi):
                    for wave in range(DQ_WAVES):
                        off = (t - t_lo) * SLOT_BYTES + (j & 1) * (SLOT_BYTES // 2) + wave * 1024
                        assert off + 1024 <= (t_hi - t_lo) * SLOT_BYTES
                        got = written.get(rbase + off)
                        assert got is not None, (L, bh, mblk, j, t, wave)
                        pair, qb_c = 2 * (j & 1) + wave // 4, wave % 4
                        assert got == (bh, nb, qt0 + t, pair, qb_c // 2, qb_c % 2)
                for w in range(DQ_WAVES):
                    qt = qt0 + (w >> 1)
                    if j <= qt < min(n_qt, cut[nb]):
                        assert t_lo <= qt - qt0 < t_hi


LENGTHS = [1, 2, 63, 64, 65, 127, 128, 129, 255, 256, 257, 513, 700, 1000, 1100, 2048]


@pytest.mark.parametrize("L", LENGTHS)
def test_stored_ds_slots_written_once_and_read_back(L):
    for BH in (1, 3):
        written = _stores(BH, L)
        _check_reads(BH, L, written)
        # the workspace size the library asks for holds exactly the slots
        assert max(written) + 1024 <= BH * slots_per_head(L) * SLOT_BYTES


def _random_cuts(BH, L, rnd):
    """Monotone cutoffs like gate-aware skipping produces: block nb stores at least
    its diagonal tiles (cut >= 2 nb + 1) and cut never decreases with nb (c never
    increases along the sequence)."""
    nq = qtiles(L)
    out = []
    for _ in range(BH):
        cut, prev = [], 0
        for nb in range(kblocks(L)):
            lo = max(prev, 2 * nb + 1)
            v = min(rnd.randint(lo, nq) if rnd.random() < 0.7 else lo, nq)
            cut.append(v)
            prev = v
        out.append(cut)
    return out


@pytest.mark.parametrize("L", [1, 63, 64, 65, 128, 129, 255, 256, 257, 700, 1000, 2048, 4097])
def test_stored_ds_with_skipping_cutoffs(L):
    rnd = random.Random(L)
    for BH in (1, 3):
        for _ in range(3):
            cuts = _random_cuts(BH, L, rnd)
            for c in cuts:
                assert all(a <= b for a, b in zip(c, c[1:]))
            written = _stores(BH, L, cuts)
            _check_reads(BH, L, written, cuts)


# -------------------------------------------------- stored dS: LDS banks
def ds_lds_pos(s):
    return s ^ ((s >> 5) << 2)


def _ds_read_addr(lane, qb, S, k2, chunk_lds, permute):
    """Byte address of a dQ-pass B-operand transposing read of stored dS in LDS:
    16-key step S (pair S // 2, keys 16 (S % 2) ..), half k2 of its 16 keys."""
    g16, j16 = lane >> 4, lane & 15
    cg, r = j16 & 3, j16 >> 2
    hh, c = g16 >> 1, g16 & 1
    hp, g2 = cg & 1, cg >> 1
    chunk = (S // 2) * 4 + qb * 2 + c
    s = hp * 32 + 16 * (S % 2) + 4 * hh + r + 8 * k2
    return chunk * chunk_lds + (ds_lds_pos(s) if permute else s) * 16 + g2 * 8


@pytest.mark.parametrize("group", [16, 32])
def test_stored_ds_reads_are_conflict_free(group):
    """With 1152-byte chunks and the (32 + k) ^ 4 slot permutation, the 16 slots a
    transposing read touches sit in distinct banks for any 16 or 32 lanes; the
    plain layout (1 KB chunks, no permutation) had 2- to 4-way conflicts."""
    def worst(chunk_lds, permute):
        w = 1
        for qb in range(2):
            for S in range(4):
                for k2 in range(2):
                    for g0 in range(0, 64, group):
                        addrs = [_ds_read_addr(l, qb, S, k2, chunk_lds, permute)
                                 for l in range(g0, g0 + group)]
                        w = max(w, _max_way(addrs, 8, 256))
        return w
    assert worst(CHUNK_LDS, True) == 1
    assert worst(1024, False) >= 2


def test_stored_ds_buffers_fit_the_immediate_offsets():
    """The dQ pass keeps three stored-dS buffers of kDsTiles x kDsStageLds bytes;
    buffers 0 and 1 are reached from one base register plus an immediate, buffer 2
    (beyond the 16-bit reach of an LDS immediate) from a second base: every
    immediate stays below 2^16 and every buffer's address is the same either way."""
    buf = 4 * (SLOT_BYTES // 2 // 1024) * CHUNK_LDS         # sizeof(sm.ds[0])
    for B in range(3):
        base = 2 * buf if B == 2 else 0
        for S in range(4):
            for k2 in range(2):
                imm = (0 if B == 2 else B * buf) + (S // 2) * 4 * CHUNK_LDS + (S % 2) * 256 + 128 * k2
                assert imm < 1 << 16, (B, S, k2)
                assert base + imm == B * buf + (S // 2) * 4 * CHUNK_LDS + (S % 2) * 256 + 128 * k2
    # the K tiles of the three stages (64 keys x D bf16 each) stay within reach too
    for D in (64, 128):
        for B in range(3):
            assert 2 * (B * 64 * D + 3 * 16 * D) < 1 << 16


def test_stored_ds_permutation_and_immediates():
    # the DMA permutation is an involution of the 64 lane slots of a chunk
    assert sorted(ds_lds_pos(s) for s in range(64)) == list(range(64))
    assert all(ds_lds_pos(ds_lds_pos(s)) == s for s in range(64))
    # the per-step part of the address (S, k2) is a constant immediate: it never
    # interacts with the permuted bit (bit 2 of the slot)
    for lane in range(64):
        for qb in range(2):
            base = _ds_read_addr(lane, qb, 0, 0, CHUNK_LDS, True)
            for S in range(4):
                for k2 in range(2):
                    imm = (S // 2) * 4 * CHUNK_LDS + (S % 2) * 256 + k2 * 128
                    assert _ds_read_addr(lane, qb, S, k2, CHUNK_LDS, True) == base + imm


# ------------------------------------------------------------------ scans, Delta
SCAN = _src("gate_scan.hip")


def test_scan_model_matches_the_kernel_source():
    assert _const(SCAN, "kScanThreads") == "1024" and _const(SCAN, "kScanPerThread") == "8"
    assert "constexpr bool FWD = MODE == 0 || MODE == 3;" in SCAN
    assert "auto pos = [&](int p) { return (size_t)(FWD ? p : L - 1 - p); };" in SCAN
    assert "const int p0 = seg + threadIdx.x * kScanPerThread;" in SCAN
    assert "const bool whole = VEC && p0 + kScanPerThread <= L;" in SCAN
    assert ("const size_t i0 = base + (FWD ? (size_t)p0 : (size_t)(L - kScanPerThread - p0));"
            in SCAN)
    assert "auto at = [&](int e) { return FWD ? e : kScanPerThread - 1 - e; };" in SCAN
    assert "if (aligned && L > kScanSegment) {" in SCAN
    assert "if (L % 4) return false;" in SCAN


@pytest.mark.parametrize("fwd", [True, False])
@pytest.mark.parametrize("L", [4, 8, 12, 2044, 2048, 8188, 8192, 8196, 16384, 24580])
def test_scan_vector_accesses_cover_each_row_once(fwd, L):
    """Rows with L % 4 == 0: every thread whose eight elements lie inside the
    row moves them as two aligned 16-byte accesses at i0 and i0 + 4, element e
    (scan order) sitting at i0 + at(e), the same position the scalar path uses;
    the rest use the scalar path.  Together they touch every position of the
    row exactly once, and nothing outside it."""
    threads, per = 1024, 8
    seen = [0] * L
    for seg in range(0, L, threads * per):
        for t in range(threads):
            p0 = seg + t * per
            whole = p0 + per <= L
            i0 = p0 if fwd else L - per - p0
            for e in range(per):
                p = p0 + e
                pos = p if fwd else L - 1 - p
                if whole:
                    at = e if fwd else per - 1 - e
                    assert i0 % 4 == 0 and 0 <= i0 and i0 + per <= L
                    assert i0 + at == pos
                    seen[i0 + at] += 1
                elif p < L:
                    seen[pos] += 1
    assert all(n == 1 for n in seen)


def test_delta_rows_model():
    """Delta kernel: LPR lanes share a row and a lane group takes kDeltaRows rows
    one workgroup pass apart; every row of every grid is reduced by exactly one
    lane group, and the clamped loads stay inside the tensor."""
    assert _const(BWD, "kDeltaRows") == "4"
    assert ("const size_t row0 = (size_t)blockIdx.x * (RPP * kDeltaRows) + threadIdx.x / LPR;"
            in BWD)
    assert "const size_t row = min(row0 + (size_t)r * RPP, rows - 1);" in BWD
    assert "const size_t per_block = (size_t)(256 / lpr) * kDeltaRows;" in BWD
    for lpr in (8, 16, 32):          # bf16 d = 64, 128; fp32 d = 128
        rpp = 256 // lpr
        for rows in (1, 5, rpp * 4 - 1, rpp * 4, rpp * 4 + 1, 1000, 4099):
            per_block = rpp * 4
            blocks = (rows + per_block - 1) // per_block
            done = [0] * rows
            for b in range(blocks):
                for sub in range(rpp):
                    row0 = b * per_block + sub
                    for r in range(4):
                        row = row0 + r * rpp
                        assert min(row, rows - 1) < rows
                        if row < rows:
                            done[row] += 1
            assert all(n == 1 for n in done)


def test_projection_backward_block_mapping():
    """gate_proj_bwd_kernel: the first n_dw workgroups are the dw_f blocks, the
    rest the dx blocks; each kind's block k covers (column block k % mblocks,
    token block k / mblocks) once."""
    proj = _src("gate_proj.hip")
    assert "const bool is_dx = i >= n_dw;  // the dw_f blocks first" in proj
    assert "const int k = is_dx ? i - n_dw : i;" in proj
    assert ("if (is_dx) proj_dx_body<BF16, HB>(sm.dx, k % mblocks, k / mblocks, w, g, dx, N, L, H, M);"
            in proj)
    assert "const dim3 grid((unsigned)(n_dx + n_dw));" in proj
    for mblocks, n_tok_dx, chunks, with_dx in ((16, 256, 64, True), (6, 128, 171, True),
                                               (1, 1, 1, True), (16, 256, 64, False)):
        n_dx = mblocks * n_tok_dx if with_dx else 0
        n_dw = mblocks * chunks
        seen = {True: set(), False: set()}
        for i in range(n_dx + n_dw):
            is_dx = i >= n_dw
            k = i - n_dw if is_dx else i
            cell = (k % mblocks, k // mblocks)
            assert cell not in seen[is_dx]
            seen[is_dx].add(cell)
        assert seen[True] == {(m, t) for m in range(mblocks) for t in range(n_tok_dx)} if with_dx \
            else not seen[True]
        assert seen[False] == {(m, c) for m in range(mblocks) for c in range(chunks)}

"""The C ABI on the host: the library loads, exports every declared entry point,
and rejects bad arguments before touching the GPU (no device needed)."""
import ctypes
import os
import re

import pytest
import torch

import paper_2503_02130_amd as fox

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fox.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fox.LIB_PATH):
        from paper_2503_02130_amd import build
        build.build()
    return fox.load()


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fox_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_symbols()
    for n in ("fox_gate_prefix", "fox_attn_fwd", "fox_attn_bwd", "fox_attn_decode",
              "fox_attn_bwd_workspace_bytes", "fox_attn_decode_workspace_bytes",
              "fox_status_string", "fox_version"):
        assert n in names


def test_header_compiles_as_c_and_cpp(tmp_path):
    """fox.h is self-contained for C (C99) and C++ consumers, its enums are
    int-sized, and the prototypes use the boundary's own types: fox_status_t
    results, fox_dtype_t dtypes and hipStream_t streams."""
    import shutil
    import subprocess
    src = tmp_path / "use_fox.c"
    src.write_text(
        '#include "fox.h"\n'
        "typedef char status_is_int[sizeof(fox_status_t) == sizeof(int) ? 1 : -1];\n"
        "typedef char dtype_is_int[sizeof(fox_dtype_t) == sizeof(int) ? 1 : -1];\n"
        "static fox_status_t (*fwd)(fox_dtype_t, const void*, const void*, const void*,\n"
        "    const float*, void*, float*, int, int, int, int, float, hipStream_t) = fox_attn_fwd;\n"
        "static fox_status_t (*bwd)(fox_dtype_t, const void*, const void*, const void*,\n"
        "    const float*, const void*, const float*, const void*, void*, void*, void*, float*,\n"
        "    void*, size_t, int, int, int, int, float, hipStream_t) = fox_attn_bwd;\n"
        "int main(void) { return (fwd && bwd) ? (int)FOX_OK : 1; }\n")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           "-D__HIP_PLATFORM_AMD__"]
    for cc, std, lang in (("gcc", "-std=c99", "c"), ("g++", "-std=c++17", "c++")):
        if shutil.which(cc) is None:
            pytest.skip(f"{cc} not available")
        r = subprocess.run([cc, std, "-x", lang, "-Wall", "-Werror", "-fsyntax-only", *inc,
                            str(src)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
    text = open(HEADER).read()
    assert "void* stream" not in text and "int dtype" not in text
    assert re.search(r"fox_status_t fox_attn_bwd\(fox_dtype_t dtype", text)


def test_every_declared_symbol_is_exported(lib):
    for n in declared_symbols():
        assert hasattr(lib, n), f"{n} is declared in fox.h but not exported"
    assert set(fox.EXPORTED) == set(declared_symbols())


def test_status_strings(lib):
    for code in range(9):
        assert lib.fox_status_string(code) and b"unknown" not in lib.fox_status_string(code)
    assert b"unknown" in lib.fox_status_string(99)
    assert lib.fox_version() >= 100


P16 = 0x10000  # a 16-byte aligned fake address: never dereferenced by these calls


def _fwd(lib, dtype=1, ptrs=(P16,) * 6, B=1, H=1, L=8, d=64):
    return lib.fox_attn_fwd(dtype, *[ctypes.c_void_p(p) if p else None for p in ptrs],
                            B, H, L, d, ctypes.c_float(0.125), None)


def test_fwd_validation(lib):
    assert _fwd(lib, ptrs=(0,) + (P16,) * 5) == 1                      # NULL
    assert _fwd(lib, B=0) == 2 and _fwd(lib, L=-3) == 2                # shape
    assert _fwd(lib, B=1 << 20, H=1 << 12, L=1 << 16) == 2             # overflow
    assert _fwd(lib, d=96) == 3 and _fwd(lib, dtype=5) == 3            # unsupported
    assert _fwd(lib, ptrs=(P16 + 2,) + (P16,) * 5) == 4                # alignment


def test_gate_prefix_validation(lib):
    c = ctypes.c_void_p
    assert lib.fox_gate_prefix(None, None, c(P16), 1, 1, 4, None) == 1
    assert lib.fox_gate_prefix(c(P16), None, c(P16), 1, 0, 4, None) == 2
    assert lib.fox_gate_prefix(c(P16), c(P16 + 4), c(P16), 1, 1, 4, None) == 4


def test_gate_projection_validation(lib):
    c = ctypes.c_void_p
    fwd = lib.fox_gate_projection
    assert fwd(1, None, c(P16), None, c(P16), 1, 4, 2, 64, None) == 1
    assert fwd(1, c(P16), c(P16), None, c(P16), 1, 0, 2, 64, None) == 2
    assert fwd(2, c(P16), c(P16), None, c(P16), 1, 4, 2, 64, None) == 3   # dtype
    assert fwd(1, c(P16), c(P16), None, c(P16), 1, 4, 65, 64, None) == 3  # H > 64
    assert fwd(1, c(P16), c(P16), None, c(P16), 1, 4, 2, 60, None) == 3   # M % 8
    assert fwd(1, c(P16 + 4), c(P16), None, c(P16), 1, 4, 2, 64, None) == 4
    ws = lib.fox_gate_projection_bwd_workspace_bytes
    assert ws(1, 1, 4, 65, 64) == 0 and ws(1, 1, 4, 2, 60) == 0
    # per chunk of tokens (at least 256 per 32 heads): dw_f and db_f partials, chunks * H * (M + 1) * 4
    assert ws(1, 1, 4, 2, 64) == 1 * 2 * 65 * 4
    assert ws(1, 2, 16384, 16, 2048) == 64 * 16 * 2049 * 4
    assert ws(0, 8, 2048, 12, 768) == 64 * 12 * 769 * 4
    bwd = lib.fox_gate_projection_bwd
    args = lambda wsp, wsb, dw=c(P16): (1, c(P16), c(P16), c(P16), None, dw, None, wsp, wsb,
                                        1, 4, 2, 64, None)
    assert bwd(*args(c(P16), 1 << 20, dw=None)) == 1
    assert bwd(*args(None, 1 << 20)) == 5
    assert bwd(*args(c(P16), 2 * 65 * 4 - 1)) == 5
    assert bwd(*args(c(P16 + 8), 1 << 20)) == 4


def test_dlogit_validation(lib):
    c = ctypes.c_void_p
    ok = [c(P16), c(P16), c(P16), None, c(P16)]
    assert lib.fox_dlogit_from_dc(c(P16), c(P16), None, None, c(P16), 1, 1, 4, None) == 1
    assert lib.fox_dlogit_from_dc(c(P16), c(P16), c(P16), c(P16), None, 1, 1, 4, None) == 1
    assert lib.fox_dlogit_from_dc(*ok, 1, 1, 0, None) == 2
    assert lib.fox_dlogit_from_dc(c(P16), c(P16), c(P16), c(P16 + 8), c(P16), 1, 1, 4, None) == 4
    assert lib.fox_dlogit_from_dc(c(P16), c(P16), c(P16 + 4), None, c(P16), 1, 1, 4, None) == 4


def test_fixed_gate_init_host(lib):
    """The host-side initialisation: the paper's worked example and argument checks."""
    import oracle
    b = fox.fox_fixed_gate_init(4, 2.0, 128.0)
    assert torch.allclose(b.double(), oracle.fixed_gate_bias_init(4, 2.0, 128.0), atol=1e-6)
    assert torch.allclose(oracle.time_constant(b.double()),
                          torch.tensor([2.0, 8.0, 32.0, 128.0], dtype=torch.float64), rtol=1e-5)
    buf = (ctypes.c_float * 4)()
    assert lib.fox_fixed_gate_init(None, 4, ctypes.c_float(2), ctypes.c_float(128)) == 1
    assert lib.fox_fixed_gate_init(buf, 0, ctypes.c_float(2), ctypes.c_float(128)) == 2
    assert lib.fox_fixed_gate_init(buf, 4, ctypes.c_float(0), ctypes.c_float(128)) == 2
    assert lib.fox_fixed_gate_init(buf, 4, ctypes.c_float(8), ctypes.c_float(2)) == 2


def test_fixed_gate_validation(lib):
    c = ctypes.c_void_p
    f = ctypes.c_float(0.1)
    assert lib.fox_attn_fwd_fixed_gate(1, c(P16), c(P16), c(P16), None, c(P16), c(P16),
                                       1, 2, 8, 64, f, None) == 1
    assert lib.fox_attn_fwd_fixed_gate(1, c(P16), c(P16), c(P16), c(P16 + 4), c(P16), c(P16),
                                       1, 2, 8, 64, f, None) == 4
    assert lib.fox_attn_fwd_fixed_gate(1, *[c(P16)] * 6, 1, 2, 8, 96, f, None) == 3
    need = lib.fox_attn_bwd_fixed_gate_workspace_bytes(1, 2, 3, 100, 64)
    assert need == 4 * 4 * 2 * 3 * 100
    args = [c(P16)] * 10
    assert lib.fox_attn_bwd_fixed_gate(1, *args, None, c(P16), need - 1, 2, 3, 100, 64, f,
                                       None) == 5
    dneed = lib.fox_attn_decode_workspace_bytes(1, 2, 3, 100, 64)
    assert lib.fox_attn_decode_fixed_gate(1, *[c(P16)] * 6, c(P16), dneed - 1, 2, 3, 100, 64, f,
                                          None) == 5


def test_skip_validation(lib):
    c = ctypes.c_void_p
    f = ctypes.c_float(0.1)
    assert lib.fox_row_norm_max(1, None, c(P16), 1, 2, 8, 64, None) == 1
    assert lib.fox_row_norm_max(1, c(P16), c(P16 + 4), 1, 2, 8, 64, None) == 4
    assert lib.fox_row_norm_max(1, c(P16), c(P16), 1, 2, 8, 80, None) == 3
    need = lib.fox_attn_decode_workspace_bytes(1, 2, 3, 100, 64)
    args = [c(P16)] * 9
    assert lib.fox_attn_decode_skip(1, *args[:6], None, c(P16), c(P16), need, 2, 3, 100, 64, f,
                                    None) == 1
    assert lib.fox_attn_decode_skip(1, *args, need - 1, 2, 3, 100, 64, f, None) == 5
    assert lib.fox_attn_decode_skip(1, *args, need, 2, 3, 0, 64, f, None) == 2


def test_pro_validation_and_workspace(lib):
    """FoX (Pro) entry points: NULLs, eps range, alignment, head dim, workspace."""
    c = ctypes.c_void_p
    f = ctypes.c_float
    B, H, L, d = 2, 3, 600, 128
    ok = [c(P16)] * 7
    out = [c(P16)] * 3
    assert lib.fox_pro_prologue(1, None, *ok[1:], f(1e-6), *out, B, H, L, d, None) == 1
    assert lib.fox_pro_prologue(1, *ok, f(-1.0), *out, B, H, L, d, None) == 7
    assert lib.fox_pro_prologue(1, *ok, f(float("inf")), *out, B, H, L, d, None) == 7
    assert lib.fox_pro_prologue(1, *ok, f(float("nan")), *out, B, H, L, d, None) == 7
    assert lib.fox_pro_prologue(1, *ok[:5], c(P16 + 4), ok[6], f(0.0), *out, B, H, L, d, None) == 4
    assert lib.fox_pro_prologue(1, *ok, f(0.0), *out, B, H, L, 96, None) == 3
    need = lib.fox_pro_prologue_bwd_workspace_bytes(1, B, H, L, d)
    assert need == 2 * B * H * 3 * d * 4          # 3 chunks of 256 rows
    assert lib.fox_pro_prologue_bwd_workspace_bytes(1, B, H, L, 80) == 0
    grads = [c(P16)] * 10
    assert lib.fox_pro_prologue_bwd(1, *ok, f(1e-6), *grads, c(P16), need - 1, B, H, L, d,
                                    None) == 5
    assert lib.fox_pro_prologue_bwd(1, *ok, f(1e-6), *grads, None, need, B, H, L, d, None) == 5
    assert lib.fox_pro_prologue_bwd(1, *ok, f(-2.0), *grads, c(P16), need, B, H, L, d, None) == 7
    assert lib.fox_pro_output_gate(1, c(P16), None, c(P16), f(1e-6), c(P16), B, H, L, d,
                                   None) == 1
    assert lib.fox_pro_output_gate(1, c(P16), c(P16), c(P16), f(-1e-3), c(P16), B, H, L, d,
                                   None) == 7
    assert lib.fox_attn_fwd_pro(1, *[c(P16)] * 6, f(float("nan")), c(P16), c(P16), c(P16),
                                B, H, L, d, f(0.1), None) == 7
    assert lib.fox_attn_fwd_pro(1, *[c(P16)] * 6, f(1e-6), c(P16), c(P16 + 8), c(P16),
                                B, H, L, d, f(0.1), None) == 4
    bneed = lib.fox_attn_bwd_pro_workspace_bytes(1, B, H, L, d)
    base = lambda x: (x + 255) // 256 * 256
    assert bneed == base(3 * 4 * B * H * L) + base(B * H * L * d * 2) + B * H * 3 * d * 4
    assert lib.fox_attn_bwd_pro_workspace_bytes(0, B, H, L, d) == \
        base(3 * 4 * B * H * L) + base(B * H * L * d * 4) + B * H * 3 * d * 4
    args = [c(P16)] * 8
    grads = [c(P16)] * 7
    assert lib.fox_attn_bwd_pro(1, *args, f(1e-6), *grads, c(P16), bneed - 1, B, H, L, d, f(0.1),
                                None) == 5
    assert lib.fox_attn_bwd_pro(1, *args, f(-1.0), *grads, c(P16), bneed, B, H, L, d, f(0.1),
                                None) == 7
    sneed = lib.fox_attn_bwd_pro_stored_workspace_bytes(1, B, H, L, d)
    assert sneed == base(bneed) + lib.fox_attn_bwd_ds_store_bytes(1, B, H, L, d)
    assert lib.fox_attn_bwd_pro_stored_workspace_bytes(0, B, H, L, d) == 0
    assert lib.fox_attn_bwd_pro_stored(1, *args, f(1e-6), *grads, c(P16), sneed - 1, B, H, L, d,
                                       f(0.1), None) == 5
    assert lib.fox_attn_bwd_pro_stored(0, *args, f(1e-6), *grads, c(P16), sneed, B, H, L, d,
                                       f(0.1), None) == 3
    assert lib.fox_attn_bwd_pro_stored(1, *args, f(-1.0), *grads, c(P16), sneed, B, H, L, d,
                                       f(0.1), None) == 7


def test_fixed_gate_skip_validation(lib):
    c = ctypes.c_void_p
    f = ctypes.c_float(0.1)
    B, H, L, d = 1, 2, 8, 64
    assert lib.fox_attn_fwd_fixed_gate_skip(1, *[c(P16)] * 4, None, c(P16), c(P16), c(P16),
                                            B, H, L, d, f, None) == 1
    assert lib.fox_attn_fwd_fixed_gate_skip(1, *[c(P16)] * 5, c(P16 + 4), c(P16), c(P16),
                                            B, H, L, d, f, None) == 4
    need = lib.fox_attn_bwd_fixed_gate_workspace_bytes(1, B, H, L, d)
    args = [c(P16)] * 12
    assert lib.fox_attn_bwd_fixed_gate_skip(1, *args, None, c(P16), need - 1, B, H, L, d, f,
                                            None) == 5
    assert lib.fox_attn_bwd_fixed_gate_skip(1, *args[:7], None, *args[8:], None, c(P16), need,
                                            B, H, L, d, f, None) == 1
    dneed = lib.fox_attn_decode_workspace_bytes(1, B, H, 100, d)
    assert lib.fox_attn_decode_fixed_gate_skip(1, *[c(P16)] * 4, None, c(P16), c(P16), c(P16),
                                               dneed, B, H, 100, d, f, None) == 1
    assert lib.fox_attn_decode_fixed_gate_skip(1, *[c(P16)] * 7, c(P16), dneed - 1, B, H, 100, d,
                                               f, None) == 5


def test_bwd_validation_and_workspace(lib):
    c = ctypes.c_void_p
    B, H, L, d = 2, 3, 100, 128
    need = lib.fox_attn_bwd_workspace_bytes(1, B, H, L, d)
    assert need == 3 * 4 * B * H * L
    assert lib.fox_attn_bwd_workspace_bytes(1, B, H, L, 80) == 0
    args = [c(P16)] * 11
    assert lib.fox_attn_bwd(1, *args, c(P16), need - 1, B, H, L, d, ctypes.c_float(0.1), None) == 5
    assert lib.fox_attn_bwd(1, *args, None, need, B, H, L, d, ctypes.c_float(0.1), None) == 5
    assert lib.fox_attn_bwd(1, *args[:-1], None, c(P16), need, B, H, L, d,
                            ctypes.c_float(0.1), None) == 1


def test_bwd_stored_validation_and_workspace(lib):
    """The backward that keeps dS: workspace = the recompute path's, aligned to
    256 bytes, plus 16 KB per causal (128-key block, 64-query tile) pair and
    head, plus a tile count per (head, key block); bf16 only."""
    c = ctypes.c_void_p
    f = ctypes.c_float(0.1)
    base = lambda x: (x + 255) // 256 * 256
    for B, H, L in ((2, 3, 100), (1, 1, 1), (1, 2, 64), (1, 2, 128), (2, 1, 129),
                    (1, 1, 1000), (2, 16, 16384)):
        nq, nk = -(-L // 64), -(-L // 128)
        pairs = sum(1 for nb in range(nk) for qt in range(nq) if qt >= 2 * nb)
        for d in (64, 128):
            tail = B * H * pairs * 16384 + B * H * nk * 4
            assert lib.fox_attn_bwd_stored_workspace_bytes(1, B, H, L, d) == \
                base(3 * 4 * B * H * L) + tail, (B, H, L, d)
            assert lib.fox_attn_bwd_fixed_gate_stored_workspace_bytes(1, B, H, L, d) == \
                base(4 * 4 * B * H * L) + tail, (B, H, L, d)
            assert lib.fox_attn_bwd_ds_store_bytes(1, B, H, L, d) == B * H * pairs * 16384
    assert lib.fox_attn_bwd_stored_workspace_bytes(1, 2, 16, 16384, 128) == \
        base(12 * 32 * 16384) + 32 * 16512 * 16384 + 32 * 128 * 4  # 8.66 GB at 16k
    B, H, L, d = 2, 3, 100, 128
    assert lib.fox_attn_bwd_stored_workspace_bytes(0, B, H, L, d) == 0  # fp32
    assert lib.fox_attn_bwd_stored_workspace_bytes(1, B, H, L, 80) == 0
    need = lib.fox_attn_bwd_stored_workspace_bytes(1, B, H, L, d)
    args = [c(P16)] * 11
    assert lib.fox_attn_bwd_stored(0, *args, c(P16), need, B, H, L, d, f, None) == 3
    assert lib.fox_attn_bwd_stored(1, *args, c(P16), need - 1, B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_stored(1, *args, None, need, B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_stored(1, *args, c(P16 + 4), need, B, H, L, d, f, None) == 4
    assert lib.fox_attn_bwd_stored(1, *args[:-1], None, c(P16), need, B, H, L, d, f, None) == 1
    assert lib.fox_attn_bwd_stored(1, *args, c(P16), need, B, H, 0, d, f, None) == 2
    store = lib.fox_attn_bwd_ds_store_bytes(1, B, H, L, d)
    assert store == need - base(3 * 4 * B * H * L) - B * H * 1 * 4
    assert lib.fox_attn_bwd_ds_store_bytes(0, B, H, L, d) == 0
    kv = [c(P16)] * 10
    assert lib.fox_attn_bwd_dkdv_store(1, *kv, c(P16), store - 1, B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_dkdv_store(1, *kv, None, store, B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_dkdv_store(0, *kv, c(P16), store, B, H, L, d, f, None) == 3
    assert lib.fox_attn_bwd_dkdv_store(1, None, *kv[1:], c(P16), store, B, H, L, d, f, None) == 1
    assert lib.fox_attn_bwd_dq_stored(1, c(P16), c(P16), store - 1, c(P16), c(P16), B, H, L, d, f,
                                      None) == 5
    assert lib.fox_attn_bwd_dq_stored(1, c(P16), None, store, c(P16), c(P16), B, H, L, d, f,
                                      None) == 5
    assert lib.fox_attn_bwd_dq_stored(1, c(P16), c(P16 + 2), store, c(P16), c(P16), B, H, L, d,
                                      f, None) == 4
    assert lib.fox_attn_bwd_dq_stored(0, c(P16), c(P16), store, c(P16), c(P16), B, H, L, d, f,
                                      None) == 3
    assert lib.fox_attn_bwd_dq_stored(1, c(P16), c(P16), store, None, c(P16), B, H, L, d, f,
                                      None) == 1
    # skipping, fixed gates and both: the same checks
    nm = [c(P16)] * 2
    a7 = [c(P16)] * 7
    g4 = [c(P16)] * 4
    assert lib.fox_attn_bwd_skip_stored(1, *a7, *nm, *g4, c(P16), need - 1, B, H, L, d, f,
                                        None) == 5
    assert lib.fox_attn_bwd_skip_stored(0, *a7, *nm, *g4, c(P16), need, B, H, L, d, f, None) == 3
    assert lib.fox_attn_bwd_skip_stored(1, *a7, None, c(P16), *g4, c(P16), need, B, H, L, d, f,
                                        None) == 1
    fneed = lib.fox_attn_bwd_fixed_gate_stored_workspace_bytes(1, B, H, L, d)
    assert lib.fox_attn_bwd_fixed_gate_stored_workspace_bytes(0, B, H, L, d) == 0
    assert lib.fox_attn_bwd_fixed_gate_stored(1, *a7, *[c(P16)] * 3, c(P16), c(P16), fneed - 1,
                                              B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_fixed_gate_stored(0, *a7, *[c(P16)] * 3, c(P16), c(P16), fneed,
                                              B, H, L, d, f, None) == 3
    assert lib.fox_attn_bwd_fixed_gate_stored(1, *a7, *[c(P16)] * 3, c(P16 + 4), c(P16), fneed,
                                              B, H, L, d, f, None) == 4
    assert lib.fox_attn_bwd_fixed_gate_skip_stored(1, *a7, *nm, *[c(P16)] * 3, c(P16), c(P16),
                                                   fneed - 1, B, H, L, d, f, None) == 5
    assert lib.fox_attn_bwd_fixed_gate_skip_stored(1, *a7, c(P16), None, *[c(P16)] * 3, c(P16),
                                                   c(P16), fneed, B, H, L, d, f, None) == 1


def test_decode_validation_and_workspace(lib):
    c = ctypes.c_void_p
    need = lib.fox_attn_decode_workspace_bytes(1, 64, 16, 32768, 128)
    assert need > 0 and need % (4 * 130) == 0
    assert lib.fox_attn_decode_workspace_bytes(1, 64, 16, 32768, 32) == 0
    args = [c(P16)] * 7
    assert lib.fox_attn_decode(1, *args, c(P16), need - 4, 64, 16, 32768, 128,
                               ctypes.c_float(0.1), None) == 5
    assert lib.fox_attn_decode(1, *args, c(P16), need, 64, 16, 0, 128,
                               ctypes.c_float(0.1), None) == 2


def test_decode_noalloc_validation(lib):
    """The allocation-free decode checks its arguments like fox_attn_decode and
    refuses, before touching the GPU, shapes whose split partials exceed its
    64 MiB scratch (B*H = 1024, d = 128: T up to 129024 fits)."""
    def call(ptrs=(P16,) * 7, B=1, H=1, T=8, d=64, dtype=1):
        return lib.fox_attn_decode_noalloc(dtype, *[ctypes.c_void_p(p) if p else None
                                                    for p in ptrs],
                                           B, H, T, d, ctypes.c_float(0.125), None)
    assert call(ptrs=(0,) + (P16,) * 6) == 1
    assert call(B=0) == 2
    assert call(d=96) == 3
    assert call(ptrs=(P16 + 4,) + (P16,) * 6) == 4
    assert call(B=64, H=16, T=129025, d=128) == 8
    assert call(B=16, H=16, T=600000, d=128) == 8
    assert lib.fox_attn_decode_workspace_bytes(1, 64, 16, 129024, 128) <= 64 << 20
    assert lib.fox_attn_decode_workspace_bytes(1, 64, 16, 129025, 128) > 64 << 20
    assert b"TOO_LARGE" in lib.fox_status_string(8)


def test_binding_refuses_host_tensors(lib):
    """There is no CPU path: host tensors are rejected before any call."""
    x = torch.zeros(1, 1, 8)
    with pytest.raises(ValueError):
        fox.fox_gate_prefix(x)
    q = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        fox.fox_attn_fwd(q, q, q, x)


def test_single_hip_runtime(lib):
    """libfox.so binds to the HIP runtime torch already loaded (one copy)."""
    maps = [l.split()[-1] for l in open("/proc/self/maps") if "libamdhip64" in l]
    assert len(set(maps)) == 1, set(maps)

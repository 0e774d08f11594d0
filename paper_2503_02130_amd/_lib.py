"""ctypes binding of libfox.so: argument marshalling only.

Every function here validates torch tensors (device, dtype, shape, contiguity),
allocates missing outputs and workspaces with torch, and calls the C entry point
of the same name on the current HIP stream.  All arithmetic runs in the HIP
kernels; there is no host or PyTorch fallback: if the library is not built or
cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

import torch  # imported before libfox.so so that both share torch's HIP runtime

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfox.so")

FOX_DTYPE_F32 = 0
FOX_DTYPE_BF16 = 1
_DT = {torch.float32: FOX_DTYPE_F32, torch.bfloat16: FOX_DTYPE_BF16}

EXPORTED = (
    "fox_status_string", "fox_version", "fox_gate_prefix", "fox_attn_fwd",
    "fox_attn_bwd_workspace_bytes", "fox_attn_bwd", "fox_attn_bwd_delta", "fox_attn_bwd_dkdv",
    "fox_attn_bwd_dq", "fox_dlogf_from_dc", "fox_dlogit_from_dc",
    "fox_attn_decode_workspace_bytes", "fox_attn_decode", "fox_attn_decode_noalloc",
    "fox_fixed_gate_init", "fox_attn_fwd_fixed_gate", "fox_attn_bwd_fixed_gate_workspace_bytes",
    "fox_attn_bwd_fixed_gate", "fox_attn_decode_fixed_gate",
    "fox_row_norm_max", "fox_attn_decode_skip", "fox_attn_fwd_skip", "fox_attn_bwd_skip",
    "fox_attn_fwd_fixed_gate_skip", "fox_attn_bwd_fixed_gate_skip",
    "fox_attn_decode_fixed_gate_skip",
    "fox_pro_prologue", "fox_pro_prologue_bwd_workspace_bytes", "fox_pro_prologue_bwd",
    "fox_pro_output_gate", "fox_attn_fwd_pro", "fox_attn_bwd_pro_workspace_bytes",
    "fox_attn_bwd_pro", "fox_attn_bwd_stored_workspace_bytes", "fox_attn_bwd_stored",
    "fox_attn_bwd_ds_store_bytes", "fox_attn_bwd_dkdv_store", "fox_attn_bwd_dq_stored",
    "fox_attn_bwd_pro_stored_workspace_bytes", "fox_attn_bwd_pro_stored",
    "fox_attn_bwd_skip_stored", "fox_attn_bwd_fixed_gate_stored_workspace_bytes",
    "fox_attn_bwd_fixed_gate_stored", "fox_attn_bwd_fixed_gate_skip_stored",
    "fox_gate_projection", "fox_gate_projection_bwd_workspace_bytes", "fox_gate_projection_bwd",
)


class FoxError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what} failed with status {status}: {status_string(status)}")


_lib = None


def load() -> ctypes.CDLL:
    """Load libfox.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2503_02130_amd.build` "
            "(the HIP library is required; there is no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    # fox_status_t and fox_dtype_t are int-sized enums (their MAX_ENUM members) and
    # hipStream_t is a pointer, so c_int and c_void_p are their exact C types
    P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.fox_status_string.restype = ctypes.c_char_p
    lib.fox_status_string.argtypes = [I]
    lib.fox_version.restype = I
    lib.fox_version.argtypes = []
    lib.fox_gate_prefix.restype = I
    lib.fox_gate_prefix.argtypes = [P, P, P, I, I, I, P]
    lib.fox_attn_fwd.restype = I
    lib.fox_attn_fwd.argtypes = [I, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_workspace_bytes.restype = Z
    lib.fox_attn_bwd_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd.restype = I
    lib.fox_attn_bwd.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_attn_bwd_stored_workspace_bytes.restype = Z
    lib.fox_attn_bwd_stored_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd_stored.restype = I
    lib.fox_attn_bwd_stored.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_attn_bwd_ds_store_bytes.restype = Z
    lib.fox_attn_bwd_ds_store_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd_dkdv_store.restype = I
    lib.fox_attn_bwd_dkdv_store.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I, F,
                                            P]
    lib.fox_attn_bwd_dq_stored.restype = I
    lib.fox_attn_bwd_dq_stored.argtypes = [I, P, P, Z, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_delta.restype = I
    lib.fox_attn_bwd_delta.argtypes = [I, P, P, P, I, I, I, I, P]
    lib.fox_attn_bwd_dkdv.restype = I
    lib.fox_attn_bwd_dkdv.argtypes = [I, P, P, P, P, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_dq.restype = I
    lib.fox_attn_bwd_dq.argtypes = [I, P, P, P, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_dlogf_from_dc.restype = I
    lib.fox_dlogf_from_dc.argtypes = [P, P, P, I, I, I, P]
    lib.fox_dlogit_from_dc.restype = I
    lib.fox_dlogit_from_dc.argtypes = [P, P, P, P, P, I, I, I, P]
    lib.fox_attn_decode_workspace_bytes.restype = Z
    lib.fox_attn_decode_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_decode.restype = I
    lib.fox_attn_decode.argtypes = [I, P, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_attn_decode_noalloc.restype = I
    lib.fox_attn_decode_noalloc.argtypes = [I, P, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_fixed_gate_init.restype = I
    lib.fox_fixed_gate_init.argtypes = [P, I, F, F]
    lib.fox_attn_fwd_fixed_gate.restype = I
    lib.fox_attn_fwd_fixed_gate.argtypes = [I, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_fixed_gate_workspace_bytes.restype = Z
    lib.fox_attn_bwd_fixed_gate_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd_fixed_gate.restype = I
    lib.fox_attn_bwd_fixed_gate.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I,
                                            F, P]
    lib.fox_attn_decode_fixed_gate.restype = I
    lib.fox_attn_decode_fixed_gate.argtypes = [I, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_row_norm_max.restype = I
    lib.fox_row_norm_max.argtypes = [I, P, P, I, I, I, I, P]
    lib.fox_attn_fwd_skip.restype = I
    lib.fox_attn_fwd_skip.argtypes = [I, P, P, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_skip.restype = I
    lib.fox_attn_bwd_skip.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, P, P, P, Z, I, I, I, I,
                                      F, P]
    lib.fox_attn_decode_skip.restype = I
    lib.fox_attn_decode_skip.argtypes = [I, P, P, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_attn_fwd_fixed_gate_skip.restype = I
    lib.fox_attn_fwd_fixed_gate_skip.argtypes = [I, P, P, P, P, P, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_fixed_gate_skip.restype = I
    lib.fox_attn_bwd_fixed_gate_skip.argtypes = [I, P, P, P, P, P, P, P, P, P, P, P, P, P, P, Z,
                                                 I, I, I, I, F, P]
    for name, twin in (("fox_attn_bwd_skip_stored", "fox_attn_bwd_skip"),
                       ("fox_attn_bwd_fixed_gate_stored", "fox_attn_bwd_fixed_gate"),
                       ("fox_attn_bwd_fixed_gate_skip_stored", "fox_attn_bwd_fixed_gate_skip")):
        getattr(lib, name).restype = I
        getattr(lib, name).argtypes = getattr(lib, twin).argtypes
    lib.fox_attn_bwd_fixed_gate_stored_workspace_bytes.restype = Z
    lib.fox_attn_bwd_fixed_gate_stored_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_decode_fixed_gate_skip.restype = I
    lib.fox_attn_decode_fixed_gate_skip.argtypes = [I, P, P, P, P, P, P, P, P, Z, I, I, I, I, F, P]
    lib.fox_pro_prologue.restype = I
    lib.fox_pro_prologue.argtypes = [I, P, P, P, P, P, P, P, F, P, P, P, I, I, I, I, P]
    lib.fox_pro_prologue_bwd_workspace_bytes.restype = Z
    lib.fox_pro_prologue_bwd_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_pro_prologue_bwd.restype = I
    lib.fox_pro_prologue_bwd.argtypes = [I, P, P, P, P, P, P, P, F, P, P, P, P, P, P, P, P, P, P,
                                         P, Z, I, I, I, I, P]
    lib.fox_pro_output_gate.restype = I
    lib.fox_pro_output_gate.argtypes = [I, P, P, P, F, P, I, I, I, I, P]
    lib.fox_attn_fwd_pro.restype = I
    lib.fox_attn_fwd_pro.argtypes = [I, P, P, P, P, P, P, F, P, P, P, I, I, I, I, F, P]
    lib.fox_attn_bwd_pro_workspace_bytes.restype = Z
    lib.fox_attn_bwd_pro_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd_pro.restype = I
    lib.fox_attn_bwd_pro.argtypes = [I, P, P, P, P, P, P, P, P, F, P, P, P, P, P, P, P, P, Z, I, I,
                                     I, I, F, P]
    lib.fox_attn_bwd_pro_stored_workspace_bytes.restype = Z
    lib.fox_attn_bwd_pro_stored_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_attn_bwd_pro_stored.restype = I
    lib.fox_attn_bwd_pro_stored.argtypes = [I, P, P, P, P, P, P, P, P, F, P, P, P, P, P, P, P, P, Z, I, I,
                                     I, I, F, P]
    lib.fox_gate_projection.restype = I
    lib.fox_gate_projection.argtypes = [I, P, P, P, P, I, I, I, I, P]
    lib.fox_gate_projection_bwd_workspace_bytes.restype = Z
    lib.fox_gate_projection_bwd_workspace_bytes.argtypes = [I, I, I, I, I]
    lib.fox_gate_projection_bwd.restype = I
    lib.fox_gate_projection_bwd.argtypes = [I, P, P, P, P, P, P, P, Z, I, I, I, I, P]
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().fox_status_string(int(status)).decode()


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _check(t: torch.Tensor, name: str, shape, dtype, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device}); the library has no CPU path")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _raise(status: int, what: str):
    if status != 0:
        raise FoxError(status, what)


def default_scale(d: int) -> float:
    """The paper's 1/sqrt(d) scale on q.k."""
    return 1.0 / math.sqrt(d)


# ---------------------------------------------------------------------------
def fox_gate_prefix(gate_logit: torch.Tensor, c: Optional[torch.Tensor] = None,
                    log_f: Optional[torch.Tensor] = None, want_log_f: bool = False):
    """c = cumsum(log sigmoid(gate_logit)) over the last axis; [B, H, L] fp32.
    Returns c, or (c, log_f) when want_log_f or log_f is given."""
    B, H, L = gate_logit.shape
    _check(gate_logit, "gate_logit", (B, H, L), torch.float32, None)
    dev = gate_logit.device
    if c is None:
        c = torch.empty_like(gate_logit)
    _check(c, "c", (B, H, L), torch.float32, dev)
    if want_log_f and log_f is None:
        log_f = torch.empty_like(gate_logit)
    if log_f is not None:
        _check(log_f, "log_f", (B, H, L), torch.float32, dev)
    st = load().fox_gate_prefix(_ptr(gate_logit), _ptr(log_f), _ptr(c), B, H, L,
                                _stream(gate_logit))
    _raise(st, "fox_gate_prefix")
    return (c, log_f) if log_f is not None else c


def fox_attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, c: torch.Tensor,
                 scale: Optional[float] = None, o: Optional[torch.Tensor] = None,
                 lse: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """O [B,H,L,d] (q's dtype) and LSE [B,H,L] fp32."""
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, H, L), device=dev, dtype=torch.float32)
    _check(o, "o", (B, H, L, d), dt, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_fwd(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(o), _ptr(lse),
                             B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_fwd")
    return o, lse


def fox_attn_bwd_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int, d: int) -> int:
    return int(load().fox_attn_bwd_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_stored_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int,
                                        d: int) -> int:
    return int(load().fox_attn_bwd_stored_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd(q, k, v, c, o, lse, d_o, scale: Optional[float] = None,
                 dq=None, dk=None, dv=None, d_log_f=None, workspace=None):
    """dq, dk, dv [B,H,L,d] and d(log f) [B,H,L] fp32."""
    return _attn_bwd_call("fox_attn_bwd", fox_attn_bwd_workspace_bytes, q, k, v, c, o, lse, d_o,
                          scale, dq, dk, dv, d_log_f, workspace)


def fox_attn_bwd_stored(q, k, v, c, o, lse, d_o, scale: Optional[float] = None,
                        dq=None, dk=None, dv=None, d_log_f=None, workspace=None):
    """fox_attn_bwd keeping dS in the workspace (about B*H*L^2 bytes) instead of
    recomputing it for dQ; bf16 only."""
    return _attn_bwd_call("fox_attn_bwd_stored", fox_attn_bwd_stored_workspace_bytes, q, k, v,
                          c, o, lse, d_o, scale, dq, dk, dv, d_log_f, workspace)


def _attn_bwd_call(entry, ws_bytes, q, k, v, c, o, lse, d_o, scale, dq, dk, dv, d_log_f,
                   workspace):
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    d_log_f = torch.empty_like(c) if d_log_f is None else d_log_f
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(d_log_f, "d_log_f", (B, H, L), torch.float32, dev)
    need = ws_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = getattr(load(), entry)(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(o), _ptr(lse),
                                _ptr(d_o), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(d_log_f),
                                _ptr(workspace), workspace.numel() * workspace.element_size(),
                                B, H, L, d, s, _stream(q))
    _raise(st, entry)
    return dq, dk, dv, d_log_f


def _check_bwd_inputs(q, k, v, c, lse, d_o):
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("d_o", d_o)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    return B, H, L, d, dt, dev


def fox_attn_bwd_delta(o, d_o, delta=None):
    """delta_i = rowsum(dO o O), [B,H,L] fp32."""
    B, H, L, d = o.shape
    dt = o.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    _check(o, "o", (B, H, L, d), dt, None)
    _check(d_o, "d_o", (B, H, L, d), dt, o.device)
    delta = torch.empty((B, H, L), device=o.device, dtype=torch.float32) if delta is None else delta
    _check(delta, "delta", (B, H, L), torch.float32, o.device)
    st = load().fox_attn_bwd_delta(_DT[dt], _ptr(o), _ptr(d_o), _ptr(delta), B, H, L, d, _stream(o))
    _raise(st, "fox_attn_bwd_delta")
    return delta


def fox_attn_bwd_dkdv(q, k, v, c, lse, d_o, delta, scale: Optional[float] = None,
                      dk=None, dv=None, dc_k=None):
    """dK, dV (q's dtype) and dc_k = -colsum(dS) [B,H,L] fp32."""
    B, H, L, d, dt, dev = _check_bwd_inputs(q, k, v, c, lse, d_o)
    _check(delta, "delta", (B, H, L), torch.float32, dev)
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    dc_k = torch.empty_like(c) if dc_k is None else dc_k
    _check(dk, "dk", (B, H, L, d), dt, dev)
    _check(dv, "dv", (B, H, L, d), dt, dev)
    _check(dc_k, "dc_k", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_bwd_dkdv(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(lse),
                                  _ptr(d_o), _ptr(delta), _ptr(dk), _ptr(dv), _ptr(dc_k),
                                  B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_bwd_dkdv")
    return dk, dv, dc_k


def fox_attn_bwd_dq(q, k, v, c, lse, d_o, delta, scale: Optional[float] = None,
                    dq=None, dc_q=None):
    """dQ (q's dtype) and dc_q = rowsum(dS) [B,H,L] fp32."""
    B, H, L, d, dt, dev = _check_bwd_inputs(q, k, v, c, lse, d_o)
    _check(delta, "delta", (B, H, L), torch.float32, dev)
    dq = torch.empty_like(q) if dq is None else dq
    dc_q = torch.empty_like(c) if dc_q is None else dc_q
    _check(dq, "dq", (B, H, L, d), dt, dev)
    _check(dc_q, "dc_q", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_bwd_dq(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(lse),
                                _ptr(d_o), _ptr(delta), _ptr(dq), _ptr(dc_q), B, H, L, d, s,
                                _stream(q))
    _raise(st, "fox_attn_bwd_dq")
    return dq, dc_q


def fox_attn_bwd_ds_store_bytes(dtype: torch.dtype, B: int, H: int, L: int, d: int) -> int:
    return int(load().fox_attn_bwd_ds_store_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_dkdv_store(q, k, v, c, lse, d_o, delta, ds_store, scale: Optional[float] = None,
                            dk=None, dv=None, dc_k=None):
    """fox_attn_bwd_dkdv that also writes dS (bf16) into ds_store, a uint8
    device tensor of at least fox_attn_bwd_ds_store_bytes() bytes."""
    B, H, L, d, dt, dev = _check_bwd_inputs(q, k, v, c, lse, d_o)
    _check(delta, "delta", (B, H, L), torch.float32, dev)
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    dc_k = torch.empty_like(c) if dc_k is None else dc_k
    _check(dk, "dk", (B, H, L, d), dt, dev)
    _check(dv, "dv", (B, H, L, d), dt, dev)
    _check(dc_k, "dc_k", (B, H, L), torch.float32, dev)
    _check_store(ds_store, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_bwd_dkdv_store(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(lse),
                                        _ptr(d_o), _ptr(delta), _ptr(dk), _ptr(dv), _ptr(dc_k),
                                        _ptr(ds_store), ds_store.numel(), B, H, L, d, s,
                                        _stream(q))
    _raise(st, "fox_attn_bwd_dkdv_store")
    return dk, dv, dc_k


def fox_attn_bwd_dq_stored(k, ds_store, scale: Optional[float] = None, dq=None, dc_q=None):
    """dQ (k's dtype) and dc_q = rowsum(dS) [B,H,L] fp32 from the dS that
    fox_attn_bwd_dkdv_store wrote."""
    B, H, L, d = k.shape
    dt, dev = k.dtype, k.device
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    _check(k, "k", (B, H, L, d), dt, dev)
    _check_store(ds_store, dev)
    dq = torch.empty_like(k) if dq is None else dq
    dc_q = torch.empty((B, H, L), device=dev, dtype=torch.float32) if dc_q is None else dc_q
    _check(dq, "dq", (B, H, L, d), dt, dev)
    _check(dc_q, "dc_q", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_bwd_dq_stored(_DT[dt], _ptr(k), _ptr(ds_store), ds_store.numel(),
                                       _ptr(dq), _ptr(dc_q), B, H, L, d, s, _stream(k))
    _raise(st, "fox_attn_bwd_dq_stored")
    return dq, dc_q


def _check_store(ds_store, dev):
    if ds_store.dtype != torch.uint8 or ds_store.dim() != 1 or not ds_store.is_contiguous():
        raise ValueError("ds_store: a contiguous 1-D uint8 tensor")
    if ds_store.device != dev:
        raise ValueError(f"ds_store on {ds_store.device}, expected {dev}")


def fox_dlogf_from_dc(dc_q, dc_k, d_log_f=None):
    """d(log f)_l = sum_{i>=l} (dc_q + dc_k)_i, [B,H,L] fp32."""
    B, H, L = dc_q.shape
    _check(dc_q, "dc_q", (B, H, L), torch.float32, None)
    _check(dc_k, "dc_k", (B, H, L), torch.float32, dc_q.device)
    d_log_f = torch.empty_like(dc_q) if d_log_f is None else d_log_f
    _check(d_log_f, "d_log_f", (B, H, L), torch.float32, dc_q.device)
    st = load().fox_dlogf_from_dc(_ptr(dc_q), _ptr(dc_k), _ptr(d_log_f), B, H, L, _stream(dc_q))
    _raise(st, "fox_dlogf_from_dc")
    return d_log_f


def fox_dlogit_from_dc(dc_q, dc_k, gate_logit, d_logit=None, d_log_f=None):
    """d(logit) = d(log f) * sigmoid(-logit) with d(log f) the reverse cumsum of
    dc_q + dc_k, [B,H,L] fp32.  Returns d_logit, or (d_logit, d_log_f) when
    d_log_f is given."""
    B, H, L = dc_q.shape
    _check(dc_q, "dc_q", (B, H, L), torch.float32, None)
    _check(dc_k, "dc_k", (B, H, L), torch.float32, dc_q.device)
    _check(gate_logit, "gate_logit", (B, H, L), torch.float32, dc_q.device)
    d_logit = torch.empty_like(dc_q) if d_logit is None else d_logit
    _check(d_logit, "d_logit", (B, H, L), torch.float32, dc_q.device)
    if d_log_f is not None:
        _check(d_log_f, "d_log_f", (B, H, L), torch.float32, dc_q.device)
    st = load().fox_dlogit_from_dc(_ptr(dc_q), _ptr(dc_k), _ptr(gate_logit),
                                   _ptr(d_log_f) if d_log_f is not None else None, _ptr(d_logit),
                                   B, H, L, _stream(dc_q))
    _raise(st, "fox_dlogit_from_dc")
    return d_logit if d_log_f is None else (d_logit, d_log_f)


def fox_attn_decode_workspace_bytes(dtype: torch.dtype, B: int, H: int, T: int, d: int) -> int:
    return int(load().fox_attn_decode_workspace_bytes(_DT[dtype], B, H, T, d))


def fox_attn_decode(q, k_cache, v_cache, c_cache, gate_logit_new, scale: Optional[float] = None,
                    o=None, lse=None, workspace=None):
    """One decode step.  q [B,H,d]; caches [B,H,T,d] (slot T-1 = new token);
    c_cache [B,H,T] fp32 (entry T-1 is written); gate_logit_new [B,H] fp32.
    Returns o [B,H,d] and lse [B,H]."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    _check(q, "q", (B, H, d), dt, dev)
    _check(k_cache, "k_cache", (B, H, T, d), dt, dev)
    _check(v_cache, "v_cache", (B, H, T, d), dt, dev)
    _check(c_cache, "c_cache", (B, H, T), torch.float32, dev)
    _check(gate_logit_new, "gate_logit_new", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, d), dt, dev)
    _check(lse, "lse", (B, H), torch.float32, dev)
    need = fox_attn_decode_workspace_bytes(dt, B, H, T, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_decode(_DT[dt], _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(c_cache),
                                _ptr(gate_logit_new), _ptr(o), _ptr(lse), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), B, H, T, d, s,
                                _stream(q))
    _raise(st, "fox_attn_decode")
    return o, lse


def fox_attn_decode_noalloc(q, k_cache, v_cache, c_cache, gate_logit_new,
                            scale: Optional[float] = None, o=None, lse=None):
    """fox_attn_decode without a workspace (the library's per-device scratch
    array holds the split partials; shapes needing more than it holds raise).
    Pass o and lse to allocate nothing at all."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    _check(q, "q", (B, H, d), dt, dev)
    _check(k_cache, "k_cache", (B, H, T, d), dt, dev)
    _check(v_cache, "v_cache", (B, H, T, d), dt, dev)
    _check(c_cache, "c_cache", (B, H, T), torch.float32, dev)
    _check(gate_logit_new, "gate_logit_new", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, d), dt, dev)
    _check(lse, "lse", (B, H), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_decode_noalloc(_DT[dt], _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                        _ptr(c_cache), _ptr(gate_logit_new), _ptr(o), _ptr(lse),
                                        B, H, T, d, s, _stream(q))
    _raise(st, "fox_attn_decode_noalloc")
    return o, lse


# ---------------------------------------------------------------- fixed gates
def fox_fixed_gate_init(H: int, t_min: float, t_max: float) -> torch.Tensor:
    """Biases b [H] (host fp32) whose time constants T(b) = -1/log sigmoid(b)
    are log-spaced from t_min to t_max (the paper's fixed-gate initialisation)."""
    out = torch.empty(H, dtype=torch.float32)
    st = load().fox_fixed_gate_init(ctypes.c_void_p(out.data_ptr()), H, float(t_min), float(t_max))
    _raise(st, "fox_fixed_gate_init")
    return out


def fox_attn_fwd_fixed_gate(q, k, v, gate_bias, scale: Optional[float] = None, o=None, lse=None):
    """O, LSE with the fixed gate f_t^(h) = sigmoid(gate_bias[h]) (ALiBi form)."""
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, L), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, L, d), dt, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_fwd_fixed_gate(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(gate_bias),
                                        _ptr(o), _ptr(lse), B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_fwd_fixed_gate")
    return o, lse


def fox_attn_bwd_fixed_gate_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int,
                                            d: int) -> int:
    return int(load().fox_attn_bwd_fixed_gate_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_fixed_gate(q, k, v, gate_bias, o, lse, d_o, scale: Optional[float] = None,
                            dq=None, dk=None, dv=None, d_gate_bias=None, want_bias_grad=True,
                            workspace=None):
    """dq, dk, dv and d gate_bias [H] (None when want_bias_grad is False)."""
    return _bwd_fixed_call("fox_attn_bwd_fixed_gate", fox_attn_bwd_fixed_gate_workspace_bytes, q,
                           k, v, gate_bias, o, lse, d_o, scale, dq, dk, dv, d_gate_bias,
                           want_bias_grad, workspace)


def fox_attn_bwd_fixed_gate_stored_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int,
                                                   d: int) -> int:
    return int(load().fox_attn_bwd_fixed_gate_stored_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_fixed_gate_stored(q, k, v, gate_bias, o, lse, d_o, scale: Optional[float] = None,
                                   dq=None, dk=None, dv=None, d_gate_bias=None,
                                   want_bias_grad=True, workspace=None):
    """fox_attn_bwd_fixed_gate keeping dS (about B*H*L^2 bytes of workspace); bf16 only."""
    return _bwd_fixed_call("fox_attn_bwd_fixed_gate_stored",
                           fox_attn_bwd_fixed_gate_stored_workspace_bytes, q, k, v, gate_bias, o,
                           lse, d_o, scale, dq, dk, dv, d_gate_bias, want_bias_grad, workspace)


def _bwd_fixed_call(entry, ws_bytes, q, k, v, gate_bias, o, lse, d_o, scale, dq, dk, dv,
                    d_gate_bias, want_bias_grad, workspace):
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check(t, name, (B, H, L, d), dt, dev)
    if want_bias_grad:
        d_gate_bias = torch.empty_like(gate_bias) if d_gate_bias is None else d_gate_bias
        _check(d_gate_bias, "d_gate_bias", (H,), torch.float32, dev)
    else:
        d_gate_bias = None
    need = ws_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = getattr(load(), entry)(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(gate_bias), _ptr(o),
                                _ptr(lse), _ptr(d_o), _ptr(dq), _ptr(dk), _ptr(dv),
                                _ptr(d_gate_bias), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), B, H, L, d, s,
                                _stream(q))
    _raise(st, entry)
    return dq, dk, dv, d_gate_bias


def fox_attn_decode_fixed_gate(q, k_cache, v_cache, gate_bias, scale: Optional[float] = None,
                               o=None, lse=None, workspace=None):
    """One decode step with fixed gates (no prefix cache).  Returns o, lse."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    _check(q, "q", (B, H, d), dt, dev)
    _check(k_cache, "k_cache", (B, H, T, d), dt, dev)
    _check(v_cache, "v_cache", (B, H, T, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, d), dt, dev)
    _check(lse, "lse", (B, H), torch.float32, dev)
    need = fox_attn_decode_workspace_bytes(dt, B, H, T, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_decode_fixed_gate(_DT[dt], _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                           _ptr(gate_bias), _ptr(o), _ptr(lse), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(),
                                           B, H, T, d, s, _stream(q))
    _raise(st, "fox_attn_decode_fixed_gate")
    return o, lse


# ------------------------------------------------------- gate-aware skipping
def fox_row_norm_max(x, out=None):
    """max_t ||x[b,h,t,:]||_2 per (b, h) as fp32 [B,H] (an upper bound)."""
    B, H, L, d = x.shape
    if x.dtype not in _DT:
        raise ValueError(f"unsupported dtype {x.dtype}")
    _check(x, "x", (B, H, L, d), x.dtype, None)
    out = torch.empty((B, H), device=x.device, dtype=torch.float32) if out is None else out
    _check(out, "out", (B, H), torch.float32, x.device)
    st = load().fox_row_norm_max(_DT[x.dtype], _ptr(x), _ptr(out), B, H, L, d, _stream(x))
    _raise(st, "fox_row_norm_max")
    return out


def fox_attn_decode_skip(q, k_cache, v_cache, c_cache, gate_logit_new, k_norm_max,
                         scale: Optional[float] = None, o=None, lse=None, workspace=None):
    """fox_attn_decode with exact gate-aware skipping of key splits."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    _check(q, "q", (B, H, d), dt, dev)
    _check(k_cache, "k_cache", (B, H, T, d), dt, dev)
    _check(v_cache, "v_cache", (B, H, T, d), dt, dev)
    _check(c_cache, "c_cache", (B, H, T), torch.float32, dev)
    _check(gate_logit_new, "gate_logit_new", (B, H), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, d), dt, dev)
    _check(lse, "lse", (B, H), torch.float32, dev)
    need = fox_attn_decode_workspace_bytes(dt, B, H, T, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_decode_skip(_DT[dt], _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                     _ptr(c_cache), _ptr(gate_logit_new), _ptr(k_norm_max),
                                     _ptr(o), _ptr(lse), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(),
                                     B, H, T, d, s, _stream(q))
    _raise(st, "fox_attn_decode_skip")
    return o, lse


def fox_attn_fwd_skip(q, k, v, c, q_norm_max, k_norm_max, scale: Optional[float] = None,
                      o=None, lse=None):
    """fox_attn_fwd with exact gate-aware skipping of key tiles (bitwise equal)."""
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(q_norm_max, "q_norm_max", (B, H), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, L), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, L, d), dt, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_fwd_skip(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(q_norm_max),
                                  _ptr(k_norm_max), _ptr(o), _ptr(lse), B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_fwd_skip")
    return o, lse


def fox_attn_bwd_skip(q, k, v, c, o, lse, d_o, q_norm_max, k_norm_max,
                      scale: Optional[float] = None, dq=None, dk=None, dv=None, d_log_f=None,
                      workspace=None):
    """fox_attn_bwd with exact gate-aware skipping of tile pairs (bitwise equal)."""
    return _bwd_skip_call("fox_attn_bwd_skip", fox_attn_bwd_workspace_bytes, q, k, v, c, o, lse,
                          d_o, q_norm_max, k_norm_max, scale, dq, dk, dv, d_log_f, workspace)


def fox_attn_bwd_skip_stored(q, k, v, c, o, lse, d_o, q_norm_max, k_norm_max,
                             scale: Optional[float] = None, dq=None, dk=None, dv=None,
                             d_log_f=None, workspace=None):
    """fox_attn_bwd_stored with exact gate-aware skipping (bitwise equal to it)."""
    return _bwd_skip_call("fox_attn_bwd_skip_stored", fox_attn_bwd_stored_workspace_bytes, q, k,
                          v, c, o, lse, d_o, q_norm_max, k_norm_max, scale, dq, dk, dv, d_log_f,
                          workspace)


def _bwd_skip_call(entry, ws_bytes, q, k, v, c, o, lse, d_o, q_norm_max, k_norm_max, scale, dq,
                   dk, dv, d_log_f, workspace):
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    _check(q_norm_max, "q_norm_max", (B, H), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    d_log_f = torch.empty_like(c) if d_log_f is None else d_log_f
    for name, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(d_log_f, "d_log_f", (B, H, L), torch.float32, dev)
    need = ws_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = getattr(load(), entry)(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(o), _ptr(lse),
                                _ptr(d_o), _ptr(q_norm_max), _ptr(k_norm_max), _ptr(dq),
                                _ptr(dk), _ptr(dv), _ptr(d_log_f), _ptr(workspace),
                                workspace.numel() * workspace.element_size(),
                                B, H, L, d, s, _stream(q))
    _raise(st, entry)
    return dq, dk, dv, d_log_f



def fox_attn_fwd_fixed_gate_skip(q, k, v, gate_bias, q_norm_max, k_norm_max,
                                 scale: Optional[float] = None, o=None, lse=None):
    """fox_attn_fwd_fixed_gate with exact gate-aware skipping (bitwise the same O, LSE)."""
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    _check(q_norm_max, "q_norm_max", (B, H), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H, L), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, L, d), dt, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_fwd_fixed_gate_skip(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(gate_bias),
                                             _ptr(q_norm_max), _ptr(k_norm_max), _ptr(o),
                                             _ptr(lse), B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_fwd_fixed_gate_skip")
    return o, lse


def fox_attn_bwd_fixed_gate_skip(q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max,
                                 scale: Optional[float] = None, want_bias_grad=True,
                                 workspace=None):
    """fox_attn_bwd_fixed_gate with exact gate-aware skipping: dq, dk, dv, d gate_bias."""
    return _bwd_fixed_skip_call("fox_attn_bwd_fixed_gate_skip",
                                fox_attn_bwd_fixed_gate_workspace_bytes, q, k, v, gate_bias, o,
                                lse, d_o, q_norm_max, k_norm_max, scale, want_bias_grad,
                                workspace)


def fox_attn_bwd_fixed_gate_skip_stored(q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max,
                                        scale: Optional[float] = None, want_bias_grad=True,
                                        workspace=None):
    """fox_attn_bwd_fixed_gate_stored with exact gate-aware skipping (bitwise equal to it)."""
    return _bwd_fixed_skip_call("fox_attn_bwd_fixed_gate_skip_stored",
                                fox_attn_bwd_fixed_gate_stored_workspace_bytes, q, k, v,
                                gate_bias, o, lse, d_o, q_norm_max, k_norm_max, scale,
                                want_bias_grad, workspace)


def _bwd_fixed_skip_call(entry, ws_bytes, q, k, v, gate_bias, o, lse, d_o, q_norm_max,
                         k_norm_max, scale, want_bias_grad, workspace):
    B, H, L, d = q.shape
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    _check(q_norm_max, "q_norm_max", (B, H), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    db = torch.empty_like(gate_bias) if want_bias_grad else None
    need = ws_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = getattr(load(), entry)(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(gate_bias), _ptr(o),
                                _ptr(lse), _ptr(d_o), _ptr(q_norm_max), _ptr(k_norm_max),
                                _ptr(dq), _ptr(dk), _ptr(dv), _ptr(db), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), B, H, L, d, s,
                                _stream(q))
    _raise(st, entry)
    return dq, dk, dv, db


def fox_attn_decode_fixed_gate_skip(q, k_cache, v_cache, gate_bias, k_norm_max,
                                    scale: Optional[float] = None, o=None, lse=None,
                                    workspace=None):
    """fox_attn_decode_fixed_gate with exact skipping of key splits.  Returns o, lse."""
    B, H, d = q.shape
    T = k_cache.shape[2]
    dt = q.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    dev = q.device
    _check(q, "q", (B, H, d), dt, dev)
    _check(k_cache, "k_cache", (B, H, T, d), dt, dev)
    _check(v_cache, "v_cache", (B, H, T, d), dt, dev)
    _check(gate_bias, "gate_bias", (H,), torch.float32, dev)
    _check(k_norm_max, "k_norm_max", (B, H), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    lse = torch.empty((B, H), device=dev, dtype=torch.float32) if lse is None else lse
    need = fox_attn_decode_workspace_bytes(dt, B, H, T, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_decode_fixed_gate_skip(_DT[dt], _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                _ptr(gate_bias), _ptr(k_norm_max), _ptr(o),
                                                _ptr(lse), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(),
                                                B, H, T, d, s, _stream(q))
    _raise(st, "fox_attn_decode_fixed_gate_skip")
    return o, lse


# ---------------------------------------------------------------------------
# FoX (Pro) prologue and epilogue
# ---------------------------------------------------------------------------
def _pro_shapes(x, name="q_raw"):
    B, H, L, d = x.shape
    dt = x.dtype
    if dt not in _DT:
        raise ValueError(f"unsupported dtype {dt}")
    return B, H, L, d, dt, x.device


def fox_pro_prologue(q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                     k_norm_weight, eps: float = 1e-6, q=None, k=None, v=None):
    """q = RMSNorm(q_raw), k = RMSNorm(shift(k_raw)), v = shift(v_raw) (FoX Pro)."""
    B, H, L, d, dt, dev = _pro_shapes(q_raw)
    for name, t in (("q_raw", q_raw), ("k_raw", k_raw), ("v_raw", v_raw)):
        _check(t, name, (B, H, L, d), dt, dev)
    for name, t in (("k_shift_logit", k_shift_logit), ("v_shift_logit", v_shift_logit)):
        _check(t, name, (B, H, L), torch.float32, dev)
    for name, t in (("q_norm_weight", q_norm_weight), ("k_norm_weight", k_norm_weight)):
        _check(t, name, (H, d), torch.float32, dev)
    q = torch.empty_like(q_raw) if q is None else q
    k = torch.empty_like(k_raw) if k is None else k
    v = torch.empty_like(v_raw) if v is None else v
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, name, (B, H, L, d), dt, dev)
    st = load().fox_pro_prologue(_DT[dt], _ptr(q_raw), _ptr(k_raw), _ptr(v_raw),
                                 _ptr(k_shift_logit), _ptr(v_shift_logit), _ptr(q_norm_weight),
                                 _ptr(k_norm_weight), float(eps), _ptr(q), _ptr(k), _ptr(v),
                                 B, H, L, d, _stream(q_raw))
    _raise(st, "fox_pro_prologue")
    return q, k, v


def fox_pro_prologue_bwd_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int,
                                         d: int) -> int:
    return int(load().fox_pro_prologue_bwd_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_pro_prologue_bwd(q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                         k_norm_weight, dq, dk, dv, eps: float = 1e-6, workspace=None):
    """Gradients (dq_raw, dk_raw, dv_raw, dk_shift_logit, dv_shift_logit,
    dq_norm_weight, dk_norm_weight) of the prologue from dq, dk, dv."""
    B, H, L, d, dt, dev = _pro_shapes(q_raw)
    for name, t in (("q_raw", q_raw), ("k_raw", k_raw), ("v_raw", v_raw), ("dq", dq),
                    ("dk", dk), ("dv", dv)):
        _check(t, name, (B, H, L, d), dt, dev)
    for name, t in (("k_shift_logit", k_shift_logit), ("v_shift_logit", v_shift_logit)):
        _check(t, name, (B, H, L), torch.float32, dev)
    for name, t in (("q_norm_weight", q_norm_weight), ("k_norm_weight", k_norm_weight)):
        _check(t, name, (H, d), torch.float32, dev)
    dqr, dkr, dvr = (torch.empty_like(q_raw) for _ in range(3))
    dka, dva = torch.empty_like(k_shift_logit), torch.empty_like(v_shift_logit)
    dwq, dwk = torch.empty_like(q_norm_weight), torch.empty_like(k_norm_weight)
    need = fox_pro_prologue_bwd_workspace_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    st = load().fox_pro_prologue_bwd(_DT[dt], _ptr(q_raw), _ptr(k_raw), _ptr(v_raw),
                                     _ptr(k_shift_logit), _ptr(v_shift_logit),
                                     _ptr(q_norm_weight), _ptr(k_norm_weight), float(eps),
                                     _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dqr), _ptr(dkr),
                                     _ptr(dvr), _ptr(dka), _ptr(dva), _ptr(dwq), _ptr(dwk),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     B, H, L, d, _stream(q_raw))
    _raise(st, "fox_pro_prologue_bwd")
    return dqr, dkr, dvr, dka, dva, dwq, dwk


def fox_pro_output_gate(o, g_logit, o_norm_weight, eps: float = 1e-6, y=None):
    """y = RMSNorm(o) * sigmoid(g_logit)."""
    B, H, L, d, dt, dev = _pro_shapes(o)
    _check(g_logit, "g_logit", (B, H, L, d), dt, dev)
    _check(o_norm_weight, "o_norm_weight", (H, d), torch.float32, dev)
    y = torch.empty_like(o) if y is None else y
    _check(y, "y", (B, H, L, d), dt, dev)
    st = load().fox_pro_output_gate(_DT[dt], _ptr(o), _ptr(g_logit), _ptr(o_norm_weight),
                                    float(eps), _ptr(y), B, H, L, d, _stream(o))
    _raise(st, "fox_pro_output_gate")
    return y


def fox_attn_fwd_pro(q, k, v, c, g_logit, o_norm_weight, scale: Optional[float] = None,
                     eps: float = 1e-6, o=None, lse=None, y=None):
    """Attention with the output norm and gate: returns (y, o, lse)."""
    B, H, L, d, dt, dev = _pro_shapes(q)
    for name, t in (("q", q), ("k", k), ("v", v), ("g_logit", g_logit)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(o_norm_weight, "o_norm_weight", (H, d), torch.float32, dev)
    o = torch.empty_like(q) if o is None else o
    y = torch.empty_like(q) if y is None else y
    lse = torch.empty((B, H, L), device=dev, dtype=torch.float32) if lse is None else lse
    _check(o, "o", (B, H, L, d), dt, dev)
    _check(y, "y", (B, H, L, d), dt, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    s = default_scale(d) if scale is None else float(scale)
    st = load().fox_attn_fwd_pro(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(g_logit),
                                 _ptr(o_norm_weight), float(eps), _ptr(o), _ptr(lse), _ptr(y),
                                 B, H, L, d, s, _stream(q))
    _raise(st, "fox_attn_fwd_pro")
    return y, o, lse


def fox_attn_bwd_pro_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int, d: int) -> int:
    return int(load().fox_attn_bwd_pro_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_pro(q, k, v, c, o, lse, g_logit, o_norm_weight, dy,
                     scale: Optional[float] = None, eps: float = 1e-6, workspace=None):
    """Gradients of sum(y * dy): (dq, dk, dv, d_log_f, dg_logit, do_norm_weight)."""
    return _attn_bwd_pro_call("fox_attn_bwd_pro", fox_attn_bwd_pro_workspace_bytes, q, k, v, c,
                              o, lse, g_logit, o_norm_weight, dy, scale, eps, workspace)


def fox_attn_bwd_pro_stored_workspace_bytes(dtype: torch.dtype, B: int, H: int, L: int,
                                            d: int) -> int:
    return int(load().fox_attn_bwd_pro_stored_workspace_bytes(_DT[dtype], B, H, L, d))


def fox_attn_bwd_pro_stored(q, k, v, c, o, lse, g_logit, o_norm_weight, dy,
                            scale: Optional[float] = None, eps: float = 1e-6, workspace=None):
    """fox_attn_bwd_pro keeping dS in the workspace (about B*H*L^2 bytes); bf16 only."""
    return _attn_bwd_pro_call("fox_attn_bwd_pro_stored", fox_attn_bwd_pro_stored_workspace_bytes,
                              q, k, v, c, o, lse, g_logit, o_norm_weight, dy, scale, eps,
                              workspace)


def _attn_bwd_pro_call(entry, ws_bytes, q, k, v, c, o, lse, g_logit, o_norm_weight, dy, scale,
                       eps, workspace):
    B, H, L, d, dt, dev = _pro_shapes(q)
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o), ("g_logit", g_logit), ("dy", dy)):
        _check(t, name, (B, H, L, d), dt, dev)
    _check(c, "c", (B, H, L), torch.float32, dev)
    _check(lse, "lse", (B, H, L), torch.float32, dev)
    _check(o_norm_weight, "o_norm_weight", (H, d), torch.float32, dev)
    dq, dk, dv, dg = (torch.empty_like(q) for _ in range(4))
    dlf = torch.empty_like(c)
    dw = torch.empty_like(o_norm_weight)
    need = ws_bytes(dt, B, H, L, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), device=dev, dtype=torch.uint8)
    s = default_scale(d) if scale is None else float(scale)
    st = getattr(load(), entry)(_DT[dt], _ptr(q), _ptr(k), _ptr(v), _ptr(c), _ptr(o), _ptr(lse),
                                _ptr(g_logit), _ptr(o_norm_weight), float(eps), _ptr(dy),
                                _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dlf), _ptr(dg), _ptr(dw),
                                _ptr(workspace), workspace.numel() * workspace.element_size(),
                                B, H, L, d, s, _stream(q))
    _raise(st, entry)
    return dq, dk, dv, dlf, dg, dw


# ---------------------------------------------------------------------------
def _proj_shapes(x, w_f):
    if x.dim() != 3 or w_f.dim() != 2:
        raise ValueError("x must be [B, L, M] and w_f [H, M]")
    B, L, M = x.shape
    H = w_f.shape[0]
    if x.dtype not in _DT:
        raise ValueError(f"x must be float32 or bfloat16 (got {x.dtype})")
    _check(x, "x", (B, L, M), None, None)
    _check(w_f, "w_f", (H, M), torch.float32, x.device)
    return B, L, H, M


def fox_gate_projection(x, w_f, b_f=None, gate_logit=None):
    """Gate logits [B, H, L] fp32: gate_logit[b, h, t] = w_f[h] . x[b, t] + b_f[h]
    for x [B, L, M] (bf16 or fp32), w_f [H, M] and b_f [H] (optional) fp32."""
    B, L, H, M = _proj_shapes(x, w_f)
    if b_f is not None:
        _check(b_f, "b_f", (H,), torch.float32, x.device)
    if gate_logit is None:
        gate_logit = torch.empty((B, H, L), dtype=torch.float32, device=x.device)
    _check(gate_logit, "gate_logit", (B, H, L), torch.float32, x.device)
    st = load().fox_gate_projection(_DT[x.dtype], _ptr(x), _ptr(w_f), _ptr(b_f), _ptr(gate_logit),
                                    B, L, H, M, _stream(x))
    _raise(st, "fox_gate_projection")
    return gate_logit


def fox_gate_projection_bwd_workspace_bytes(dtype, B, L, H, M) -> int:
    return int(load().fox_gate_projection_bwd_workspace_bytes(_DT[dtype], B, L, H, M))


def fox_gate_projection_bwd(x, w_f, d_logit, want_dx=True, want_db=True, workspace=None,
                            dx=None, dw=None, db=None):
    """Gradients of sum(gate_logit * d_logit): returns (dx or None, dw_f, db_f or None).
    dx, dw, db: optional preallocated outputs (giving one implies wanting it)."""
    B, L, H, M = _proj_shapes(x, w_f)
    _check(d_logit, "d_logit", (B, H, L), torch.float32, x.device)
    if dx is None and want_dx:
        dx = torch.empty_like(x)
    if dx is not None:
        _check(dx, "dx", (B, L, M), x.dtype, x.device)
    if dw is None:
        dw = torch.empty((H, M), dtype=torch.float32, device=x.device)
    _check(dw, "dw", (H, M), torch.float32, x.device)
    if db is None and want_db:
        db = torch.empty((H,), dtype=torch.float32, device=x.device)
    if db is not None:
        _check(db, "db", (H,), torch.float32, x.device)
    need = fox_gate_projection_bwd_workspace_bytes(x.dtype, B, L, H, M)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=x.device)
    st = load().fox_gate_projection_bwd(_DT[x.dtype], _ptr(x), _ptr(w_f), _ptr(d_logit), _ptr(dx),
                                        _ptr(dw), _ptr(db), _ptr(workspace), workspace.numel(),
                                        B, L, H, M, _stream(x))
    _raise(st, "fox_gate_projection_bwd")
    return dx, dw, db

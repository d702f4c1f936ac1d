"""ctypes binding of libsata.so: argument marshalling only.

Every computation runs in the library's HIP kernels.  Torch is used for device
memory (output allocation) and for the current stream.  If the library has
not been built, loading fails with an error; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Tuple

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libsata.so")
HEADER_PATH = os.path.join(os.path.dirname(PKG_DIR), "include", "sata.h")

SATA_F32, SATA_BF16 = 0, 1
SATA_OK = 0

_lib = None


class SataError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        super().__init__(f"{func} failed with status {status}: {detail}")
        self.status = status


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libsata.so once and declares every signature of include/sata.h."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it first with __graft_entry__.build() "
                           "or python -m paper_2602_00294_amd.build")
    lib = ctypes.CDLL(p)
    i32, i64, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
    lib.sata_feature_count.argtypes = [i32, i32]
    lib.sata_feature_count.restype = i64
    lib.sata_state_elems.argtypes = [i32, i32, i32]
    lib.sata_state_elems.restype = i64
    lib.sata_feature_index.argtypes = [i32, i32, i64, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.sata_feature_index.restype = i32
    lib.sata_feature_map.argtypes = [vp, i32, i64, i32, i32, vp, vp]
    lib.sata_feature_map.restype = i32
    lib.sata_prefill.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp]
    lib.sata_prefill.restype = i32
    lib.sata_prefill_grouped.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp]
    lib.sata_prefill_grouped.restype = i32
    lib.sata_backward.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp]
    lib.sata_backward.restype = i32
    lib.sata_prefill_operands.argtypes = [i32, i32, i32, i32, i32, i32, i32, i32, ctypes.POINTER(i32)]
    lib.sata_prefill_operands.restype = i32
    lib.sata_prefill_parts.argtypes = [i32, i32, i32, i32, i32, i32, i32, i32, ctypes.POINTER(i32)]
    lib.sata_prefill_parts.restype = i32
    lib.sata_decode_step.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp]
    lib.sata_decode_step.restype = i32
    lib.sata_decode_step_noalloc.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp]
    lib.sata_decode_step_noalloc.restype = i32
    lib.sata_residual_elems.argtypes = [i32, i32, i32]
    lib.sata_residual_elems.restype = i64
    lib.sata_decode_step_compensated.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp]
    lib.sata_decode_step_compensated.restype = i32
    lib.sata_decode_step_grouped.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp, vp]
    lib.sata_decode_step_grouped.restype = i32
    lib.sata_status_string.argtypes = [i32]
    lib.sata_status_string.restype = ctypes.c_char_p
    lib.sata_last_error.argtypes = []
    lib.sata_last_error.restype = ctypes.c_char_p
    lib.sata_release.argtypes = []
    lib.sata_release.restype = None
    if path is None:
        _lib = lib
    return lib


def header_functions(path: str = HEADER_PATH):
    """Names of the functions that include/sata.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sata_[a-z_]+)\s*\(", text)))


def _check(status: int, func: str):
    if status != SATA_OK:
        detail = load_library().sata_last_error().decode()
        raise SataError(status, func, detail)


def feature_count(d: int, P: int) -> int:
    return int(load_library().sata_feature_count(d, P))


def state_elems(d_k: int, d_v: int, P: int) -> int:
    return int(load_library().sata_state_elems(d_k, d_v, P))


def feature_index(d: int, P: int, f: int) -> Tuple[int, ...]:
    """Index tuple (i1 <= ... <= ip) of feature f in the library's feature order."""
    deg = ctypes.c_int(0)
    idx = (ctypes.c_int * max(1, P - 1))()
    _check(load_library().sata_feature_index(d, P, f, ctypes.byref(deg), idx), "sata_feature_index")
    return tuple(idx[j] for j in range(deg.value))


# ------------------------------------------------------------------ tensor calls

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return SATA_F32
    if t.dtype == torch.bfloat16:
        return SATA_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _check_tensor(t, name: str, device=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_same_dtype(ref, **tensors):
    for name, t in tensors.items():
        if t.dtype != ref.dtype:
            raise TypeError(f"{name} is {t.dtype}, expected {ref.dtype} like q")


def _check_shape(t, name: str, shape):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _check_state(S, shape):
    if S.dtype != _torch().float32:
        raise TypeError("S must be float32")
    _check_shape(S, "S", shape)


def _stream_ptr():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(None)


def _features(d: int, P: int) -> int:
    D = feature_count(d, P)
    if D < 0:
        raise ValueError(f"invalid d={d} or P={P}")
    return D


def feature_map(x, P: int, phi=None):
    """phi(x) for x [..., d] (float32 or bfloat16) -> float32 [..., D].

    A preallocated float32 output [..., D] may be passed as phi=."""
    torch = _torch()
    code = _dtype_code(x)
    d = x.shape[-1]
    rows = x.numel() // d if d else 0
    D = _features(d, P)
    if phi is not None:
        if phi.dtype != torch.float32:
            raise TypeError(f"phi is {phi.dtype}, expected torch.float32")
        _check_shape(phi, "phi", (*x.shape[:-1], D))
    _check_tensor(x, "x")
    if phi is None:
        phi = torch.empty(*x.shape[:-1], D, dtype=torch.float32, device=x.device)
    _check_tensor(phi, "phi", x.device)
    with torch.cuda.device(x.device):
        _check(load_library().sata_feature_map(_ptr(x), code, rows, d, P, _ptr(phi), _stream_ptr()),
               "sata_feature_map")
    return phi


def prefill_operands(dtype, B: int, H: int, n: int, d_k: int, d_v: int, P: int, chunk: int = 64) -> str:
    """Operand precision of the state contractions that prefill uses for these
    arguments (host only): 'bf16' (bfloat16 operands), 'split' (float32
    operands as bfloat16 hi + lo pairs, three products each) or 'f32'."""
    torch = _torch()
    code = {torch.float32: SATA_F32, torch.bfloat16: SATA_BF16}.get(dtype)
    if code is None:
        raise TypeError(f"unsupported dtype {dtype}; use float32 or bfloat16")
    out = ctypes.c_int(-1)
    _check(load_library().sata_prefill_operands(code, B, H, n, d_k, d_v, P, chunk, ctypes.byref(out)),
           "sata_prefill_operands")
    return {0: "f32", 1: "bf16", 2: "split"}[out.value]


def prefill_parts(dtype, B: int, H: int, n: int, d_k: int, d_v: int, P: int, chunk: int = 64) -> int:
    """Number of parts of the sequence that prefill runs side by side for these
    arguments (host only; 1: one scan from the first token to the last)."""
    torch = _torch()
    code = {torch.float32: SATA_F32, torch.bfloat16: SATA_BF16}.get(dtype)
    if code is None:
        raise TypeError(f"unsupported dtype {dtype}; use float32 or bfloat16")
    out = ctypes.c_int(-1)
    _check(load_library().sata_prefill_parts(code, B, H, n, d_k, d_v, P, chunk, ctypes.byref(out)),
           "sata_prefill_parts")
    return out.value


def prefill(q, k, v, P: int, chunk: int = 64, want_state: bool = True, y=None, S=None):
    """Causal prefill.  q, k: [B, H, n, d_k]; v: [B, H, n, d_v].

    Returns (y [B, H, n, d_v] in the input dtype, S [B, H, D, d_v+1] float32 or None).
    Preallocated outputs may be passed as y= and S=.  Shapes and dtypes are
    checked before anything is launched.
    """
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v)
    if q.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v must be [B, H, n, d]")
    B, H, n, dk = q.shape
    dv = v.shape[-1]
    _check_shape(k, "k", (B, H, n, dk))
    _check_shape(v, "v", (B, H, n, dv))
    D = _features(dk, P)
    if y is not None:
        _check_same_dtype(q, y=y)
        _check_shape(y, "y", (B, H, n, dv))
    if S is not None:
        _check_state(S, (B, H, D, dv + 1))
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(t, name, q.device)
    if y is None:
        y = torch.empty(B, H, n, dv, dtype=q.dtype, device=q.device)
    if want_state and S is None:
        S = torch.empty(B, H, D, dv + 1, dtype=torch.float32, device=q.device)
    _check_tensor(y, "y", q.device)
    if S is not None:
        _check_tensor(S, "S", q.device)
    with torch.cuda.device(q.device):
        _check(load_library().sata_prefill(_ptr(q), _ptr(k), _ptr(v), code, B, H, n, dk, dv, P, chunk,
                                           _ptr(y), _ptr(S) if S is not None else ctypes.c_void_p(None),
                                           _stream_ptr()), "sata_prefill")
    return y, S


def prefill_grouped(q, k, v, P: int, chunk: int = 64, want_state: bool = True, y=None, S=None):
    """Causal prefill with grouped query heads.  q: [B, H_q, n, d_k] with
    H_q = G * H_kv (query head g + G*h reads key/value head h); k: [B, H_kv, n, d_k];
    v: [B, H_kv, n, d_v].  Returns (y [B, H_q, n, d_v], S [B, H_kv, D, d_v+1] or None)."""
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v)
    if q.dim() != 4 or k.dim() != 4 or v.dim() != 4:
        raise ValueError("q [B, G*H_kv, n, d_k], k [B, H_kv, n, d_k], v [B, H_kv, n, d_v] expected")
    B, Hq, n, dk = q.shape
    Hkv = k.shape[1]
    dv = v.shape[-1]
    if Hkv < 1 or Hq % Hkv:
        raise ValueError("the query head count must be a multiple of the key/value head count")
    G = Hq // Hkv
    _check_shape(k, "k", (B, Hkv, n, dk))
    _check_shape(v, "v", (B, Hkv, n, dv))
    D = _features(dk, P)
    if y is not None:
        _check_same_dtype(q, y=y)
        _check_shape(y, "y", (B, Hq, n, dv))
    if S is not None:
        _check_state(S, (B, Hkv, D, dv + 1))
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_tensor(t, name, q.device)
    if y is None:
        y = torch.empty(B, Hq, n, dv, dtype=q.dtype, device=q.device)
    if want_state and S is None:
        S = torch.empty(B, Hkv, D, dv + 1, dtype=torch.float32, device=q.device)
    _check_tensor(y, "y", q.device)
    if S is not None:
        _check_tensor(S, "S", q.device)
    with torch.cuda.device(q.device):
        _check(load_library().sata_prefill_grouped(_ptr(q), _ptr(k), _ptr(v), code, B, Hkv, G, n, dk, dv, P, chunk,
                                                   _ptr(y), _ptr(S) if S is not None else ctypes.c_void_p(None),
                                                   _stream_ptr()), "sata_prefill_grouped")
    return y, S


def backward(q, k, v, dy, P: int, chunk: int = 64):
    """Gradients of the causal prefill's output y for dL/dy = dy.
    q, k: [B, H, n, d_k]; v, dy: [B, H, n, d_v].  Returns (dq, dk, dv) in q's dtype."""
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v, dy=dy)
    if q.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v, dy must be [B, H, n, d]")
    B, H, n, dk = q.shape
    dv = v.shape[-1]
    _check_shape(k, "k", (B, H, n, dk))
    _check_shape(v, "v", (B, H, n, dv))
    _check_shape(dy, "dy", (B, H, n, dv))
    _features(dk, P)
    for name, t in (("q", q), ("k", k), ("v", v), ("dy", dy)):
        _check_tensor(t, name, q.device)
    dq, dkk, dvv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    with torch.cuda.device(q.device):
        _check(load_library().sata_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(dy), code, B, H, n, dk, dv, P, chunk,
                                            _ptr(dq), _ptr(dkk), _ptr(dvv), _stream_ptr()), "sata_backward")
    return dq, dkk, dvv


def decode_step(S, q, k, v, P: int, y=None):
    """One decode step in place on S [B, H, D, d_v+1]; q, k: [B, H, d_k]; v: [B, H, d_v].

    Returns y [B, H, d_v] in the input dtype.  Shapes and dtypes are checked
    before anything is launched.
    """
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v)
    if q.dim() != 3 or v.dim() != 3:
        raise ValueError("q, k, v must be [B, H, d]")
    B, H, dk = q.shape
    dv = v.shape[-1]
    _check_shape(k, "k", (B, H, dk))
    _check_shape(v, "v", (B, H, dv))
    _check_state(S, (B, H, _features(dk, P), dv + 1))
    if y is not None:
        _check_same_dtype(q, y=y)
        _check_shape(y, "y", (B, H, dv))
    for name, t in (("S", S), ("q", q), ("k", k), ("v", v)):
        _check_tensor(t, name, q.device)
    if y is None:
        y = torch.empty(B, H, dv, dtype=q.dtype, device=q.device)
    _check_tensor(y, "y", q.device)
    with torch.cuda.device(q.device):
        _check(load_library().sata_decode_step(_ptr(S), _ptr(q), _ptr(k), _ptr(v), code, B, H, dk, dv, P,
                                               _ptr(y), _stream_ptr()), "sata_decode_step")
    return y


def residual_elems(d_k: int, d_v: int, P: int) -> int:
    return int(load_library().sata_residual_elems(d_k, d_v, P))


def decode_step_compensated(S, R, q, k, v, P: int, y=None):
    """decode_step with compensated summation of the normaliser column and the
    degree-0/1 rows: R [B, H, residual_elems(d_k, d_v, P)] float32, zero when
    the state is created, updated in place with S.  Returns y [B, H, d_v]."""
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v)
    if q.dim() != 3 or v.dim() != 3:
        raise ValueError("q, k, v must be [B, H, d]")
    B, H, dk = q.shape
    dv = v.shape[-1]
    _check_shape(k, "k", (B, H, dk))
    _check_shape(v, "v", (B, H, dv))
    _check_state(S, (B, H, _features(dk, P), dv + 1))
    if R.dtype != torch.float32:
        raise TypeError("R must be float32")
    _check_shape(R, "R", (B, H, residual_elems(dk, dv, P)))
    if y is not None:
        _check_same_dtype(q, y=y)
        _check_shape(y, "y", (B, H, dv))
    for name, t in (("S", S), ("R", R), ("q", q), ("k", k), ("v", v)):
        _check_tensor(t, name, q.device)
    if y is None:
        y = torch.empty(B, H, dv, dtype=q.dtype, device=q.device)
    _check_tensor(y, "y", q.device)
    with torch.cuda.device(q.device):
        _check(load_library().sata_decode_step_compensated(_ptr(S), _ptr(R), _ptr(q), _ptr(k), _ptr(v), code, B, H,
                                                           dk, dv, P, _ptr(y), _stream_ptr()),
               "sata_decode_step_compensated")
    return y


def decode_step_grouped(S, q, k, v, P: int, y=None):
    """One decode step with grouped query heads, in place on S [B, H_kv, D, d_v+1].

    q: [B, H_q, d_k] with H_q = G * H_kv (query head g + G*h reads key/value
    head h); k: [B, H_kv, d_k]; v: [B, H_kv, d_v].  Returns y [B, H_q, d_v].
    """
    torch = _torch()
    code = _dtype_code(q)
    _check_same_dtype(q, k=k, v=v)
    if q.dim() != 3 or k.dim() != 3 or v.dim() != 3:
        raise ValueError("q [B, G*H_kv, d_k], k [B, H_kv, d_k], v [B, H_kv, d_v] expected")
    B, Hq, dk = q.shape
    Hkv = k.shape[1]
    dv = v.shape[-1]
    if Hkv < 1 or Hq % Hkv:
        raise ValueError("the query head count must be a multiple of the key/value head count")
    _check_shape(k, "k", (B, Hkv, dk))
    _check_shape(v, "v", (B, Hkv, dv))
    G = Hq // Hkv
    _check_state(S, (B, Hkv, _features(dk, P), dv + 1))
    if y is not None:
        _check_same_dtype(q, y=y)
        _check_shape(y, "y", (B, Hq, dv))
    for name, t in (("S", S), ("q", q), ("k", k), ("v", v)):
        _check_tensor(t, name, q.device)
    if y is None:
        y = torch.empty(B, Hq, dv, dtype=q.dtype, device=q.device)
    _check_tensor(y, "y", q.device)
    with torch.cuda.device(q.device):
        _check(load_library().sata_decode_step_grouped(_ptr(S), _ptr(q), _ptr(k), _ptr(v), code, B, Hkv, G,
                                                       dk, dv, P, _ptr(y), _stream_ptr()),
               "sata_decode_step_grouped")
    return y


def release():
    load_library().sata_release()

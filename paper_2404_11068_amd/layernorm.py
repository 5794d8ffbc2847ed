"""Python binding of the C ABI in include/evo_layernorm.h (argument marshalling only).

The LayerNorm runs in the HIP library ``libevoattn.so``; this module turns
torch tensors into device pointers and nonzero status codes into exceptions.
It has no fallback: a missing library raises.

  x, y, dy, dx : contiguous [..., C] (fp32 or bf16), normalised over the last axis
  weight, bias, dweight, dbias : contiguous fp32 [C]
  mean, rstd : contiguous fp32 [...] (x's shape without its last axis)
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from .evo_attn import EvoAttnError, _DTYPES, _ptr, _stream, load_library

LN_COLS = (32, 64, 128, 256, 512, 1024)


class evo_ln_dims(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_cols", ctypes.c_int32), ("n_rows", ctypes.c_int64),
                ("eps", ctypes.c_float), ("reserved", ctypes.c_int32)]


_bound = False


def _lib():
    global _bound
    lib = load_library()
    if not _bound:
        P = ctypes.c_void_p
        D = ctypes.POINTER(evo_ln_dims)
        lib.evo_layernorm_fwd.argtypes = [D] + [P] * 7
        lib.evo_layernorm_fwd.restype = ctypes.c_int
        lib.evo_layernorm_bwd_workspace_size.argtypes = [D]
        lib.evo_layernorm_bwd_workspace_size.restype = ctypes.c_size_t
        lib.evo_layernorm_bwd.argtypes = [D] + [P] * 9 + [ctypes.c_size_t, P]
        lib.evo_layernorm_bwd.restype = ctypes.c_int
        lib.evo_layernorm_bwd_traced.argtypes = [D] + [P] * 9 + [ctypes.c_size_t, ctypes.POINTER(P),
                                                               ctypes.c_int, P]
        lib.evo_layernorm_bwd_traced.restype = ctypes.c_int
        _bound = True
    return lib


def make_dims(x: torch.Tensor, eps: float) -> evo_ln_dims:
    if x.dtype not in _DTYPES:
        raise ValueError("dtype must be float32 or bfloat16")
    if not x.is_contiguous() or x.dim() < 1:
        raise ValueError("x must be contiguous with the normalised axis last")
    C = x.shape[-1]
    return evo_ln_dims(_DTYPES[x.dtype], C, x.numel() // C if C else 0, float(eps), 0)


def _check_param(t: Optional[torch.Tensor], C: int, name: str):
    if t is None or t.dtype != torch.float32 or not t.is_contiguous() or t.shape != (C,):
        raise ValueError("%s must be a contiguous float32 tensor of shape (%d,)" % (name, C))


def workspace_size(x: torch.Tensor, eps: float = 1e-5) -> int:
    d = make_dims(x, eps)
    return int(_lib().evo_layernorm_bwd_workspace_size(ctypes.byref(d)))


def layernorm_fwd(x, weight, bias, eps: float = 1e-5, *, y=None, mean=None, rstd=None,
                  need_stats: bool = True, stream=None):
    """y = LayerNorm(x) over the last axis; returns (y, mean, rstd) (the
    statistics are None when need_stats is False and none were given)."""
    lib = _lib()
    d = make_dims(x, eps)
    C = x.shape[-1]
    _check_param(weight, C, "weight")
    _check_param(bias, C, "bias")
    y = torch.empty_like(x) if y is None else y
    if y.shape != x.shape or y.dtype != x.dtype or not y.is_contiguous():
        raise ValueError("y must be contiguous and shaped like x")
    if need_stats:
        mean = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if mean is None else mean
        rstd = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if rstd is None else rstd
    st = lib.evo_layernorm_fwd(ctypes.byref(d), _ptr(x), _ptr(weight), _ptr(bias), _ptr(y), _ptr(mean),
                               _ptr(rstd), _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_layernorm_fwd")
    return y, mean, rstd


def layernorm_bwd(x, weight, mean, rstd, dy, *, dx=None, dweight=None, dbias=None, workspace=None,
                  eps: float = 1e-5, stream=None, events=None):
    """Gradients (dx, dweight, dbias) of the LayerNorm for upstream dy.

    With `events` (at least 3 torch.cuda.Event(enable_timing=True)) the call
    goes to evo_layernorm_bwd_traced, which records them around its kernels."""
    lib = _lib()
    d = make_dims(x, eps)
    C = x.shape[-1]
    _check_param(weight, C, "weight")
    if dy.shape != x.shape or dy.dtype != x.dtype or not dy.is_contiguous():
        raise ValueError("dy must be contiguous and shaped like x")
    dx = torch.empty_like(x) if dx is None else dx
    dweight = torch.empty(C, dtype=torch.float32, device=x.device) if dweight is None else dweight
    dbias = torch.empty(C, dtype=torch.float32, device=x.device) if dbias is None else dbias
    need = int(lib.evo_layernorm_bwd_workspace_size(ctypes.byref(d)))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    args = [ctypes.byref(d), _ptr(x), _ptr(weight), _ptr(mean), _ptr(rstd), _ptr(dy), _ptr(dx),
            _ptr(dweight), _ptr(dbias), _ptr(workspace),
            ctypes.c_size_t(workspace.numel() * workspace.element_size())]
    if events is None:
        st = lib.evo_layernorm_bwd(*args, _stream(stream))
        where = "evo_layernorm_bwd"
    else:
        for e in events:  # torch creates the HIP event lazily, on its first record
            if not e.cuda_event:
                e.record(torch.cuda.current_stream() if stream is None else stream)
        handles = (ctypes.c_void_p * len(events))(*[ctypes.c_void_p(e.cuda_event) for e in events])
        st = lib.evo_layernorm_bwd_traced(*args, handles, len(events), _stream(stream))
        where = "evo_layernorm_bwd_traced"
    if st:
        raise EvoAttnError(st, where)
    return dx, dweight, dbias

"""Python binding of the C ABI in include/evo_proj.h (argument marshalling only).

The fused LayerNorm + batched projections run in ``libevoattn.so``; this
module passes torch tensors' device pointers and raises on a nonzero status.
No fallback exists.

  x : contiguous [..., C] bf16
  ln_weight, ln_bias : fp32 [C]
  weight : contiguous [n_proj * HD, C] bf16 (torch Linear layout, projections stacked)
  bias : fp32 [n_proj * HD] or None
  returns n_proj tensors [..., HD] bf16 (view them as [..., H, d] for the attention)
"""
from __future__ import annotations

import ctypes
from typing import List, Optional

import torch

from .evo_attn import EvoAttnError, _ptr, _stream, load_library, EVO_DTYPE_BF16


class evo_proj_dims(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("c_in", ctypes.c_int32), ("n_proj", ctypes.c_int32),
                ("proj_dim", ctypes.c_int32), ("n_rows", ctypes.c_int64), ("eps", ctypes.c_float),
                ("reserved", ctypes.c_int32)]


_bound = False


def _lib():
    global _bound
    lib = load_library()
    if not _bound:
        P = ctypes.c_void_p
        lib.evo_ln_proj_fwd.argtypes = [ctypes.POINTER(evo_proj_dims), P, P, P, P, P, ctypes.POINTER(P), P, P, P]
        lib.evo_ln_proj_fwd.restype = ctypes.c_int
        lib.evo_ln_proj_fwd_ex.argtypes = [ctypes.POINTER(evo_proj_dims), P, P, P, P, P, ctypes.POINTER(P), P, P,
                                           P, P]
        lib.evo_ln_proj_fwd_ex.restype = ctypes.c_int
        lib.evo_ln_proj_bwd_workspace_size.argtypes = [ctypes.POINTER(evo_proj_dims)]
        lib.evo_ln_proj_bwd_workspace_size.restype = ctypes.c_size_t
        lib.evo_ln_proj_bwd.argtypes = [ctypes.POINTER(evo_proj_dims), P, P, P, P, P, P, ctypes.POINTER(P), P, P, P,
                                        P, P, P, ctypes.c_size_t, P]
        lib.evo_ln_proj_bwd.restype = ctypes.c_int
        lib.evo_linear_fwd.argtypes = [ctypes.POINTER(evo_proj_dims), P, P, P, ctypes.POINTER(P), P]
        lib.evo_linear_fwd.restype = ctypes.c_int
        lib.evo_linear_bwd_workspace_size.argtypes = [ctypes.POINTER(evo_proj_dims)]
        lib.evo_linear_bwd_workspace_size.restype = ctypes.c_size_t
        lib.evo_linear_bwd.argtypes = [ctypes.POINTER(evo_proj_dims), P, P, ctypes.POINTER(P), P, P, P, P,
                                       ctypes.c_size_t, P]
        lib.evo_linear_bwd.restype = ctypes.c_int
        _bound = True
    return lib


def ln_proj_fwd(x: torch.Tensor, ln_weight: torch.Tensor, ln_bias: torch.Tensor, weight: torch.Tensor,
                bias: Optional[torch.Tensor] = None, n_proj: int = 4, eps: float = 1e-5, *,
                outs: Optional[List[torch.Tensor]] = None, mean=None, rstd=None, need_stats: bool = False,
                y_norm: Optional[torch.Tensor] = None, stream=None) -> List[torch.Tensor]:
    """outs[p] = LayerNorm(x) @ weight[p*HD:(p+1)*HD].T + bias[p*HD:(p+1)*HD].

    With need_stats (or mean/rstd given) the LayerNorm statistics are stored
    too and returned after the outputs: (outs, mean, rstd).  With y_norm (a
    bf16 tensor shaped like x) the normalised input is saved there for
    ln_proj_bwd."""
    lib = _lib()
    if x.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16:
        raise ValueError("x and weight must be bfloat16")
    if not x.is_contiguous() or not weight.is_contiguous() or weight.dim() != 2:
        raise ValueError("x and weight must be contiguous; weight is [n_proj*HD, C]")
    C = x.shape[-1]
    if weight.shape[1] != C or weight.shape[0] % n_proj:
        raise ValueError("weight must be [n_proj*HD, C]")
    HD = weight.shape[0] // n_proj
    R = x.numel() // C if C else 0
    if outs is None:
        outs = [torch.empty(x.shape[:-1] + (HD,), dtype=torch.bfloat16, device=x.device) for _ in range(n_proj)]
    if len(outs) != n_proj or any(o.dtype != torch.bfloat16 or not o.is_contiguous() or o.numel() != R * HD
                                  for o in outs):
        raise ValueError("outs must be n_proj contiguous bf16 tensors of R*HD elements")
    if need_stats or mean is not None:
        mean = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if mean is None else mean
        rstd = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device) if rstd is None else rstd
    d = evo_proj_dims(EVO_DTYPE_BF16, C, n_proj, HD, R, float(eps), 0)
    ptrs = (ctypes.c_void_p * n_proj)(*[ctypes.c_void_p(o.data_ptr()) for o in outs])
    if y_norm is not None and (y_norm.dtype != torch.bfloat16 or not y_norm.is_contiguous()
                               or y_norm.numel() != x.numel()):
        raise ValueError("y_norm must be a contiguous bf16 tensor shaped like x")
    st = lib.evo_ln_proj_fwd_ex(ctypes.byref(d), _ptr(x), _ptr(ln_weight), _ptr(ln_bias), _ptr(weight),
                                _ptr(bias), ptrs, _ptr(mean), _ptr(rstd), _ptr(y_norm), _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_ln_proj_fwd_ex")
    if mean is not None:
        return outs, mean, rstd
    return outs


def ln_proj_bwd(x, ln_weight, mean, rstd, y_norm, weight, douts, *, eps: float = 1e-5, has_bias: bool = True,
                dx=None, dweight=None, dbias=None, dln_weight=None, dln_bias=None, workspace=None, stream=None):
    """Gradients (dx, dweight, dbias or None, dln_weight, dln_bias) of
    ln_proj_fwd for upstream gradients douts (one [..., HD] bf16 tensor per
    projection), from the forward's statistics and saved normalised input."""
    lib = _lib()
    P = len(douts)
    C = x.shape[-1]
    HD = weight.shape[0] // P
    R = x.numel() // C if C else 0
    for t in list(douts) + [x, y_norm, weight]:
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError("x, y_norm, weight and douts must be contiguous bfloat16")
    if any(t.numel() != R * HD for t in douts) or y_norm.numel() != R * C:
        raise ValueError("douts must hold R*HD elements and y_norm R*C")
    dev = x.device
    dx = torch.empty_like(x) if dx is None else dx
    dweight = torch.empty((P * HD, C), dtype=torch.float32, device=dev) if dweight is None else dweight
    if has_bias and dbias is None:
        dbias = torch.empty(P * HD, dtype=torch.float32, device=dev)
    dln_weight = torch.empty(C, dtype=torch.float32, device=dev) if dln_weight is None else dln_weight
    dln_bias = torch.empty(C, dtype=torch.float32, device=dev) if dln_bias is None else dln_bias
    d = evo_proj_dims(EVO_DTYPE_BF16, C, P, HD, R, float(eps), 0)
    need = int(lib.evo_ln_proj_bwd_workspace_size(ctypes.byref(d)))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    ptrs = (ctypes.c_void_p * P)(*[ctypes.c_void_p(t.data_ptr()) for t in douts])
    st = lib.evo_ln_proj_bwd(ctypes.byref(d), _ptr(x), _ptr(ln_weight), _ptr(mean), _ptr(rstd), _ptr(y_norm),
                             _ptr(weight), ptrs, _ptr(dx), _ptr(dweight), _ptr(dbias if has_bias else None),
                             _ptr(dln_weight), _ptr(dln_bias), _ptr(workspace),
                             ctypes.c_size_t(workspace.numel() * workspace.element_size()), _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_ln_proj_bwd")
    return dx, dweight, (dbias if has_bias else None), dln_weight, dln_bias


def linear_fwd(x: torch.Tensor, weight: torch.Tensor, bias: Optional[torch.Tensor] = None, n_proj: int = 1, *,
               outs: Optional[List[torch.Tensor]] = None, stream=None) -> List[torch.Tensor]:
    """outs[p] = x @ weight[p*HD:(p+1)*HD].T + bias[p*HD:(p+1)*HD] (no LayerNorm),
    e.g. the attention module's output projection."""
    lib = _lib()
    if x.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16:
        raise ValueError("x and weight must be bfloat16")
    if not x.is_contiguous() or not weight.is_contiguous() or weight.dim() != 2:
        raise ValueError("x and weight must be contiguous; weight is [n_proj*HD, C]")
    C = x.shape[-1]
    if weight.shape[1] != C or weight.shape[0] % n_proj:
        raise ValueError("weight must be [n_proj*HD, C]")
    HD = weight.shape[0] // n_proj
    R = x.numel() // C if C else 0
    if outs is None:
        outs = [torch.empty(x.shape[:-1] + (HD,), dtype=torch.bfloat16, device=x.device) for _ in range(n_proj)]
    if len(outs) != n_proj or any(o.dtype != torch.bfloat16 or not o.is_contiguous() or o.numel() != R * HD
                                  for o in outs):
        raise ValueError("outs must be n_proj contiguous bf16 tensors of R*HD elements")
    d = evo_proj_dims(EVO_DTYPE_BF16, C, n_proj, HD, R, 0.0, 0)
    ptrs = (ctypes.c_void_p * n_proj)(*[ctypes.c_void_p(o.data_ptr()) for o in outs])
    st = lib.evo_linear_fwd(ctypes.byref(d), _ptr(x), _ptr(weight), _ptr(bias), ptrs, _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_linear_fwd")
    return outs


def linear_bwd(x, weight, douts, *, has_bias: bool = True, dx=None, dweight=None, dbias=None, workspace=None,
               stream=None):
    """Gradients (dx, dweight, dbias or None) of linear_fwd for upstream
    gradients douts (one [..., HD] bf16 tensor per projection)."""
    lib = _lib()
    P = len(douts)
    C = x.shape[-1]
    HD = weight.shape[0] // P
    R = x.numel() // C if C else 0
    for t in list(douts) + [x, weight]:
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise ValueError("x, weight and douts must be contiguous bfloat16")
    if any(t.numel() != R * HD for t in douts):
        raise ValueError("douts must hold R*HD elements")
    dev = x.device
    dx = torch.empty_like(x) if dx is None else dx
    dweight = torch.empty((P * HD, C), dtype=torch.float32, device=dev) if dweight is None else dweight
    if has_bias and dbias is None:
        dbias = torch.empty(P * HD, dtype=torch.float32, device=dev)
    d = evo_proj_dims(EVO_DTYPE_BF16, C, P, HD, R, 0.0, 0)
    need = int(lib.evo_linear_bwd_workspace_size(ctypes.byref(d)))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    ptrs = (ctypes.c_void_p * P)(*[ctypes.c_void_p(t.data_ptr()) for t in douts])
    st = lib.evo_linear_bwd(ctypes.byref(d), _ptr(x), _ptr(weight), ptrs, _ptr(dx), _ptr(dweight),
                            _ptr(dbias if has_bias else None), _ptr(workspace),
                            ctypes.c_size_t(workspace.numel() * workspace.element_size()), _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_linear_bwd")
    return dx, dweight, (dbias if has_bias else None)


class evo_pair_bias_dims(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("c_in", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("transpose", ctypes.c_int32), ("n_batch", ctypes.c_int64), ("len_i", ctypes.c_int64),
                ("len_j", ctypes.c_int64), ("eps", ctypes.c_float), ("reserved", ctypes.c_int32)]


_pb_bound = False


def _pb_lib():
    global _pb_bound
    lib = load_library()
    if not _pb_bound:
        P = ctypes.c_void_p
        lib.evo_ln_pair_bias_fwd.argtypes = [ctypes.POINTER(evo_pair_bias_dims)] + [P] * 8
        lib.evo_ln_pair_bias_bwd_workspace_size.argtypes = [ctypes.POINTER(evo_pair_bias_dims)]
        lib.evo_ln_pair_bias_bwd_workspace_size.restype = ctypes.c_size_t
        lib.evo_ln_pair_bias_bwd.argtypes = [ctypes.POINTER(evo_pair_bias_dims)] + [P] * 10 + [ctypes.c_size_t, P]
        lib.evo_ln_pair_bias_bwd.restype = ctypes.c_int
        lib.evo_ln_pair_bias_fwd.restype = ctypes.c_int
        _pb_bound = True
    return lib


def ln_pair_bias_fwd(z: torch.Tensor, ln_weight: torch.Tensor, ln_bias: torch.Tensor, weight: torch.Tensor,
                     eps: float = 1e-5, transpose: bool = False, *, out: Optional[torch.Tensor] = None,
                     need_stats: bool = False, stream=None):
    """Pair bias [B, H, Li, Lj] (or [B, H, Lj, Li] with transpose) from the
    pair representation z [B, Li, Lj, C]: LayerNorm of each entry, then a
    bias-free linear map with weight [H, C].  With need_stats also returns
    the LayerNorm mean and rstd [B, Li, Lj]."""
    lib = _pb_lib()
    if z.dim() == 3:
        z = z.unsqueeze(0)
    if z.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16 or not z.is_contiguous() \
            or not weight.is_contiguous():
        raise ValueError("z and weight must be contiguous bfloat16")
    B, Li, Lj, C = z.shape
    H = weight.shape[0]
    if weight.shape != (H, C):
        raise ValueError("weight must be [H, C]")
    shape = (B, H, Lj, Li) if transpose else (B, H, Li, Lj)
    if out is None:
        out = torch.empty(shape, dtype=torch.bfloat16, device=z.device)
    if tuple(out.shape) != shape or out.dtype != torch.bfloat16 or not out.is_contiguous():
        raise ValueError("out must be a contiguous bf16 tensor of shape %s" % (shape,))
    mean = rstd = None
    if need_stats:
        mean = torch.empty((B, Li, Lj), dtype=torch.float32, device=z.device)
        rstd = torch.empty((B, Li, Lj), dtype=torch.float32, device=z.device)
    d = evo_pair_bias_dims(EVO_DTYPE_BF16, C, H, 1 if transpose else 0, B, Li, Lj, float(eps), 0)
    st = lib.evo_ln_pair_bias_fwd(ctypes.byref(d), _ptr(z), _ptr(ln_weight), _ptr(ln_bias), _ptr(weight),
                                  _ptr(out), _ptr(mean), _ptr(rstd), _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_ln_pair_bias_fwd")
    return (out, mean, rstd) if need_stats else out


def pair_bias_bwd_workspace_size(B: int, Li: int, Lj: int, C: int, H: int, transpose: bool = False,
                                 eps: float = 1e-5) -> int:
    d = evo_pair_bias_dims(EVO_DTYPE_BF16, C, H, 1 if transpose else 0, B, Li, Lj, float(eps), 0)
    return int(_pb_lib().evo_ln_pair_bias_bwd_workspace_size(ctypes.byref(d)))


def ln_pair_bias_bwd(z: torch.Tensor, ln_weight: torch.Tensor, ln_bias: torch.Tensor, weight: torch.Tensor,
                     dbias: torch.Tensor, eps: float = 1e-5, transpose: bool = False, *,
                     dz: Optional[torch.Tensor] = None, dweight: Optional[torch.Tensor] = None,
                     dln_weight: Optional[torch.Tensor] = None, dln_bias: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None):
    """Gradients (dz, dweight [H, C], dln_weight, dln_bias) of ln_pair_bias_fwd
    for the upstream gradient dbias (fp32, the forward's output layout)."""
    lib = _pb_lib()
    if z.dim() == 3:
        z = z.unsqueeze(0)
    if z.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16 or not z.is_contiguous() \
            or not weight.is_contiguous():
        raise ValueError("z and weight must be contiguous bfloat16")
    B, Li, Lj, C = z.shape
    H = weight.shape[0]
    if weight.shape != (H, C):
        raise ValueError("weight must be [H, C]")
    shape = (B, H, Lj, Li) if transpose else (B, H, Li, Lj)
    if dbias.dim() == 3:
        dbias = dbias.unsqueeze(0)
    if tuple(dbias.shape) != shape or dbias.dtype != torch.float32 or not dbias.is_contiguous():
        raise ValueError("dbias must be a contiguous float32 tensor of shape %s" % (shape,))
    dz = torch.empty_like(z) if dz is None else dz
    if dz.shape != z.shape or dz.dtype != torch.bfloat16 or not dz.is_contiguous():
        raise ValueError("dz must be contiguous and shaped like z")
    f32 = lambda n: torch.empty(n, dtype=torch.float32, device=z.device)
    dweight = f32((H, C)) if dweight is None else dweight
    dln_weight = f32(C) if dln_weight is None else dln_weight
    dln_bias = f32(C) if dln_bias is None else dln_bias
    d = evo_pair_bias_dims(EVO_DTYPE_BF16, C, H, 1 if transpose else 0, B, Li, Lj, float(eps), 0)
    need = int(lib.evo_ln_pair_bias_bwd_workspace_size(ctypes.byref(d)))
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=z.device)
    st = lib.evo_ln_pair_bias_bwd(ctypes.byref(d), _ptr(z), _ptr(ln_weight), _ptr(ln_bias), _ptr(weight),
                                  _ptr(dbias), _ptr(dz), _ptr(dweight), _ptr(dln_weight), _ptr(dln_bias),
                                  _ptr(workspace), ctypes.c_size_t(workspace.numel() * workspace.element_size()),
                                  _stream(stream))
    if st:
        raise EvoAttnError(st, "evo_ln_pair_bias_bwd")
    return dz, dweight, dln_weight, dln_bias

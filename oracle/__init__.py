"""fp64 CPU oracle for the Evoformer gated attention with pair bias.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The product path (the HIP library and
its Python binding) never imports this package, and this package imports
nothing from the product.

The arithmetic lives in ``evo_attn_oracle.c`` (plain loops, fp64, OpenMP over
(row, head) pairs); this file only builds and calls it through ctypes.
Every function cites what it computes in the C source header.

``EVO_ORACLE_LIB``, when set, names an already compiled oracle library to load
instead of the one built here (the mutation test points it at copies of the C
source with planted mistakes, to show that the pins catch them).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "evo_attn_oracle.c")
_SRCS = [_SRC, os.path.join(_HERE, "layernorm_oracle.c")]
_LIB = os.path.join(_HERE, "liboracle_evoattn.so")

_lib = None


class _Dims(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("seq_len", ctypes.c_int64),
                ("n_heads", ctypes.c_int64), ("head_dim", ctypes.c_int64),
                ("rows_per_bias", ctypes.c_int64)]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, IEEE semantics, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-o", tmp] + _SRCS + ["-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("EVO_ORACLE_LIB")
        if not path:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(map(os.path.getmtime, _SRCS)):
                build(force=True)
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        lib.evo_oracle_fwd.argtypes = [ctypes.POINTER(_Dims), P, P, P, P, P, P, P, P]
        lib.evo_oracle_bwd.argtypes = [ctypes.POINTER(_Dims)] + [P] * 12
        lib.evo_oracle_probs.argtypes = [ctypes.POINTER(_Dims), P, P, P, P, ctypes.c_int64,
                                         ctypes.c_int64, P]
        for f in (lib.evo_oracle_fwd, lib.evo_oracle_bwd, lib.evo_oracle_probs):
            f.restype = ctypes.c_int
        lib.evo_oracle_threads.restype = ctypes.c_int
        I, D = ctypes.c_int64, ctypes.c_double
        lib.ln_oracle_fwd.argtypes = [I, I, D] + [P] * 6
        lib.ln_oracle_bwd.argtypes = [I, I, D] + [P] * 6
        lib.ln_oracle_fwd.restype = lib.ln_oracle_bwd.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle uses (OMP_NUM_THREADS, else all cores)."""
    return int(_load().evo_oracle_threads())


def _f64(x: Optional[np.ndarray]) -> Optional[np.ndarray]:
    return None if x is None else np.ascontiguousarray(x, dtype=np.float64)


def _ptr(x: Optional[np.ndarray]):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def _dims(q: np.ndarray, rows_per_bias: int) -> _Dims:
    N, L, H, d = q.shape
    return _Dims(N, L, H, d, rows_per_bias)


def _mask(m: Optional[np.ndarray]) -> Optional[np.ndarray]:
    return None if m is None else np.ascontiguousarray(m, dtype=np.uint8)


def forward(q, k, v, gate=None, bias=None, mask=None, rows_per_bias: Optional[int] = None
            ) -> Tuple[np.ndarray, np.ndarray]:
    """o [N,L,H,d] and lse [N,H,L] (natural log); fp64 inputs of shape [N,L,H,d]."""
    q, k, v, gate, bias = map(_f64, (q, k, v, gate, bias))
    mask = _mask(mask)
    N, L, H, d = q.shape
    rpb = rows_per_bias or max(N, 1)
    out = np.zeros_like(q)
    lse = np.zeros((N, H, L), np.float64)
    dm = _dims(q, rpb)
    st = _load().evo_oracle_fwd(ctypes.byref(dm), _ptr(q), _ptr(k), _ptr(v), _ptr(gate),
                                _ptr(bias), _ptr(mask), _ptr(out), _ptr(lse))
    if st:
        raise ValueError("oracle forward failed with status %d" % st)
    return out, lse


def backward(q, k, v, dout, gate=None, bias=None, mask=None, rows_per_bias: Optional[int] = None):
    """Gradients (dq, dk, dv, dgate or None, dbias or None)."""
    q, k, v, dout, gate, bias = map(_f64, (q, k, v, dout, gate, bias))
    mask = _mask(mask)
    N, L, H, d = q.shape
    rpb = rows_per_bias or max(N, 1)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(q), np.zeros_like(q)
    dg = np.zeros_like(q) if gate is not None else None
    db = np.zeros_like(bias) if bias is not None else None
    dm = _dims(q, rpb)
    st = _load().evo_oracle_bwd(ctypes.byref(dm), _ptr(q), _ptr(k), _ptr(v), _ptr(gate),
                                _ptr(bias), _ptr(mask), _ptr(dout), _ptr(dq), _ptr(dk), _ptr(dv),
                                _ptr(dg), _ptr(db))
    if st:
        raise ValueError("oracle backward failed with status %d" % st)
    return dq, dk, dv, dg, db


def probs(q, k, bias=None, mask=None, row: int = 0, head: int = 0,
          rows_per_bias: Optional[int] = None) -> np.ndarray:
    """Softmax matrix P [L,L] of one (row, head)."""
    q, k, bias = map(_f64, (q, k, bias))
    mask = _mask(mask)
    N, L, H, d = q.shape
    rpb = rows_per_bias or max(N, 1)
    P = np.zeros((L, L), np.float64)
    dm = _dims(q, rpb)
    st = _load().evo_oracle_probs(ctypes.byref(dm), _ptr(q), _ptr(k), _ptr(bias), _ptr(mask),
                                  row, head, _ptr(P))
    if st:
        raise ValueError("oracle probs failed with status %d" % st)
    return P


def layernorm_forward(x, weight=None, bias=None, eps: float = 1e-5):
    """LayerNorm over the last axis: (y, mean, rstd), y shaped like x, the
    statistics shaped like x without its last axis (layernorm_oracle.c)."""
    x = _f64(x)
    C = x.shape[-1]
    R = x.size // C if C else 0
    w, b = _f64(weight), _f64(bias)
    for p_ in (w, b):
        if p_ is not None and p_.shape != (C,):
            raise ValueError("weight and bias must have shape (%d,)" % C)
    y = np.zeros_like(x)
    mean = np.zeros(x.shape[:-1], np.float64)
    rstd = np.zeros(x.shape[:-1], np.float64)
    st = _load().ln_oracle_fwd(R, C, float(eps), _ptr(x), _ptr(w), _ptr(b), _ptr(y),
                               _ptr(mean), _ptr(rstd))
    if st:
        raise ValueError("oracle layernorm forward failed with status %d" % st)
    return y, mean, rstd


def layernorm_backward(x, dy, weight=None, eps: float = 1e-5):
    """Gradients (dx, dweight, dbias) of the LayerNorm above for upstream dy."""
    x, dy, w = _f64(x), _f64(dy), _f64(weight)
    if dy.shape != x.shape:
        raise ValueError("dy must be shaped like x")
    C = x.shape[-1]
    R = x.size // C if C else 0
    dx = np.zeros_like(x)
    dw = np.zeros(C, np.float64)
    db = np.zeros(C, np.float64)
    st = _load().ln_oracle_bwd(R, C, float(eps), _ptr(x), _ptr(w), _ptr(dy), _ptr(dx),
                               _ptr(dw), _ptr(db))
    if st:
        raise ValueError("oracle layernorm backward failed with status %d" % st)
    return dx, dw, db


def ln_proj_forward(x, ln_weight, ln_bias, weight, bias=None, n_proj: int = 1, eps: float = 1e-5):
    """LayerNorm over the last axis followed by n_proj independent linear
    projections that share the normalised input (ScaleFold Section 3.3,
    GEMM Batching: the query, key, value and gate projections in front of
    the attention are mutually independent, so they form one batched
    product).

    x [..., C]; weight [n_proj * HD, C] (torch Linear layout: row f of
    projection p is weight[p * HD + f]); bias [n_proj * HD] or None.
    Returns a list of n_proj arrays [..., HD]:
        out_p = LN(x) @ weight[p*HD:(p+1)*HD].T + bias[p*HD:(p+1)*HD]
    The matmul is a library primitive (numpy, fp64)."""
    x = _f64(x)
    W = _f64(weight)
    C = x.shape[-1]
    if W.ndim != 2 or W.shape[1] != C or W.shape[0] % n_proj:
        raise ValueError("weight must be [n_proj * HD, C]")
    HD = W.shape[0] // n_proj
    y, _, _ = layernorm_forward(x, ln_weight, ln_bias, eps)
    outs = []
    for p in range(n_proj):
        o = y @ W[p * HD:(p + 1) * HD].T
        if bias is not None:
            o = o + _f64(bias)[p * HD:(p + 1) * HD]
        outs.append(o)
    return outs


def pair_bias_forward(z, ln_weight, ln_bias, weight, eps: float = 1e-5, transpose: bool = False):
    """Pair bias of the Evoformer attentions: a LayerNorm of each pair entry
    followed by a linear map without bias to one value per head (the bias
    term that ScaleFold Section 3.3 adds to the logits).

    z [B, Li, Lj, C]; weight [H, C].  Returns [B, H, Li, Lj] with
        out[b, h, i, j] = sum_c LN(z[b, i, j, :])[c] * weight[h, c]
    or, with transpose, [B, H, Lj, Li] with out[b, h, j, i] equal to the
    same value (the layout triangle attention around the ending node reads).
    The contraction is a library primitive (numpy matmul, fp64)."""
    z = _f64(z)
    W = _f64(weight)
    if z.ndim != 4 or W.ndim != 2 or W.shape[1] != z.shape[3]:
        raise ValueError("z is [B, Li, Lj, C] and weight [H, C]")
    y, _, _ = layernorm_forward(z, ln_weight, ln_bias, eps)
    out = np.moveaxis(y @ W.T, 3, 1)          # [B, H, Li, Lj]
    if transpose:
        out = np.swapaxes(out, 2, 3)          # [B, H, Lj, Li]
    return np.ascontiguousarray(out)


def linear_forward(x, weight, bias=None, n_proj: int = 1):
    """n_proj linear layers sharing the input x [..., C]: outs[p] = x W_p^T + b_p
    with W_p = weight[p*HD:(p+1)*HD] (torch Linear layout) -- the output
    projection after the gated attention, and the batched projections of
    ln_proj_forward without their LayerNorm.  numpy matmul, fp64."""
    x = _f64(x)
    W = _f64(weight)
    if W.ndim != 2 or W.shape[1] != x.shape[-1] or W.shape[0] % n_proj:
        raise ValueError("weight must be [n_proj * HD, C]")
    HD = W.shape[0] // n_proj
    b = None if bias is None else _f64(bias)
    outs = []
    for p in range(n_proj):
        o = x @ W[p * HD:(p + 1) * HD].T
        if b is not None:
            o = o + b[p * HD:(p + 1) * HD]
        outs.append(o)
    return outs


def linear_backward(x, weight, douts):
    """Gradients of linear_forward: (dx, dweight [n_proj*HD, C], dbias [n_proj*HD])
    with dx = sum_p dout_p W_p, dW_p = dout_p^T x, db_p = sum over tokens of dout_p."""
    x = _f64(x)
    W = _f64(weight)
    C = x.shape[-1]
    P = len(douts)
    HD = W.shape[0] // P
    x2 = x.reshape(-1, C)
    d2 = [_f64(d).reshape(-1, HD) for d in douts]
    dx = sum(d2[p] @ W[p * HD:(p + 1) * HD] for p in range(P))
    dW = np.concatenate([d2[p].T @ x2 for p in range(P)], axis=0)
    db = np.concatenate([d2[p].sum(axis=0) for p in range(P)])
    return dx.reshape(x.shape), dW, db


def pair_bias_backward(z, ln_weight, ln_bias, weight, dbias, eps: float = 1e-5, transpose: bool = False):
    """Gradients of pair_bias_forward for the upstream gradient dbias (the
    attention backward's dL/dbias, [B, H, Li, Lj], or [B, H, Lj, Li] with
    transpose): (dz, dln_weight, dln_bias, dweight [H, C]).

    With y = LN(z) and g[b, i, j, h] the upstream value of entry (i, j):
    dY = g @ W;  (dz, dln_weight, dln_bias) is the LayerNorm backward of dY;
    dW = sum over entries of g^T y.  Matmuls are library primitives (numpy,
    fp64)."""
    z = _f64(z)
    W = _f64(weight)
    g = _f64(dbias)
    if z.ndim != 4 or W.ndim != 2 or W.shape[1] != z.shape[3]:
        raise ValueError("z is [B, Li, Lj, C] and weight [H, C]")
    B, Li, Lj, C = z.shape
    H = W.shape[0]
    want = (B, H, Lj, Li) if transpose else (B, H, Li, Lj)
    if g.shape != want:
        raise ValueError("dbias must be %s" % (want,))
    if transpose:
        g = np.swapaxes(g, 2, 3)                 # [B, H, Li, Lj]
    g = np.moveaxis(g, 1, 3)                     # [B, Li, Lj, H]
    y, _, _ = layernorm_forward(z, ln_weight, ln_bias, eps)
    dY = g @ W                                   # [B, Li, Lj, C]
    dz, dlw, dlb = layernorm_backward(z, dY, ln_weight, eps)
    dW = g.reshape(-1, H).T @ y.reshape(-1, C)   # [H, C]
    return dz, dlw, dlb, dW


def ln_proj_backward(x, ln_weight, ln_bias, weight, douts, eps: float = 1e-5):
    """Gradients of ln_proj_forward for upstream gradients douts[p] ([..., HD]):
    (dx, dln_weight, dln_bias, dweight [n_proj*HD, C], dbias [n_proj*HD]).

    With y = LN(x):  dY = sum_p dout_p @ W_p;  (dx, dln_weight, dln_bias) is the
    LayerNorm backward of dY;  dW_p = dout_p^T @ y;  dbias_p = sum over tokens
    of dout_p.  Matmuls are library primitives (numpy, fp64)."""
    x = _f64(x)
    W = _f64(weight)
    C = x.shape[-1]
    P = len(douts)
    HD = W.shape[0] // P
    x2 = x.reshape(-1, C)
    y, _, _ = layernorm_forward(x2, ln_weight, ln_bias, eps)
    d2 = [_f64(d).reshape(-1, HD) for d in douts]
    dY = np.zeros_like(x2)
    for p in range(P):
        dY += d2[p] @ W[p * HD:(p + 1) * HD]
    dx, dlw, dlb = layernorm_backward(x2, dY, ln_weight, eps)
    dW = np.concatenate([d2[p].T @ y for p in range(P)], axis=0)
    db = np.concatenate([d2[p].sum(axis=0) for p in range(P)])
    return dx.reshape(x.shape), dlw, dlb, dW, db

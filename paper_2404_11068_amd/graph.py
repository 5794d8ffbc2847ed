"""Python binding of include/evo_graph.h (the shape-keyed HIP graph cache) and
an attention module step that uses it.

`GraphCache.run(key, record, stream)` captures `record(stream_handle)` into a
HIP graph the first time a key is seen and launches the graph on every call.
`record` receives the raw hipStream_t (an int) and must only enqueue this
library's kernels on it (no allocation, no synchronisation).

`MSARowAttentionStep` is the work of one MSA row attention with pair bias
(LayerNorm + q/k/v/gate projections, LayerNorm(z) + pair-bias projection,
attention forward, attention backward, backward of the projections and their
LayerNorm) on static buffers, runnable eagerly (one C-ABI call per stage) or
through the cache (one graph launch).
"""
from __future__ import annotations

import ctypes
from typing import Callable, Optional

import numpy as np
import torch

from . import evo_attn as ea
from . import proj as pj
from .evo_attn import EvoAttnError, _stream, load_library

RECORD_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)

_bound = False


def _lib():
    global _bound
    lib = load_library()
    if not _bound:
        P = ctypes.c_void_p
        lib.evo_graph_cache_create.argtypes = [ctypes.c_int32, ctypes.POINTER(P)]
        lib.evo_graph_cache_create.restype = ctypes.c_int
        lib.evo_graph_cache_destroy.argtypes = [P]
        lib.evo_graph_cache_destroy.restype = ctypes.c_int
        lib.evo_graph_cache_run.argtypes = [P, ctypes.c_uint64, RECORD_FN, P, P, ctypes.POINTER(ctypes.c_int32)]
        lib.evo_graph_cache_run.restype = ctypes.c_int
        lib.evo_graph_cache_size.argtypes = [P]
        lib.evo_graph_cache_size.restype = ctypes.c_int32
        lib.evo_graph_cache_clear.argtypes = [P]
        lib.evo_graph_cache_clear.restype = ctypes.c_int
        _bound = True
    return lib


class GraphCache:
    def __init__(self, capacity: int = 8):
        self._lib = _lib()
        h = ctypes.c_void_p()
        st = self._lib.evo_graph_cache_create(int(capacity), ctypes.byref(h))
        if st:
            raise EvoAttnError(st, "evo_graph_cache_create")
        self._h = h
        self.captures = 0
        # one C callback for the cache's lifetime; it calls the record function
        # of the run in progress (only on a miss)
        self._record = None
        self._err = []
        self._cb = RECORD_FN(self._dispatch)
        self._cap = ctypes.c_int32(0)
        self._run = self._lib.evo_graph_cache_run

    def _dispatch(self, _user, s):
        try:
            self._record(int(s or 0))
        except Exception as e:  # surfaced after the capture ends
            self._err.append(e)

    def run(self, key: int, record: Callable[[int], None], stream) -> bool:
        """Launch the graph for key (capturing record first on a miss); returns
        True when this call captured."""
        self._record = record
        st = self._run(self._h, key & 0xFFFFFFFFFFFFFFFF, self._cb, None, _stream(stream), ctypes.byref(self._cap))
        self._record = None
        if self._err:
            e, self._err = self._err[0], []
            raise e
        if st:
            raise EvoAttnError(st, "evo_graph_cache_run")
        self.captures += int(self._cap.value)
        return bool(self._cap.value)

    def __len__(self):
        return int(self._lib.evo_graph_cache_size(self._h))

    def clear(self):
        self._lib.evo_graph_cache_clear(self._h)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.evo_graph_cache_destroy(h)
            self._h = None


class MSARowAttentionStep:
    """Static buffers and weights of one MSA row attention with pair bias:
    m [N, L, c_m], z [L, L, c_z] -> q, k, v, g, bias -> o, lse -> m_out = o W_out^T + b_out; backward
    from d_m_out: dout (at o), dW_out, db_out -> dq, dk, dv, dg, dbias -> dm and the projection weight
    gradients, dz and the pair-bias weight gradients."""

    def __init__(self, N: int, L: int, c_m: int = 256, c_z: int = 128, H: int = 8, d: int = 32, seed: int = 0,
                 device="cuda"):
        g = torch.Generator(device="cpu").manual_seed(seed)
        bf = dict(dtype=torch.bfloat16, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        r = lambda *s, scale=1.0: (torch.randn(*s, generator=g) * scale)
        self.N, self.L, self.H, self.d = N, L, H, d
        self.m = r(N, L, c_m).to(**bf)
        self.z = r(1, L, L, c_z).to(**bf)
        self.ln_m_w, self.ln_m_b = (1 + 0.1 * r(c_m)).to(**f32), (0.1 * r(c_m)).to(**f32)
        self.ln_z_w, self.ln_z_b = (1 + 0.1 * r(c_z)).to(**f32), (0.1 * r(c_z)).to(**f32)
        self.w_qkvg = r(4 * H * d, c_m, scale=c_m ** -0.5).to(**bf)
        self.b_qkvg = torch.cat([torch.zeros(3 * H * d), torch.ones(H * d)]).to(**f32)  # gate bias 1
        self.w_bias = r(H, c_z, scale=c_z ** -0.5).to(**bf)
        self.mask = torch.ones(N, L, dtype=torch.uint8, device=device)
        # output projection of the gated attention back to c_m, and the module's upstream gradient
        self.w_out = r(c_m, H * d, scale=(H * d) ** -0.5).to(**bf)
        self.b_out = (0.1 * r(c_m)).to(**f32)
        self.m_out = torch.empty(N, L, c_m, **bf)
        self.d_m_out = r(N, L, c_m).to(**bf)
        self.dout = torch.empty(N, L, H, d, **bf)  # gradient at the attention output (from the projection)
        self.dw_out = torch.empty(c_m, H * d, **f32)
        self.db_out = torch.empty(c_m, **f32)
        self.q, self.k, self.v, self.gate = (torch.empty(N, L, H, d, **bf) for _ in range(4))
        self.bias = torch.empty(1, H, L, L, **bf)
        self.out = torch.empty(N, L, H, d, **bf)
        self.lse = torch.empty(N, H, L, **f32)
        self.dq, self.dk, self.dv, self.dg = (torch.empty(N, L, H, d, **bf) for _ in range(4))
        self.dbias = torch.empty(1, H, L, L, **f32)
        self.ws = torch.empty(max(ea.evo_attn_bwd_workspace_size(self.q, N), 1), dtype=torch.uint8, device=device)
        # training forward state of the projections and their gradients
        self.y_norm = torch.empty_like(self.m)
        self.mean = torch.empty(N, L, **f32)
        self.rstd = torch.empty(N, L, **f32)
        self.dm = torch.empty_like(self.m)
        self.dw_qkvg = torch.empty(4 * H * d, c_m, **f32)
        self.db_qkvg = torch.empty(4 * H * d, **f32)
        self.dln_m_w = torch.empty(c_m, **f32)
        self.dln_m_b = torch.empty(c_m, **f32)
        dims = pj.evo_proj_dims(1, c_m, 4, H * d, N * L, 1e-5, 0)
        self.ws_proj = torch.empty(max(int(pj._lib().evo_ln_proj_bwd_workspace_size(ctypes.byref(dims))), 1),
                                   dtype=torch.uint8, device=device)
        dims_o = pj.evo_proj_dims(1, H * d, 1, c_m, N * L, 0.0, 0)
        self.ws_out = torch.empty(max(int(pj._lib().evo_linear_bwd_workspace_size(ctypes.byref(dims_o))), 1),
                                  dtype=torch.uint8, device=device)
        # pair-bias gradients (the attention's dbias through LN(z) and the projection to heads)
        self.dz = torch.empty_like(self.z)
        self.dw_bias = torch.empty(H, c_z, **f32)
        self.dln_z_w = torch.empty(c_z, **f32)
        self.dln_z_b = torch.empty(c_z, **f32)
        self.ws_pb = torch.empty(max(pj.pair_bias_bwd_workspace_size(1, L, L, c_z, H), 16), dtype=torch.uint8,
                                 device=device)

        self._key = hash((N, L, H, d, self.m.data_ptr(), self.z.data_ptr(), self.dq.data_ptr())) & \
            0xFFFFFFFFFFFFFFFF

    def key(self) -> int:
        """Shape-and-buffer key of this step's graph (the buffers are static)."""
        return self._key

    def record(self, stream):
        """Enqueue the step (8 C-ABI calls, 17 kernels) on `stream` (torch stream or raw handle):
        projections, pair bias, attention, output projection; then the backward in reverse."""
        pj.ln_proj_fwd(self.m, self.ln_m_w, self.ln_m_b, self.w_qkvg, self.b_qkvg, n_proj=4,
                       outs=[t.view(self.N, self.L, -1) for t in (self.q, self.k, self.v, self.gate)],
                       mean=self.mean, rstd=self.rstd, y_norm=self.y_norm, stream=stream)
        pj.ln_pair_bias_fwd(self.z, self.ln_z_w, self.ln_z_b, self.w_bias, out=self.bias, stream=stream)
        ea.evo_attn_fwd(self.q, self.k, self.v, self.gate, self.bias, self.mask, rows_per_bias=self.N,
                        out=self.out, lse=self.lse, stream=stream)
        HDm = self.H * self.d
        pj.linear_fwd(self.out.view(self.N, self.L, HDm), self.w_out, self.b_out,
                      outs=[self.m_out], stream=stream)
        pj.linear_bwd(self.out.view(self.N, self.L, HDm), self.w_out, [self.d_m_out],
                      dx=self.dout.view(self.N, self.L, HDm), dweight=self.dw_out, dbias=self.db_out,
                      workspace=self.ws_out, stream=stream)
        ea.evo_attn_bwd(self.q, self.k, self.v, self.gate, self.bias, self.mask, self.out, self.lse, self.dout,
                        rows_per_bias=self.N, dq=self.dq, dk=self.dk, dv=self.dv, dgate=self.dg, dbias=self.dbias,
                        workspace=self.ws, stream=stream)
        pj.ln_proj_bwd(self.m, self.ln_m_w, self.mean, self.rstd, self.y_norm, self.w_qkvg,
                       [t.view(self.N, self.L, -1) for t in (self.dq, self.dk, self.dv, self.dg)],
                       dx=self.dm, dweight=self.dw_qkvg, dbias=self.db_qkvg, dln_weight=self.dln_m_w,
                       dln_bias=self.dln_m_b, workspace=self.ws_proj, stream=stream)
        pj.ln_pair_bias_bwd(self.z, self.ln_z_w, self.ln_z_b, self.w_bias, self.dbias, dz=self.dz,
                            dweight=self.dw_bias, dln_weight=self.dln_z_w, dln_bias=self.dln_z_b, workspace=self.ws_pb,
                            stream=stream)

    def outputs(self):
        return {k: getattr(self, k) for k in ("q", "k", "v", "gate", "bias", "out", "lse", "dq", "dk", "dv", "dg",
                                               "dbias", "y_norm", "dm", "dw_qkvg", "db_qkvg", "dln_m_w", "dln_m_b",
                                               "dz", "dw_bias", "dln_z_w", "dln_z_b", "m_out", "dout", "dw_out",
                                               "db_out")}

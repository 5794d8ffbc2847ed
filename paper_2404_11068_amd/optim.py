"""Python binding of the C ABI in include/evo_optim.h (argument marshalling only).

`FusedAdamSWA` packs the pointers of every parameter, gradient and optimizer
state tensor into a device table once (and the chunk list that splits them
into EVO_MT_CHUNK-element work items), then each `step` enqueues the
gradient-norm clipping kernels and the fused Adam + SWA kernel of
``libevoattn.so``.  The table holds raw pointers: rebuild the object if any
of the tensors is reallocated.  No fallback exists.
"""
from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence

import numpy as np
import torch

from .evo_attn import EvoAttnError, _stream, load_library

EVO_MT_CHUNK = 4096


class evo_mt_tensor(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("swa", ctypes.c_void_p), ("numel", ctypes.c_int64)]


class evo_mt_chunk(ctypes.Structure):
    _fields_ = [("tensor", ctypes.c_int32), ("index", ctypes.c_int32)]


class evo_adam_swa_hparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("weight_decay", ctypes.c_double), ("swa_decay", ctypes.c_double),
                ("step", ctypes.c_int64)]


_bound = False


def _lib():
    global _bound
    lib = load_library()
    if not _bound:
        P = ctypes.c_void_p
        lib.evo_mt_chunk_count.argtypes = [ctypes.POINTER(ctypes.c_int64), ctypes.c_int32]
        lib.evo_mt_chunk_count.restype = ctypes.c_int64
        lib.evo_mt_build_chunks.argtypes = [ctypes.POINTER(ctypes.c_int64), ctypes.c_int32, P, ctypes.c_int64]
        lib.evo_mt_build_chunks.restype = ctypes.c_int64
        lib.evo_grad_clip_scale.argtypes = [P, ctypes.c_int32, P, ctypes.c_int32, ctypes.c_float, P, P, P, P]
        lib.evo_grad_clip_scale.restype = ctypes.c_int
        lib.evo_adam_swa_step.argtypes = [ctypes.POINTER(evo_adam_swa_hparams), P, ctypes.c_int32, P, ctypes.c_int32,
                                          P, P]
        lib.evo_adam_swa_step.restype = ctypes.c_int
        _bound = True
    return lib


def _check(t: torch.Tensor, name: str, n: int):
    if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or t.numel() != n:
        raise ValueError("%s must be a contiguous float32 CUDA tensor of %d elements" % (name, n))


class FusedAdamSWA:
    """Adam + SWA over packed tensors, with optional gradient-norm clipping."""

    def __init__(self, params: Sequence[torch.Tensor], grads: Sequence[torch.Tensor],
                 exp_avg: Optional[Sequence[torch.Tensor]] = None, exp_avg_sq: Optional[Sequence[torch.Tensor]] = None,
                 swa: Optional[Sequence[torch.Tensor]] = None, *, lr=1e-3, betas=(0.9, 0.999), eps=1e-6,
                 weight_decay=0.0, swa_decay=0.999):
        lib = _lib()
        self.params = list(params)
        self.grads = list(grads)
        n = len(self.params)
        if len(self.grads) != n:
            raise ValueError("one gradient per parameter")
        self.exp_avg = list(exp_avg) if exp_avg is not None else [torch.zeros_like(p) for p in self.params]
        self.exp_avg_sq = list(exp_avg_sq) if exp_avg_sq is not None else [torch.zeros_like(p) for p in self.params]
        self.swa = list(swa) if swa is not None else [p.detach().clone() for p in self.params]
        numels = np.array([p.numel() for p in self.params], dtype=np.int64)
        for i in range(n):
            for t, nm in ((self.params[i], "param"), (self.grads[i], "grad"), (self.exp_avg[i], "exp_avg"),
                          (self.exp_avg_sq[i], "exp_avg_sq"), (self.swa[i], "swa")):
                _check(t, "%s[%d]" % (nm, i), int(numels[i]))
        tab = (evo_mt_tensor * max(n, 1))()
        for i in range(n):
            tab[i] = evo_mt_tensor(self.params[i].data_ptr(), self.grads[i].data_ptr(), self.exp_avg[i].data_ptr(),
                                   self.exp_avg_sq[i].data_ptr(), self.swa[i].data_ptr(), int(numels[i]))
        nptr = numels.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
        nch = int(lib.evo_mt_chunk_count(nptr, n))
        if nch < 0:
            raise ValueError("tensor sizes too large for the chunk table")
        ch = (evo_mt_chunk * max(nch, 1))()
        if int(lib.evo_mt_build_chunks(nptr, n, ch, nch)) != nch:
            raise RuntimeError("evo_mt_build_chunks failed")
        dev = self.params[0].device if n else torch.device("cuda")
        self.tensor_table = torch.frombuffer(bytearray(bytes(tab)), dtype=torch.uint8).to(dev)
        self.chunk_table = torch.frombuffer(bytearray(bytes(ch)), dtype=torch.uint8).to(dev)
        self.n_tensors, self.n_chunks = n, nch
        self.workspace = torch.empty(max(nch, 1), dtype=torch.float32, device=dev)
        self.norm = torch.zeros(1, dtype=torch.float32, device=dev)
        self.scale = torch.ones(1, dtype=torch.float32, device=dev)
        self.lr, self.betas, self.eps, self.weight_decay, self.swa_decay = lr, betas, eps, weight_decay, swa_decay
        self.step_count = 0

    def clip(self, max_norm: float, stream=None):
        """Gradient norm and clipping scale into self.norm / self.scale (device)."""
        st = _lib().evo_grad_clip_scale(self.tensor_table.data_ptr(), self.n_tensors, self.chunk_table.data_ptr(),
                                        self.n_chunks, float(max_norm), self.workspace.data_ptr(),
                                        self.norm.data_ptr(), self.scale.data_ptr(), _stream(stream))
        if st:
            raise EvoAttnError(st, "evo_grad_clip_scale")

    def step(self, max_norm: Optional[float] = None, stream=None, step: Optional[int] = None):
        """One optimizer step (clipping first when max_norm is given)."""
        if max_norm is not None:
            self.clip(max_norm, stream)
        self.step_count = self.step_count + 1 if step is None else step
        hp = evo_adam_swa_hparams(self.lr, self.betas[0], self.betas[1], self.eps, self.weight_decay,
                                  self.swa_decay, self.step_count)
        st = _lib().evo_adam_swa_step(ctypes.byref(hp), self.tensor_table.data_ptr(), self.n_tensors,
                                      self.chunk_table.data_ptr(), self.n_chunks,
                                      self.scale.data_ptr() if max_norm is not None else None, _stream(stream))
        if st:
            raise EvoAttnError(st, "evo_adam_swa_step")

"""Host-side checks of the optimizer-step ABI (no GPU): exports, the host
chunk-table helpers, and rejection of invalid calls before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import optim as op

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7f0000000000


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return op._lib()


def test_exports_declared_symbols():
    lib = _lib()
    decls = re.findall(r"^\s*(?:int|int64_t)\s*(evo_\w+)\s*\(", open(os.path.join(ROOT, "include", "evo_optim.h")).read(),
                       flags=re.M)
    assert set(decls) == {"evo_mt_chunk_count", "evo_mt_build_chunks", "evo_grad_clip_scale", "evo_adam_swa_step"}
    for n in decls:
        assert hasattr(lib, n), n


def test_chunk_helpers():
    lib = _lib()
    sizes = np.array([0, 1, 4096, 4097, 9000], dtype=np.int64)
    p = sizes.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    n = lib.evo_mt_chunk_count(p, len(sizes))
    assert n == 0 + 1 + 1 + 2 + 3
    buf = (op.evo_mt_chunk * n)()
    assert lib.evo_mt_build_chunks(p, len(sizes), buf, n) == n
    assert [(c.tensor, c.index) for c in buf] == [(1, 0), (2, 0), (3, 0), (3, 1), (4, 0), (4, 1), (4, 2)]
    assert lib.evo_mt_build_chunks(p, len(sizes), buf, n - 1) == -1
    bad = np.array([5, -1], dtype=np.int64)
    assert lib.evo_mt_chunk_count(bad.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 2) == -1
    huge = np.array([1 << 50], dtype=np.int64)
    assert lib.evo_mt_chunk_count(huge.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 1) == -1


def _hp(**kw):
    d = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6, weight_decay=0.0, swa_decay=0.999, step=1)
    d.update(kw)
    return op.evo_adam_swa_hparams(d["lr"], d["beta1"], d["beta2"], d["eps"], d["weight_decay"], d["swa_decay"],
                                   d["step"])


@pytest.mark.parametrize("kw", [dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=-1.0),
                                dict(swa_decay=1.5), dict(lr=float("nan")), dict(weight_decay=float("inf"))])
def test_step_rejects_bad_hparams(kw):
    lib = _lib()
    assert lib.evo_adam_swa_step(ctypes.byref(_hp(**kw)), FAKE, 1, FAKE + 4096, 1, None, None) == 1


def test_step_and_clip_reject_bad_tables():
    lib = _lib()
    hp = _hp()
    assert lib.evo_adam_swa_step(None, FAKE, 1, FAKE, 1, None, None) == 1
    assert lib.evo_adam_swa_step(ctypes.byref(hp), None, 1, FAKE, 1, None, None) == 1
    assert lib.evo_adam_swa_step(ctypes.byref(hp), FAKE, 1, None, 1, None, None) == 1
    assert lib.evo_adam_swa_step(ctypes.byref(hp), FAKE, -1, FAKE, 1, None, None) == 1
    assert lib.evo_adam_swa_step(ctypes.byref(hp), FAKE + 4, 1, FAKE, 1, None, None) == 3
    assert lib.evo_adam_swa_step(ctypes.byref(hp), FAKE, 1, FAKE, 1, FAKE + 2, None) == 3
    assert lib.evo_adam_swa_step(ctypes.byref(hp), None, 0, None, 0, None, None) == 0
    assert lib.evo_grad_clip_scale(FAKE, 1, FAKE, 1, ctypes.c_float(0.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.evo_grad_clip_scale(FAKE, 1, FAKE, 1, ctypes.c_float(1.0), None, FAKE, FAKE, None) == 1
    assert lib.evo_grad_clip_scale(None, 1, FAKE, 1, ctypes.c_float(1.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.evo_grad_clip_scale(FAKE, 1, FAKE, 1, ctypes.c_float(1.0), FAKE, None, None, None) == 0

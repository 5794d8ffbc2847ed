"""Host-side checks of evo_ln_pair_bias_fwd (no GPU): exported, and every
invalid call rejected before any HIP call (fake addresses never touched)."""
import ctypes
import os

import pytest

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import proj as pj

FAKE = 0x7f0000000000
P = lambda x: None if x is None else ctypes.c_void_p(x)


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return pj._pb_lib()


def _dims(**kw):
    d = dict(dtype=1, c_in=128, n_heads=8, transpose=0, n_batch=1, len_i=256, len_j=256, eps=1e-5, reserved=0)
    d.update(kw)
    return pj.evo_pair_bias_dims(*[d[k] for k in ("dtype", "c_in", "n_heads", "transpose", "n_batch", "len_i",
                                                  "len_j", "eps", "reserved")])


def _call(dims, z=FAKE, lnw=FAKE + 0x1000000, lnb=FAKE + 0x1001000, w=FAKE + 0x1002000, out=FAKE + 0x2000000,
          mean=None, rstd=None):
    return _lib().evo_ln_pair_bias_fwd(ctypes.byref(dims) if dims is not None else None, P(z), P(lnw), P(lnb),
                                       P(w), P(out), P(mean), P(rstd), None)


def test_exported():
    assert hasattr(_lib(), "evo_ln_pair_bias_fwd")


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=0), 2), (dict(c_in=96), 2), (dict(n_heads=3), 2), (dict(n_heads=32), 2),
    (dict(len_i=250), 2), (dict(len_j=12), 2), (dict(transpose=2), 1), (dict(n_batch=-1), 1),
    (dict(eps=-1.0), 1), (dict(reserved=7), 1), (dict(n_heads=0), 1),
    (dict(len_i=1 << 16, len_j=1 << 16), 2),
])
def test_rejects_bad_dims(kw, status):
    assert _call(_dims(**kw)) == status


def test_rejects_bad_pointers():
    d = _dims()
    assert _call(None) == 1
    for k in ("z", "lnw", "lnb", "w", "out"):
        assert _call(d, **{k: None}) == 1, k
    assert _call(d, out=FAKE) == 1
    assert _call(d, mean=FAKE + 0x3000000) == 1
    assert _call(d, z=FAKE + 8) == 3
    assert _call(d, out=FAKE + 0x2000004) == 3


def test_empty_needs_no_pointers():
    assert _call(_dims(len_i=0), z=None, lnw=None, lnb=None, w=None, out=None) == 0


# ---- backward ---------------------------------------------------------------

def _call_bwd(dims, z=FAKE, lnw=FAKE + 0x1000000, lnb=FAKE + 0x1001000, w=FAKE + 0x1002000, g=FAKE + 0x3000000,
              dz=FAKE + 0x5000000, dw=FAKE + 0x7000000, dlw=FAKE + 0x7100000, dlb=FAKE + 0x7200000,
              ws=FAKE + 0x8000000, ws_bytes=1 << 30):
    return _lib().evo_ln_pair_bias_bwd(ctypes.byref(dims) if dims is not None else None, P(z), P(lnw), P(lnb),
                                       P(w), P(g), P(dz), P(dw), P(dlw), P(dlb), P(ws), ctypes.c_size_t(ws_bytes),
                                       None)


def test_bwd_exported():
    lib = _lib()
    assert hasattr(lib, "evo_ln_pair_bias_bwd") and hasattr(lib, "evo_ln_pair_bias_bwd_workspace_size")


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=0), 2), (dict(c_in=96), 2), (dict(n_heads=3), 2), (dict(n_heads=16), 2),
    (dict(len_i=250), 2), (dict(len_j=12), 2), (dict(transpose=2), 1), (dict(n_batch=-1), 1),
    (dict(eps=-1.0), 1), (dict(reserved=7), 1), (dict(n_heads=0), 1),
    (dict(len_i=1 << 14, len_j=1 << 14), 2),
])
def test_bwd_rejects_bad_dims(kw, status):
    d = _dims(**kw)
    assert _call_bwd(d) == status
    assert _lib().evo_ln_pair_bias_bwd_workspace_size(ctypes.byref(d)) == 0


def test_bwd_rejects_bad_pointers_and_workspace():
    d = _dims()
    need = _lib().evo_ln_pair_bias_bwd_workspace_size(ctypes.byref(d))
    # one partial row (H*C + 2C floats) per workgroup, at most 512 workgroups
    assert need == 512 * (8 * 128 + 2 * 128) * 4
    assert _call_bwd(None) == 1
    for k in ("z", "lnw", "lnb", "w", "g", "dz", "dw", "dlw", "dlb"):
        assert _call_bwd(d, **{k: None}) == 1, k
    assert _call_bwd(d, dz=FAKE) == 1                      # dz aliases z
    assert _call_bwd(d, dlw=FAKE + 0x7000000) == 1         # dln_weight aliases dweight
    assert _call_bwd(d, dlb=FAKE + 0x7100000) == 1         # dln_bias aliases dln_weight
    assert _call_bwd(d, z=FAKE + 8) == 3
    assert _call_bwd(d, g=FAKE + 0x3000004) == 3
    assert _call_bwd(d, dw=FAKE + 0x7000004) == 3
    assert _call_bwd(d, ws=None) == 4
    assert _call_bwd(d, ws_bytes=need - 1) == 4
    assert _call_bwd(d, ws=FAKE + 0x8000008) == 3


def test_bwd_empty_needs_no_pointers():
    d = _dims(len_j=0)
    assert _lib().evo_ln_pair_bias_bwd_workspace_size(ctypes.byref(d)) == 0
    assert _call_bwd(d, z=None, lnw=None, lnb=None, w=None, g=None, dz=None, dw=None, dlw=None, dlb=None,
                     ws=None, ws_bytes=0) == 0

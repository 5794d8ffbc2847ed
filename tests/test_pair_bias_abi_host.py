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

"""Host-side checks of evo_ln_proj_fwd (no GPU): the symbol is exported and
every invalid call is rejected before any HIP call (fake device addresses
are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import proj as pj

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7f0000000000
P = lambda x: None if x is None else ctypes.c_void_p(x)


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return pj._lib()


def test_exports_declared_symbol():
    lib = _lib()
    decls = re.findall(r"^\s*(?:int|size_t)\s*(evo_\w+)\s*\(",
                       open(os.path.join(ROOT, "include", "evo_proj.h")).read(), flags=re.M)
    assert set(decls) == {"evo_ln_proj_fwd", "evo_ln_proj_fwd_ex", "evo_ln_proj_bwd_workspace_size",
                          "evo_ln_proj_bwd", "evo_ln_pair_bias_fwd", "evo_ln_pair_bias_bwd_workspace_size",
                          "evo_ln_pair_bias_bwd", "evo_linear_fwd", "evo_linear_bwd_workspace_size",
                          "evo_linear_bwd"}
    for name in decls:
        assert hasattr(lib, name), name


def _call(dims, x=FAKE, lnw=FAKE + 0x10000, lnb=FAKE + 0x11000, w=FAKE + 0x20000, b=None,
          outs=(FAKE + 0x100000, FAKE + 0x200000, FAKE + 0x300000, FAKE + 0x400000), mean=None, rstd=None,
          n_out=None):
    lib = _lib()
    arr = None
    if outs is not None:
        n = len(outs) if n_out is None else n_out
        arr = (ctypes.c_void_p * max(n, 1))(*[ctypes.c_void_p(o) if o is not None else None for o in outs[:n]])
    return lib.evo_ln_proj_fwd(ctypes.byref(dims) if dims is not None else None, P(x), P(lnw), P(lnb), P(w), P(b),
                               arr, P(mean), P(rstd), None)


def _dims(**kw):
    d = dict(dtype=1, c_in=128, n_proj=4, proj_dim=128, n_rows=1000, eps=1e-5, reserved=0)
    d.update(kw)
    return pj.evo_proj_dims(d["dtype"], d["c_in"], d["n_proj"], d["proj_dim"], d["n_rows"], d["eps"], d["reserved"])


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=0), 2), (dict(c_in=96), 2), (dict(c_in=512), 2), (dict(proj_dim=48), 2),
    (dict(proj_dim=2048), 2), (dict(n_proj=5), 2), (dict(n_proj=0), 1), (dict(n_rows=-2), 1),
    (dict(eps=-1.0), 1), (dict(eps=float("nan")), 1), (dict(reserved=1), 1), (dict(n_rows=1 << 40), 2),
])
def test_rejects_bad_dims(kw, status):
    assert _call(_dims(**kw)) == status


def test_rejects_bad_pointers():
    d = _dims()
    assert _call(None) == 1
    for k in ("x", "lnw", "lnb", "w"):
        assert _call(d, **{k: None}) == 1, k
    assert _call(d, outs=None) == 1
    assert _call(d, outs=(FAKE + 0x100000, None, FAKE + 0x300000, FAKE + 0x400000)) == 1
    assert _call(d, outs=(FAKE + 0x100000, FAKE + 0x100000, FAKE + 0x300000, FAKE + 0x400000)) == 1
    assert _call(d, outs=(FAKE, FAKE + 0x200000, FAKE + 0x300000, FAKE + 0x400000)) == 1   # aliases x
    assert _call(d, mean=FAKE + 0x500000) == 1                                             # rstd missing
    assert _call(d, x=FAKE + 8) == 3
    assert _call(d, w=FAKE + 0x20004) == 3
    assert _call(d, b=FAKE + 0x30008) == 3
    assert _call(d, outs=(FAKE + 0x100008, FAKE + 0x200000, FAKE + 0x300000, FAKE + 0x400000)) == 3


def test_empty_needs_no_pointers():
    assert _call(_dims(n_rows=0), x=None, lnw=None, lnb=None, w=None, outs=None) == 0


def _bwd(dims, x=FAKE, lnw=FAKE + 0x10000, mean=FAKE + 0x11000, rstd=FAKE + 0x12000, y=FAKE + 0x100000,
         w=FAKE + 0x200000, douts=(FAKE + 0x300000, FAKE + 0x400000, FAKE + 0x500000, FAKE + 0x600000),
         dx=FAKE + 0x700000, dW=FAKE + 0x800000, db=None, dlw=FAKE + 0x900000, dlb=FAKE + 0x901000,
         ws=FAKE + 0x1000000, ws_bytes=1 << 30):
    lib = _lib()
    arr = None if douts is None else (ctypes.c_void_p * len(douts))(*[ctypes.c_void_p(o) if o else None
                                                                      for o in douts])
    return lib.evo_ln_proj_bwd(ctypes.byref(dims) if dims is not None else None, P(x), P(lnw), P(mean), P(rstd),
                               P(y), P(w), arr, P(dx), P(dW), P(db), P(dlw), P(dlb), P(ws),
                               ctypes.c_size_t(ws_bytes), None)


def test_backward_rejects_bad_calls():
    lib = _lib()
    d = _dims()
    assert _bwd(_dims(c_in=96)) == 2
    assert _bwd(None) == 1
    for k in ("x", "lnw", "mean", "rstd", "y", "w", "dx", "dW", "dlw", "dlb"):
        assert _bwd(d, **{k: None}) == 1, k
    assert _bwd(d, douts=None) == 1
    assert _bwd(d, douts=(FAKE + 0x300000, None, FAKE + 0x500000, FAKE + 0x600000)) == 1
    assert _bwd(d, dx=FAKE) == 1
    assert _bwd(d, dlb=FAKE + 0x900000) == 1
    assert _bwd(d, y=FAKE + 0x100008) == 3
    assert _bwd(d, douts=(FAKE + 0x300004, FAKE + 0x400000, FAKE + 0x500000, FAKE + 0x600000)) == 3
    need = lib.evo_ln_proj_bwd_workspace_size(ctypes.byref(d))
    assert need > 0
    assert _bwd(d, ws_bytes=need - 1) == 4
    assert _bwd(d, ws=None) == 4
    assert _bwd(_dims(n_rows=0), x=None, y=None, w=None, douts=None, dx=None) == 0
    assert lib.evo_ln_proj_bwd_workspace_size(ctypes.byref(_dims(c_in=96))) == 0



# ---- linear layers (no LayerNorm) ---------------------------------------------

def _lin_fwd(dims, x=FAKE, w=FAKE + 0x20000, b=None, outs=(FAKE + 0x100000,)):
    arr = None if outs is None else (ctypes.c_void_p * len(outs))(*[ctypes.c_void_p(o) if o else None for o in outs])
    return _lib().evo_linear_fwd(ctypes.byref(dims) if dims is not None else None, P(x), P(w), P(b), arr, None)


def _lin_bwd(dims, x=FAKE, w=FAKE + 0x20000, douts=(FAKE + 0x100000,), dx=FAKE + 0x500000, dw=FAKE + 0x600000,
             db=None, ws=FAKE + 0x1000000, ws_bytes=1 << 30):
    arr = None if douts is None else (ctypes.c_void_p * len(douts))(*[ctypes.c_void_p(o) if o else None
                                                                      for o in douts])
    return _lib().evo_linear_bwd(ctypes.byref(dims) if dims is not None else None, P(x), P(w), arr, P(dx), P(dw),
                                 P(db), P(ws), ctypes.c_size_t(ws_bytes), None)


def test_linear_validation():
    d = pj.evo_proj_dims(1, 256, 1, 256, 4096, 0.0, 0)
    assert _lin_fwd(None) == 1
    assert _lin_fwd(pj.evo_proj_dims(0, 256, 1, 256, 4096, 0.0, 0)) == 2
    assert _lin_fwd(pj.evo_proj_dims(1, 96, 1, 256, 4096, 0.0, 0)) == 2
    assert _lin_fwd(d, x=None) == 1 and _lin_fwd(d, w=None) == 1 and _lin_fwd(d, outs=None) == 1
    assert _lin_fwd(d, outs=(FAKE,)) == 1                    # output aliases x
    assert _lin_fwd(d, x=FAKE + 8) == 3 and _lin_fwd(d, outs=(FAKE + 0x100004,)) == 3
    assert _lin_fwd(pj.evo_proj_dims(1, 256, 1, 256, 0, 0.0, 0), x=None, w=None, outs=None) == 0
    need = _lib().evo_linear_bwd_workspace_size(ctypes.byref(d))
    # no LayerNorm: only the weight-gradient partial sums
    assert 0 < need < _lib().evo_ln_proj_bwd_workspace_size(ctypes.byref(d))
    assert _lin_bwd(d, dx=None) == 1 and _lin_bwd(d, douts=(0,)) == 1
    assert _lin_bwd(d, dx=FAKE) == 1                         # dx aliases x
    assert _lin_bwd(d, ws_bytes=need - 1) == 4 and _lin_bwd(d, ws=FAKE + 0x1000010) == 4
    assert _lin_bwd(d, douts=(FAKE + 0x100002,)) == 3
    assert _lin_bwd(pj.evo_proj_dims(1, 256, 1, 256, 0, 0.0, 0), x=None, w=None, douts=None, dx=None, dw=None,
                    ws=None, ws_bytes=0) == 0

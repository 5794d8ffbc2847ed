"""C ABI host-side checks of the LayerNorm entry points (no GPU needed): the
library exports every symbol include/evo_layernorm.h declares, and every
invalid call is rejected before any HIP call.  Each call below is invalid in
exactly one way, so nothing is launched and the fake device addresses are
never dereferenced."""
import ctypes
import os
import re

import pytest

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import layernorm as ln

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "evo_layernorm.h")
FAKE = 0x7f0000000000  # 256-byte aligned, never dereferenced
P = lambda x: None if x is None else ctypes.c_void_p(x)


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return ln._lib()


def test_exports_every_declared_symbol():
    lib = _lib()
    decls = re.findall(r"^\s*(?:int|size_t)\s*(evo_layernorm_\w+)\s*\(", open(HEADER).read(), flags=re.M)
    assert set(decls) == {"evo_layernorm_fwd", "evo_layernorm_bwd", "evo_layernorm_bwd_workspace_size",
                          "evo_layernorm_bwd_traced"}
    for name in decls:
        assert hasattr(lib, name), name


def _dims(**kw):
    d = dict(dtype=1, n_cols=128, n_rows=1000, eps=1e-5, reserved=0)
    d.update(kw)
    return ln.evo_ln_dims(d["dtype"], d["n_cols"], d["n_rows"], d["eps"], d["reserved"])


def _fwd(dims, x=FAKE, w=FAKE + 0x100000, b=FAKE + 0x101000, y=FAKE + 0x200000, mean=FAKE + 0x300000,
         rstd=FAKE + 0x400000):
    lib = _lib()
    return lib.evo_layernorm_fwd(ctypes.byref(dims) if dims is not None else None, P(x), P(w), P(b), P(y),
                                 P(mean), P(rstd), None)


def _bwd(dims, x=FAKE, w=FAKE + 0x100000, mean=FAKE + 0x300000, rstd=FAKE + 0x400000, dy=FAKE + 0x500000,
         dx=FAKE + 0x600000, dw=FAKE + 0x700000, db=FAKE + 0x701000, ws=FAKE + 0x800000, ws_bytes=1 << 30):
    lib = _lib()
    return lib.evo_layernorm_bwd(ctypes.byref(dims) if dims is not None else None, P(x), P(w), P(mean),
                                 P(rstd), P(dy), P(dx), P(dw), P(db), P(ws), ctypes.c_size_t(ws_bytes), None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 2),
    (dict(n_cols=48), 2),
    (dict(n_cols=2048), 2),
    (dict(n_cols=0), 1),
    (dict(n_rows=-1), 1),
    (dict(eps=-1e-3), 1),
    (dict(eps=float("nan")), 1),
    (dict(eps=float("inf")), 1),
    (dict(reserved=3), 1),
    (dict(n_rows=1 << 40), 2),
])
def test_rejects_bad_dims(kw, status):
    assert _fwd(_dims(**kw)) == status
    assert _bwd(_dims(**kw)) == status
    assert _lib().evo_layernorm_bwd_workspace_size(ctypes.byref(_dims(**kw))) == 0


def test_rejects_bad_pointers():
    d = _dims()
    assert _fwd(None) == 1
    assert _fwd(d, x=None) == 1
    assert _fwd(d, w=None) == 1
    assert _fwd(d, b=None) == 1
    assert _fwd(d, y=None) == 1
    assert _fwd(d, y=FAKE) == 1                  # y aliases x
    assert _fwd(d, x=FAKE + 8) == 3
    assert _fwd(d, w=FAKE + 0x100004) == 3
    assert _fwd(d, mean=FAKE + 0x300002) == 3
    assert _bwd(None) == 1
    for k in ("x", "w", "mean", "rstd", "dy", "dx", "dw", "db"):
        assert _bwd(d, **{k: None}) == 1, k
    assert _bwd(d, dx=FAKE) == 1                 # dx aliases x
    assert _bwd(d, db=FAKE + 0x700000) == 1      # dweight aliases dbias
    assert _bwd(d, dy=FAKE + 0x500008) == 3
    assert _bwd(d, dw=FAKE + 0x700004) == 3
    need = _lib().evo_layernorm_bwd_workspace_size(ctypes.byref(d))
    assert need > 0
    assert _bwd(d, ws=None) == 4
    assert _bwd(d, ws_bytes=need - 1) == 4
    assert _bwd(d, ws=FAKE + 0x800010) == 4


def test_empty_forward_needs_no_pointers():
    assert _fwd(_dims(n_rows=0), x=None, w=None, b=None, y=None, mean=None, rstd=None) == 0


def test_workspace_size_grows_then_saturates():
    lib = _lib()
    sizes = [lib.evo_layernorm_bwd_workspace_size(ctypes.byref(_dims(n_rows=r))) for r in
             (0, 1, 100, 10_000, 1_000_000, 100_000_000)]
    assert sizes == sorted(sizes) and sizes[0] > 0
    assert sizes[-1] == sizes[-2]   # one partial row per workgroup, capped
    assert sizes[-1] % (2 * 128 * 4) == 0


def test_traced_rejects_missing_events():
    lib = _lib()
    d = _dims()
    args = [ctypes.byref(d)] + [P(FAKE + i * 0x100000) for i in range(9)] + [ctypes.c_size_t(1 << 30)]
    assert lib.evo_layernorm_bwd_traced(*args, None, 0, None) == 1
    two = (ctypes.c_void_p * 2)(FAKE, FAKE)
    assert lib.evo_layernorm_bwd_traced(*args, two, 2, None) == 1
    nulls = (ctypes.c_void_p * 3)(None, None, None)
    assert lib.evo_layernorm_bwd_traced(*args, nulls, 3, None) == 1

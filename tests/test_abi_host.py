"""C ABI host-side checks that need no GPU: the library loads, exports every
symbol include/evo_attn.h declares, and rejects invalid calls before any HIP
call.  Every call here is invalid in exactly one way, so nothing is ever
launched (the fake device addresses are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2404_11068_amd import evo_attn as ea

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "evo_attn.h")

FAKE = 0x7f0000000000  # 256-byte aligned, never dereferenced


def _lib():
    if not os.path.exists(ea.LIB_PATH):
        pytest.skip("libevoattn.so not built")
    return ea.load_library()


def test_exports_every_declared_symbol():
    lib = _lib()
    decls = re.findall(r"^\s*(?:int|size_t|const char \*)\s*(evo_attn_\w+)\s*\(",
                       open(HEADER).read(), flags=re.M)
    assert set(decls) == {"evo_attn_fwd", "evo_attn_bwd", "evo_attn_bwd_workspace_size",
                          "evo_attn_bwd_traced", "evo_attn_bwd_kernel_count",
                          "evo_attn_bwd_noalloc", "evo_attn_bwd_noalloc_scratch_bytes",
                          "evo_attn_strerror", "evo_attn_version"}
    for name in decls:
        assert hasattr(lib, name), name


def test_strerror_and_version():
    _lib()
    for st in range(7):
        assert isinstance(ea.evo_attn_strerror(st), str) and ea.evo_attn_strerror(st)
    assert "unknown" in ea.evo_attn_strerror(99)
    assert ea.evo_attn_version() >= 10000


def _dims(**kw):
    d = dict(dtype=1, n_heads=2, head_dim=32, reserved=0, n_rows=4, seq_len=16, rows_per_bias=4)
    d.update(kw)
    H, hd = d["n_heads"], d["n_heads"] * d["head_dim"]
    d.setdefault("stride_tok", hd)
    d.setdefault("stride_row", d["seq_len"] * d["stride_tok"])
    return ea.evo_attn_dims(d["dtype"], d["n_heads"], d["head_dim"], d["reserved"], d["n_rows"],
                            d["seq_len"], d["rows_per_bias"], d["stride_row"], d["stride_tok"])


def _fwd(dims, q=FAKE, k=FAKE + 4096, v=FAKE + 8192, g=None, bias=None, mask=None,
         out=FAKE + 16384, lse=FAKE + 32768):
    lib = _lib()
    P = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.evo_attn_fwd(ctypes.byref(dims) if dims is not None else None, P(q), P(k), P(v), P(g),
                            P(bias), P(mask), P(out), P(lse), None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 2),
    (dict(head_dim=24), 2),
    (dict(head_dim=128), 2),
    (dict(dtype=0, head_dim=64, seq_len=129), 2),   # fp32 d=64: at most 128 keys
    (dict(seq_len=513), 2),
    (dict(dtype=0, seq_len=257), 2),                # fp32: at most 256 keys
    (dict(head_dim=64, seq_len=257), 2),            # head_dim 64: at most 256 keys
    (dict(n_heads=0), 1),
    (dict(n_rows=-1), 1),
    (dict(seq_len=-3), 1),
    (dict(reserved=1), 1),
    (dict(stride_tok=32), 1),                   # < H*d
    (dict(stride_row=64, stride_tok=64), 1),    # rows and tokens overlap
    (dict(stride_tok=68, stride_row=68 * 16), 3),  # bf16 stride not 16-byte multiple
])
def test_fwd_rejects_bad_dims(kw, status):
    assert _fwd(_dims(**kw)) == status


def test_fwd_rejects_null_and_misaligned_pointers():
    assert _fwd(None) == 1
    assert _fwd(_dims(), q=None) == 1
    assert _fwd(_dims(), lse=None) == 1
    assert _fwd(_dims(), out=FAKE) == 1             # output aliases q
    assert _fwd(_dims(), k=FAKE + 4098) == 3
    assert _fwd(_dims(), lse=FAKE + 2) == 3
    assert _fwd(_dims(), bias=FAKE + 8) == 3


def test_fwd_rejects_bad_rows_per_bias_only_with_bias():
    assert _fwd(_dims(rows_per_bias=3), bias=FAKE + 65536) == 1
    assert _fwd(_dims(rows_per_bias=0), bias=FAKE + 65536) == 1


def _bwd(dims, **over):
    lib = _lib()
    a = dict(q=FAKE, k=FAKE + 1 * 4096, v=FAKE + 2 * 4096, g=None, bias=None, mask=None,
             out=FAKE + 3 * 4096, lse=FAKE + 4 * 4096, dout=FAKE + 5 * 4096, dq=FAKE + 6 * 4096,
             dk=FAKE + 7 * 4096, dv=FAKE + 8 * 4096, dg=None, dbias=None, ws=FAKE + (1 << 20),
             ws_bytes=1 << 40)
    a.update(over)
    P = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.evo_attn_bwd(ctypes.byref(dims), P(a["q"]), P(a["k"]), P(a["v"]), P(a["g"]),
                            P(a["bias"]), P(a["mask"]), P(a["out"]), P(a["lse"]), P(a["dout"]),
                            P(a["dq"]), P(a["dk"]), P(a["dv"]), P(a["dg"]), P(a["dbias"]),
                            P(a["ws"]), ctypes.c_size_t(a["ws_bytes"]), None)


def test_bwd_rejects_invalid_calls():
    d = _dims()
    assert _bwd(d, dq=None) == 1
    assert _bwd(d, g=FAKE + 9 * 4096) == 1                 # gate without dgate
    assert _bwd(d, dbias=FAKE + 10 * 4096) == 1            # dbias without bias
    assert _bwd(d, dv=FAKE + 8 * 4096 + 8) == 3
    assert _bwd(_dims(seq_len=520)) == 2
    # workspace checks, on plans that need scratch: fp32 (two passes, dA and
    # Dsum in the workspace) and bf16 with a bias over many rows (partial
    # dBias planes of the single pass)
    bias = dict(bias=FAKE + 9 * 4096, dbias=FAKE + 10 * 4096)
    for dd, extra in ((_dims(dtype=0), {}), (_dims(n_rows=64, seq_len=64, rows_per_bias=64), bias)):
        assert _lib().evo_attn_bwd_workspace_size(ctypes.byref(dd)) > 256
        assert _bwd(dd, ws=None, **extra) == 4
        assert _bwd(dd, ws_bytes=16, **extra) == 4
        assert _bwd(dd, ws=FAKE + (1 << 20) + 16, **extra) == 4      # workspace not 256-byte aligned


def test_traced_backward_validates_events():
    lib = _lib()
    d = _dims()
    P = ctypes.c_void_p
    n = lib.evo_attn_bwd_kernel_count(0)
    assert n >= 1 and lib.evo_attn_bwd_kernel_count(1) >= n
    args = [ctypes.byref(d)] + [P(FAKE + i * 4096) for i in range(3)] + [None, None, None] + \
           [P(FAKE + i * 4096) for i in range(3, 9)] + [None, None, P(FAKE + (1 << 20)),
                                                        ctypes.c_size_t(1 << 40)]
    few = (P * n)(*[P(FAKE)] * n)                     # one event short
    assert lib.evo_attn_bwd_traced(*args, few, n, None) == 1
    nulls = (P * (n + 1))()                          # NULL handles
    assert lib.evo_attn_bwd_traced(*args, nulls, n + 1, None) == 1
    assert lib.evo_attn_bwd_traced(*args, None, 0, None) == 1


def test_workspace_size_is_positive_and_monotone():
    lib = _lib()
    s1 = lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(n_rows=4)))
    s2 = lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(n_rows=8, rows_per_bias=8)))
    assert 0 < s1 < s2
    assert lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(head_dim=24))) == 0
    # head_dim 64: accepted (bf16 up to 256 keys, fp32 up to 128)
    assert lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(head_dim=64, seq_len=256))) > 0
    assert lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(dtype=0, head_dim=64, seq_len=128))) > 0
    assert lib.evo_attn_bwd_workspace_size(ctypes.byref(_dims(dtype=0, head_dim=64, seq_len=136))) == 0


def test_empty_problems_need_no_pointers():
    """N == 0 or L == 0: EVO_OK without looking at any pointer."""
    lib = _lib()
    for kw in (dict(n_rows=0, rows_per_bias=1), dict(seq_len=0, stride_row=64)):
        d = _dims(**kw)
        assert lib.evo_attn_bwd_workspace_size(ctypes.byref(d)) >= 0
        assert _fwd(d, q=None, k=None, v=None, out=None, lse=None) == 0
        assert _bwd(d, q=None, k=None, v=None, out=None, lse=None, dout=None, dq=None, dk=None,
                    dv=None, ws=None, ws_bytes=0) == 0
        # with a bias the plan must not divide by the zero plane count
        assert _fwd(d, q=None, bias=None) == 0


def _bwd_noalloc(dims, **over):
    lib = _lib()
    a = dict(q=FAKE, k=FAKE + 1 * 4096, v=FAKE + 2 * 4096, g=None, bias=None, mask=None,
             out=FAKE + 3 * 4096, lse=FAKE + 4 * 4096, dout=FAKE + 5 * 4096, dq=FAKE + 6 * 4096,
             dk=FAKE + 7 * 4096, dv=FAKE + 8 * 4096, dg=None, dbias=None)
    a.update(over)
    P = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.evo_attn_bwd_noalloc(ctypes.byref(dims), P(a["q"]), P(a["k"]), P(a["v"]), P(a["g"]),
                                    P(a["bias"]), P(a["mask"]), P(a["out"]), P(a["lse"]), P(a["dout"]),
                                    P(a["dq"]), P(a["dk"]), P(a["dv"]), P(a["dg"]), P(a["dbias"]), None)


def test_noalloc_backward_validates_before_any_hip_call():
    """The no-alloc backward checks its arguments like evo_attn_bwd and refuses
    a problem whose scratch exceeds the fixed buffer with its own status, all
    before any HIP call (nothing here touches a device)."""
    lib = _lib()
    limit = lib.evo_attn_bwd_noalloc_scratch_bytes()
    assert limit == 64 << 20
    d = _dims()
    assert _bwd_noalloc(d, dq=None) == 1
    assert _bwd_noalloc(d, g=FAKE + 9 * 4096) == 1                 # gate without dgate
    assert _bwd_noalloc(d, dbias=FAKE + 10 * 4096) == 1            # dbias without bias
    assert _bwd_noalloc(d, dv=FAKE + 8 * 4096 + 8) == 3
    assert _bwd_noalloc(_dims(seq_len=520)) == 2
    # fp32, 2048 rows x 128 keys x 8 heads x 32 channels: the two-pass plan's
    # dA alone is 256 MiB
    big = _dims(dtype=0, n_rows=2048, seq_len=128, n_heads=8, rows_per_bias=2048)
    assert lib.evo_attn_bwd_workspace_size(ctypes.byref(big)) > limit
    assert _bwd_noalloc(big) == 6
    assert "no-alloc" in ea.evo_attn_strerror(6)
    # empty problems: EVO_OK without any pointer
    e = _dims(n_rows=0, rows_per_bias=1)
    assert _bwd_noalloc(e, q=None, k=None, v=None, out=None, lse=None, dout=None, dq=None, dk=None,
                        dv=None) == 0


def test_probe_exported_and_validates():
    """include/evo_probe.h: every declared symbol exported; invalid calls are
    refused before any HIP call."""
    lib = _lib()
    probe = os.path.join(ROOT, "include", "evo_probe.h")
    decls = re.findall(r"^\s*int\s+(evo_\w+)\s*\(", open(probe).read(), flags=re.M)
    assert decls == ["evo_probe_rate"]
    lib.evo_probe_rate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.evo_probe_rate.restype = ctypes.c_int
    P = ctypes.c_void_p
    assert lib.evo_probe_rate(7, 1, 1, P(FAKE), None) == 1
    assert lib.evo_probe_rate(0, 0, 1, P(FAKE), None) == 1
    assert lib.evo_probe_rate(0, 1, 0, P(FAKE), None) == 1
    assert lib.evo_probe_rate(1, 1, 1, None, None) == 1

"""GPU test of the backward entry point that allocates nothing
(evo_attn_bwd_noalloc, the library's fixed per-device scratch): through the C
ABI, its results against evo_attn_bwd's (caller workspace) on the same inputs,
on two calls in a row where the second is smaller than the first (the scratch
keeps the first call's contents, which must not leak into the second), and on
a problem whose default plan is larger than the fixed buffer (the no-alloc call
then takes fewer dBias row chunks; results within the bf16 parity bounds)."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import workloads as W
from tests.parity_util import compare, make_inputs, to_device, to_f64

pytestmark = pytest.mark.gpu

NAMES = ("dq", "dk", "dv", "dgate", "dbias")


def _inputs(x, dtype):
    dev = {n: to_device(x[n], dtype) for n in ("q", "k", "v", "gate", "bias", "dout")}
    mask = None if x["mask"] is None else torch.from_numpy(x["mask"]).cuda()
    return dev, mask


def _both(x, dtype, rpb):
    """Forward once, then the backward through both entry points; returns the
    two result dicts (fp64 numpy) and whether the default plan fits."""
    dev, mask = _inputs(x, dtype)
    args = (dev["q"], dev["k"], dev["v"], dev["gate"], dev["bias"], mask)
    out, lse = ea.evo_attn_fwd(*args, rows_per_bias=rpb)
    ref = ea.evo_attn_bwd(*args, out, lse, dev["dout"], rows_per_bias=rpb)
    # outputs preallocated, so the no-alloc call itself allocates nothing
    pre = [torch.full_like(t, float("nan")) if t is not None else None for t in ref]
    got = ea.evo_attn_bwd_noalloc(*args, out, lse, dev["dout"], rows_per_bias=rpb, dq=pre[0], dk=pre[1],
                                  dv=pre[2], dgate=pre[3], dbias=pre[4])
    torch.cuda.synchronize()
    fits = ea.evo_attn_bwd_workspace_size(dev["q"], rpb) <= ea.evo_attn_bwd_noalloc_scratch_bytes()
    conv = lambda r: {n: (None if t is None else to_f64(t)) for n, t in zip(NAMES, r)}
    return conv(ref), conv(got), fits


def _check(ref, got, fits, dtype, label):
    for n in NAMES:
        if ref[n] is None:
            assert got[n] is None, (label, n)
            continue
        assert np.isfinite(got[n]).all(), (label, n)
        if fits:  # same plan, same kernels: identical bits
            assert np.array_equal(got[n], ref[n]), (label, n)
    if not fits:
        compare(got, ref, dtype, names=[n for n in NAMES if ref[n] is not None], label=label)


def test_noalloc_matches_workspace_backward_on_two_calls():
    # first call: a 32-row slice of MSA row attention with pair bias (bf16, d=32)
    w1 = W.by_name("msa_row_bias_bf16").with_rows(32)
    x1 = W.generate(w1)
    print("\n[case] noalloc call 1: %s rows=%d" % (w1.name, w1.n_rows), flush=True)
    ref1, got1, fits1 = _both(x1, w1.dtype, w1.rows_per_bias)
    assert fits1
    _check(ref1, got1, fits1, w1.dtype, "call 1")
    # second call, smaller: 3 rows x 70 keys, head dim 16, Bernoulli mask
    w2, x2 = make_inputs(3, 70, 2, 16, "bf16", seed=77, rpb=3)
    print("[case] noalloc call 2: N=3 L=70 H=2 d=16", flush=True)
    ref2, got2, fits2 = _both(x2, "bf16", w2.rows_per_bias)
    assert fits2
    _check(ref2, got2, fits2, "bf16", "call 2")


def test_noalloc_fp32_and_no_bias():
    for (N, L, H, d, dtype, kw) in [(2, 40, 2, 32, "f32", dict()),
                                    (4, 64, 2, 8, "bf16", dict(bias=False, gate=False))]:
        w, x = make_inputs(N, L, H, d, dtype, seed=5 + L, **kw)
        print("\n[case] noalloc", (N, L, H, d, dtype, kw), flush=True)
        ref, got, fits = _both(x, dtype, w.rows_per_bias)
        _check(ref, got, fits, dtype, str((N, L, H, d, dtype)))


def test_noalloc_refuses_what_does_not_fit():
    """fp32, 2048 rows x 128 keys x 8 heads x 32 channels: the per-row scratch
    of the two-pass backward (dA, 256 MiB) is past the fixed buffer; the call
    is refused before any work is queued and the outputs are untouched."""
    N, L, H, d = 2048, 128, 8, 32
    q = torch.zeros((N, L, H, d), dtype=torch.float32, device="cuda")
    lse = torch.zeros((N, H, L), dtype=torch.float32, device="cuda")
    dq = torch.full_like(q, 3.0)
    with pytest.raises(ea.EvoAttnError) as e:
        ea.evo_attn_bwd_noalloc(q, q, q, None, None, None, q, lse, q, dq=dq, dk=dq.clone(), dv=dq.clone())
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert bool((dq == 3.0).all())

"""GPU parity of the LayerNorm kernels (through the C ABI) against the fp64 oracle.

* every LayerNorm workload at its full size, all elements of every output;
* every compiled row length in both dtypes with ragged row counts;
* edge cases: one row, no rows, constant rows (zero variance), rows with a
  large offset against their spread;
* properties: bitwise-repeatable parameter gradients, non-default stream.

Tolerances (|x - ref| <= atol + rtol |ref| element-wise, plus a normwise
bound ||x - ref|| <= norm ||ref||):
  bf16 y, dx: atol = rtol = 1e-2, norm 4e-3.  The kernel computes in fp32 and
      rounds once to bf16 (relative 2^-9 = 2e-3 per element at worst, about
      1e-3 in the norm), so 4e-3 catches any real arithmetic slip.
  fp32 y, dx: atol = rtol = 1e-5, norm 1e-5.
  mean, rstd (fp32): rtol 1e-5, atol 1e-5 * max|x|: an fp32 sum of C terms.
  dweight, dbias (fp32 sums over R rows): rtol 1e-4, atol 1e-4 * sqrt(R):
      R fp32 additions of terms of size ~1 in a fixed but different order.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2404_11068_amd import layernorm as ln
from paper_2404_11068_amd import workloads as W
from tests.parity_util import to_device, to_f64

pytestmark = pytest.mark.gpu

TOK_TOL = {"bf16": dict(atol=1e-2, rtol=1e-2, norm=4e-3), "f32": dict(atol=1e-5, rtol=1e-5, norm=1e-5)}


def _close(name, got, ref, atol, rtol, norm=None):
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), (name, "non-finite")
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    i = int(np.argmax(err - bound)) if err.size else 0
    assert (err <= bound).all(), (name, "max err %.3g at ref %.3g (bound %.3g)" %
                                  (err.flat[i], ref.flat[i], bound.flat[i]))
    if norm is not None and err.size:
        rn = np.linalg.norm(ref)
        rel = np.linalg.norm(got - ref) / rn if rn > 0 else np.linalg.norm(got - ref)
        assert rel <= norm, (name, "normwise rel err %.3g" % rel)
        return float(rel)
    return None


def run_gpu(x, dtype, eps, stream=None):
    xd = to_device(x["x"], dtype)
    dyd = to_device(x["dy"], dtype)
    w = torch.from_numpy(x["weight"]).cuda()
    b = torch.from_numpy(x["bias"]).cuda()
    y, mean, rstd = ln.layernorm_fwd(xd, w, b, eps, stream=stream)
    dx, dw, db = ln.layernorm_bwd(xd, w, mean, rstd, dyd, eps=eps, stream=stream)
    torch.cuda.synchronize()
    return {k: to_f64(v) for k, v in dict(y=y, mean=mean, rstd=rstd, dx=dx, dw=dw, db=db).items()}


def run_oracle(x, dtype, eps):
    xf = W.as_float64(x["x"], dtype)
    dyf = W.as_float64(x["dy"], dtype)
    w = x["weight"].astype(np.float64)
    b = x["bias"].astype(np.float64)
    y, mean, rstd = oracle.layernorm_forward(xf, w, b, eps)
    dx, dw, db = oracle.layernorm_backward(xf, dyf, w, eps)
    return dict(y=y, mean=mean, rstd=rstd, dx=dx, dw=dw, db=db), xf


def check(x, dtype, eps, label, stream=None):
    print("\n[case]", label, flush=True)
    got = run_gpu(x, dtype, eps, stream)
    ref, xf = run_oracle(x, dtype, eps)
    t = TOK_TOL[dtype]
    R = xf.shape[0]
    rep = {}
    for n in ("y", "dx"):
        rep[n] = _close(label + ":" + n, got[n], ref[n], t["atol"], t["rtol"], t["norm"])
    xmax = float(np.abs(xf).max()) if xf.size else 0.0
    _close(label + ":mean", got["mean"], ref["mean"], 1e-5 * max(xmax, 1.0), 1e-5)
    _close(label + ":rstd", got["rstd"], ref["rstd"], 0.0, 1e-5)
    for n in ("dw", "db"):
        _close(label + ":" + n, got[n], ref[n], 1e-4 * max(np.sqrt(R), 1.0), 1e-4)
    print("  normwise rel err y %.2e dx %.2e" % (rep["y"] or 0, rep["dx"] or 0), flush=True)
    return got


@pytest.mark.parametrize("name", [w.name for w in W.LN_WORKLOADS])
def test_full_workload(name):
    w = W.ln_by_name(name)
    check(W.generate_ln(w), w.dtype, w.eps, name)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("C", ln.LN_COLS)
@pytest.mark.parametrize("R", [1, 37, 1000])
def test_row_lengths_and_ragged_rows(dtype, C, R):
    w = W.LnWorkload("adhoc", R, C, dtype, seed=31 * C + R)
    check(W.generate_ln(w), dtype, 1e-5, "C%d_R%d_%s" % (C, R, dtype))


def test_large_offset_forward():
    # rows with mean ~1e4 and spread ~1e-2 (fp32): a sum/sum-of-squares
    # variance would lose every digit here.  Forward only: the backward reads
    # the mean saved in fp32, whose rounding (half an ulp of 1e4) is 5% of
    # this spread, so its parity is checked at a moderate offset below.
    rng = np.random.default_rng(5)
    R, C = 300, 128
    x = (1e4 + 1e-2 * rng.standard_normal((R, C))).astype(np.float32)
    w = (1.0 + 0.2 * rng.standard_normal(C)).astype(np.float32)
    b = (0.2 * rng.standard_normal(C)).astype(np.float32)
    for eps in (1e-5, 0.25):
        print("\n[case] large offset, eps", eps, flush=True)
        y, mean, rstd = ln.layernorm_fwd(torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda(),
                                         torch.from_numpy(b).cuda(), eps)
        ry, rm, rr = oracle.layernorm_forward(x.astype(np.float64), w.astype(np.float64),
                                              b.astype(np.float64), eps)
        _close("y", to_f64(y), ry, 1e-5, 1e-5, 1e-5)
        _close("mean", to_f64(mean), rm, 1e-3, 1e-7)
        _close("rstd", to_f64(rstd), rr, 0.0, 1e-5)


@pytest.mark.parametrize("eps", [1e-5, 0.25])
def test_moderate_offset_forward_backward(eps):
    rng = np.random.default_rng(6)
    R, C = 300, 256
    x = (100.0 + rng.standard_normal((R, C))).astype(np.float32)
    d = {"x": x, "dy": rng.standard_normal((R, C)).astype(np.float32),
         "weight": (1.0 + 0.2 * rng.standard_normal(C)).astype(np.float32),
         "bias": (0.2 * rng.standard_normal(C)).astype(np.float32)}
    check(d, "f32", eps, "offset-100 f32 eps=%g" % eps)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_constant_rows_give_bias(dtype):
    R, C = 50, 256
    w = W.LnWorkload("const", R, C, dtype, seed=3)
    d = W.generate_ln(w)
    d["x"] = np.repeat(d["x"][:, :1], C, axis=1)  # every row constant
    got = check(d, dtype, 1e-5, "constant rows " + dtype)
    expect = W.as_float64(W._store(np.broadcast_to(d["bias"].astype(np.float64), (R, C)), dtype), dtype)
    np.testing.assert_array_equal(got["y"], expect)


def test_empty_rows():
    x = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    w = torch.ones(128, device="cuda")
    b = torch.zeros(128, device="cuda")
    y, mean, rstd = ln.layernorm_fwd(x, w, b)
    assert y.shape == (0, 128) and mean.shape == (0,)
    dw = torch.full((128,), 7.0, device="cuda")
    db = torch.full((128,), 7.0, device="cuda")
    ln.layernorm_bwd(x, w, mean, rstd, x, dweight=dw, dbias=db)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dw).item() == 0 and torch.count_nonzero(db).item() == 0


def test_repeatable_and_stream():
    w = W.ln_by_name("ln_pair_bf16")
    d = W.generate_ln(w, n_rows=20000)
    a = run_gpu(d, w.dtype, w.eps)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = run_gpu(d, w.dtype, w.eps, stream=s)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_3d_input_and_no_stats():
    w = W.LnWorkload("adhoc", 6 * 11, 64, "bf16", seed=9)
    d = W.generate_ln(w)
    x = to_device(d["x"], "bf16").view(6, 11, 64)
    wt = torch.from_numpy(d["weight"]).cuda()
    bt = torch.from_numpy(d["bias"]).cuda()
    y, m, r = ln.layernorm_fwd(x, wt, bt, need_stats=False)
    assert m is None and r is None
    y2, _, _ = ln.layernorm_fwd(x.view(66, 64), wt, bt)
    torch.cuda.synchronize()
    assert torch.equal(y.view(66, 64), y2)

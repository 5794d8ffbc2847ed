"""Pins for the fp64 LayerNorm oracle, against things other than the oracle.

* a library routine: torch-CPU fp64 ``layer_norm`` and autograd through it
  (dx, dweight, dbias);
* a closed form worked by hand at C = 2;
* central finite differences of a random projection of the output;
* invariants the definition implies: normalised rows have mean 0 and
  variance 1 (eps = 0), invariance to x -> a x + c (a > 0, eps = 0), a
  constant row maps to the bias, every row of dx sums to 0 and is
  orthogonal to x-hat (eps = 0), and rows are independent while dweight and
  dbias add over rows.

A plausible slip (biased vs unbiased variance, eps outside the square root,
a dropped term of dx, dweight without the normalisation, a transposed
weight index) fails at least one of them.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _case(seed, R=7, C=12, scale=1.0, shift=0.0):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((R, C)) * scale + shift
    w = 1.0 + 0.5 * rng.standard_normal(C)
    b = 0.5 * rng.standard_normal(C)
    dy = rng.standard_normal((R, C))
    return x, w, b, dy


@pytest.mark.parametrize("eps", [0.0, 1e-5, 0.3])
@pytest.mark.parametrize("shape", [(7, 12), (3, 1, 5), (1, 256)])
def test_matches_torch_layer_norm(eps, shape):
    rng = np.random.default_rng(7)
    x = rng.standard_normal(shape) * 3.0 + 1.5
    C = shape[-1]
    w = rng.standard_normal(C)
    b = rng.standard_normal(C)
    dy = rng.standard_normal(shape)
    y, mean, rstd = oracle.layernorm_forward(x, w, b, eps)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    yt = F.layer_norm(xt, (C,), wt, bt, eps)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mean, x.mean(-1), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt(x.var(-1) + eps), rtol=1e-12)
    yt.backward(torch.tensor(dy))
    dx, dw, db = oracle.layernorm_backward(x, dy, w, eps)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-10)


def test_closed_form_two_channels():
    # C = 2, eps = 0: mean = (a+b)/2 and the standard deviation is |a-b|/2, so
    # x-hat = (sign(a-b), -sign(a-b)) whatever the magnitudes
    x = np.array([[3.0, 1.0], [-2.0, 5.0], [0.25, 0.5]])
    w = np.array([2.0, -3.0])
    b = np.array([0.5, 1.0])
    y, mean, rstd = oracle.layernorm_forward(x, w, b, 0.0)
    s = np.sign(x[:, 0] - x[:, 1])
    expect = np.stack([2.0 * s + 0.5, -3.0 * -s + 1.0], axis=1)
    np.testing.assert_allclose(y, expect, rtol=0, atol=1e-15)
    np.testing.assert_allclose(mean, [2.0, 1.5, 0.375], rtol=0, atol=1e-15)
    np.testing.assert_allclose(rstd, [1.0, 2.0 / 7.0, 8.0], rtol=1e-15)
    # x-hat does not depend on x at C = 2 (away from a == b), so dx = 0,
    # dweight = sum of dy * x-hat, dbias = sum of dy
    dy = np.array([[1.0, 2.0], [3.0, -1.0], [0.5, 0.5]])
    dx, dw, db = oracle.layernorm_backward(x, dy, w, 0.0)
    np.testing.assert_allclose(dx, 0.0, atol=1e-14)
    # x-hat rows: (1, -1), (-1, 1), (-1, 1)
    np.testing.assert_allclose(dw, [1.0 - 3.0 - 0.5, -2.0 - 1.0 + 0.5], atol=1e-14)
    np.testing.assert_allclose(db, [4.5, 1.5], atol=1e-14)


@pytest.mark.parametrize("eps", [0.0, 0.2])
def test_finite_differences(eps):
    x, w, b, _ = _case(3, R=3, C=5)
    proj = np.random.default_rng(4).standard_normal(x.shape)

    def f(x_, w_, b_):
        return float((oracle.layernorm_forward(x_, w_, b_, eps)[0] * proj).sum())

    dx, dw, db = oracle.layernorm_backward(x, proj, w, eps)
    h = 1e-6
    for arr, grad, idx in ((x, dx, 0), (w, dw, 1), (b, db, 2)):
        num = np.zeros_like(arr)
        it = np.nditer(arr, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            args = [x.copy(), w.copy(), b.copy()]
            args[idx][i] += h
            fp = f(*args)
            args[idx][i] -= 2 * h
            fm = f(*args)
            num[i] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_normalised_rows_and_affine_invariance():
    x, _, _, _ = _case(5, R=6, C=33, scale=4.0, shift=-7.0)
    ones, zeros = np.ones(33), np.zeros(33)
    y, _, _ = oracle.layernorm_forward(x, ones, zeros, 0.0)
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-13)
    np.testing.assert_allclose((y * y).mean(-1), 1.0, rtol=1e-13)
    y2, _, _ = oracle.layernorm_forward(2.5 * x + 11.0, ones, zeros, 0.0)
    np.testing.assert_allclose(y2, y, rtol=1e-12, atol=1e-12)


def test_constant_row_maps_to_bias():
    C = 16
    x = np.full((2, C), 3.25)
    w = np.linspace(-1, 1, C)
    b = np.linspace(5, 6, C)
    y, mean, rstd = oracle.layernorm_forward(x, w, b, 1e-5)
    np.testing.assert_allclose(y, np.broadcast_to(b, y.shape), rtol=0, atol=0)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt(1e-5), rtol=1e-15)


def test_gradient_invariants():
    x, w, b, dy = _case(9, R=5, C=24, scale=2.0, shift=3.0)
    dx, _, _ = oracle.layernorm_backward(x, dy, w, 0.0)
    xhat = (x - x.mean(-1, keepdims=True)) / x.std(-1, keepdims=True)
    np.testing.assert_allclose(dx.sum(-1), 0.0, atol=1e-12)
    np.testing.assert_allclose((dx * xhat).sum(-1), 0.0, atol=1e-12)
    # with eps > 0 the first still holds, the second no longer does
    dx2, _, _ = oracle.layernorm_backward(x, dy, w, 0.5)
    np.testing.assert_allclose(dx2.sum(-1), 0.0, atol=1e-12)
    assert np.abs((dx2 * xhat).sum(-1)).max() > 1e-3


def test_rows_independent_and_parameter_sums_add():
    x, w, b, dy = _case(11, R=6, C=10)
    y, _, _ = oracle.layernorm_forward(x, w, b, 1e-5)
    dx, dw, db = oracle.layernorm_backward(x, dy, w, 1e-5)
    dws, dbs = np.zeros(10), np.zeros(10)
    for r in range(6):
        yr, _, _ = oracle.layernorm_forward(x[r:r + 1], w, b, 1e-5)
        dxr, dwr, dbr = oracle.layernorm_backward(x[r:r + 1], dy[r:r + 1], w, 1e-5)
        np.testing.assert_array_equal(yr[0], y[r])
        np.testing.assert_array_equal(dxr[0], dx[r])
        dws += dwr
        dbs += dbr
    np.testing.assert_allclose(dw, dws, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(db, dbs, rtol=1e-13, atol=1e-13)


def test_no_affine_defaults():
    x, _, _, dy = _case(13, R=4, C=9)
    y0, _, _ = oracle.layernorm_forward(x, None, None, 1e-5)
    y1, _, _ = oracle.layernorm_forward(x, np.ones(9), np.zeros(9), 1e-5)
    np.testing.assert_array_equal(y0, y1)
    d0 = oracle.layernorm_backward(x, dy, None, 1e-5)
    d1 = oracle.layernorm_backward(x, dy, np.ones(9), 1e-5)
    for a, b_ in zip(d0, d1):
        np.testing.assert_array_equal(a, b_)

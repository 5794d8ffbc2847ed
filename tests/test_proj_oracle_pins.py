"""Pins for the oracle of the fused LayerNorm + batched projections.

* a library routine: torch-CPU fp64 layer_norm followed by torch linear,
  one call per projection;
* special cases: an identity weight returns the normalised input itself,
  rows of a permutation matrix pick its channels, a zero weight returns the
  bias;
* structure: n_proj projections equal one projection with the stacked
  weight, split; rows are independent; the output is linear in the weight.
* backward: torch-CPU fp64 autograd through layer_norm + linear; central
  finite differences; zero / linear in the upstream gradients, per-row
  channel sums of dx vanish, dbias = column sums, per-projection locality.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _case(seed, R=9, C=16, HD=8, P=4, bias=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((R, C)) * 2.0 + 0.5
    lw = 1.0 + 0.3 * rng.standard_normal(C)
    lb = 0.3 * rng.standard_normal(C)
    W = rng.standard_normal((P * HD, C)) / np.sqrt(C)
    b = rng.standard_normal(P * HD) if bias else None
    return x, lw, lb, W, b


@pytest.mark.parametrize("P,bias", [(1, False), (2, True), (4, True), (4, False)])
def test_matches_torch(P, bias):
    x, lw, lb, W, b = _case(1, P=P, bias=bias)
    outs = oracle.ln_proj_forward(x, lw, lb, W, b, n_proj=P, eps=1e-5)
    y = F.layer_norm(torch.tensor(x), (x.shape[-1],), torch.tensor(lw), torch.tensor(lb), 1e-5)
    HD = W.shape[0] // P
    for p in range(P):
        ref = F.linear(y, torch.tensor(W[p * HD:(p + 1) * HD]),
                       None if b is None else torch.tensor(b[p * HD:(p + 1) * HD]))
        np.testing.assert_allclose(outs[p], ref.numpy(), rtol=1e-12, atol=1e-12)


def test_identity_permutation_and_zero_weights():
    x, lw, lb, _, _ = _case(2, C=8)
    y, _, _ = oracle.layernorm_forward(x, lw, lb, 1e-5)
    (o,) = oracle.ln_proj_forward(x, lw, lb, np.eye(8), None, n_proj=1)
    np.testing.assert_allclose(o, y, rtol=0, atol=1e-15)
    perm = np.array([3, 0, 7, 5, 1, 2, 6, 4])
    a, b_ = oracle.ln_proj_forward(x, lw, lb, np.eye(8)[np.concatenate([perm, perm[::-1]])], None, n_proj=2)
    np.testing.assert_allclose(a, y[:, perm], rtol=0, atol=1e-15)
    np.testing.assert_allclose(b_, y[:, perm[::-1]], rtol=0, atol=1e-15)
    bias = np.arange(16.0)
    outs = oracle.ln_proj_forward(x, lw, lb, np.zeros((16, 8)), bias, n_proj=4)
    for p in range(4):
        np.testing.assert_array_equal(outs[p], np.broadcast_to(bias[4 * p:4 * p + 4], (x.shape[0], 4)))


def test_split_rows_and_linearity():
    x, lw, lb, W, b = _case(3)
    outs = oracle.ln_proj_forward(x, lw, lb, W, b, n_proj=4)
    (whole,) = oracle.ln_proj_forward(x, lw, lb, W, b, n_proj=1)
    np.testing.assert_allclose(np.concatenate(outs, axis=1), whole, rtol=1e-14, atol=1e-14)
    for r in range(x.shape[0]):
        o_r = oracle.ln_proj_forward(x[r:r + 1], lw, lb, W, b, n_proj=4)
        for p in range(4):
            # BLAS may block one row differently from many: last-bit differences only
            np.testing.assert_allclose(o_r[p][0], outs[p][r], rtol=1e-14, atol=1e-14)
    W2 = np.random.default_rng(4).standard_normal(W.shape)
    o1 = oracle.ln_proj_forward(x, lw, lb, W, None, n_proj=4)
    o2 = oracle.ln_proj_forward(x, lw, lb, W2, None, n_proj=4)
    o3 = oracle.ln_proj_forward(x, lw, lb, 2.0 * W - 3.0 * W2, None, n_proj=4)
    for p in range(4):
        np.testing.assert_allclose(o3[p], 2.0 * o1[p] - 3.0 * o2[p], rtol=1e-12, atol=1e-12)


def test_three_dim_input():
    x, lw, lb, W, b = _case(5, R=12)
    o2 = oracle.ln_proj_forward(x, lw, lb, W, b, n_proj=4)
    o3 = oracle.ln_proj_forward(x.reshape(3, 4, -1), lw, lb, W, b, n_proj=4)
    for p in range(4):
        np.testing.assert_allclose(o3[p].reshape(12, -1), o2[p], rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("P", [1, 4])
def test_backward_matches_torch_autograd(P):
    x, lw, lb, W, b = _case(6, R=11, C=16, HD=8, P=P)
    rng = np.random.default_rng(8)
    douts = [rng.standard_normal((11, 8)) for _ in range(P)]
    xt = torch.tensor(x, requires_grad=True)
    lwt = torch.tensor(lw, requires_grad=True)
    lbt = torch.tensor(lb, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    y = F.layer_norm(xt, (16,), lwt, lbt, 1e-5)
    loss = sum((F.linear(y, Wt[p * 8:(p + 1) * 8], bt[p * 8:(p + 1) * 8]) * torch.tensor(douts[p])).sum()
               for p in range(P))
    loss.backward()
    dx, dlw, dlb, dW, db = oracle.ln_proj_backward(x, lw, lb, W, douts, 1e-5)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dlw, lwt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dlb, lbt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_backward_finite_differences():
    x, lw, lb, W, b = _case(9, R=3, C=5, HD=2, P=2)
    rng = np.random.default_rng(10)
    douts = [rng.standard_normal((3, 2)) for _ in range(2)]

    def loss(x_, W_):
        outs = oracle.ln_proj_forward(x_, lw, lb, W_, b, n_proj=2)
        return sum(float((o * d).sum()) for o, d in zip(outs, douts))

    dx, _, _, dW, _ = oracle.ln_proj_backward(x, lw, lb, W, douts)
    h = 1e-6
    for arr, grad, which in ((x, dx, 0), (W, dW, 1)):
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            a1, a2 = arr.copy(), arr.copy()
            a1[i] += h
            a2[i] -= h
            num[i] = ((loss(a1, W) - loss(a2, W)) if which == 0 else (loss(x, a1) - loss(x, a2))) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_backward_structure():
    """Zero upstream gradient gives zero gradients; every gradient is linear
    in the upstream gradients; the input gradient of each row sums to zero
    over the channels (the LayerNorm removes the row mean); dbias is the
    column sum of the upstream gradient; a gradient on one projection only
    touches that projection's weight rows."""
    x, lw, lb, W, b = _case(12, R=7, C=16, HD=8, P=3)
    rng = np.random.default_rng(13)
    d1 = [rng.standard_normal((7, 8)) for _ in range(3)]
    d2 = [rng.standard_normal((7, 8)) for _ in range(3)]
    zero = oracle.ln_proj_backward(x, lw, lb, W, [np.zeros((7, 8))] * 3)
    for g in zero:
        assert np.abs(g).max() == 0.0
    g1 = oracle.ln_proj_backward(x, lw, lb, W, d1)
    g2 = oracle.ln_proj_backward(x, lw, lb, W, d2)
    g12 = oracle.ln_proj_backward(x, lw, lb, W, [2.0 * a - 3.0 * c for a, c in zip(d1, d2)])
    for a, c, ac in zip(g1, g2, g12):
        np.testing.assert_allclose(ac, 2.0 * a - 3.0 * c, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(g1[0].sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose(g1[4], np.concatenate([d.sum(axis=0) for d in d1]), rtol=1e-13, atol=1e-13)
    only1 = oracle.ln_proj_backward(x, lw, lb, W, [np.zeros((7, 8)), d1[1], np.zeros((7, 8))])
    dW = only1[3]
    assert np.abs(dW[:8]).max() == 0.0 and np.abs(dW[16:]).max() == 0.0
    assert np.abs(dW[8:16]).max() > 0.0


def test_linear_matches_torch_forward_and_autograd():
    """The linear layers (no LayerNorm) against torch linear and autograd; a
    linear layer on LN(x) is the LayerNorm variant's projection."""
    x, lw, lb, W, b = _case(30, R=9, C=16, HD=8, P=3)
    outs = oracle.linear_forward(x, W, b, n_proj=3)
    xt = torch.tensor(x, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    rng = np.random.default_rng(31)
    douts = [rng.standard_normal((9, 8)) for _ in range(3)]
    loss = 0.0
    for p in range(3):
        ref = F.linear(xt, Wt[p * 8:(p + 1) * 8], bt[p * 8:(p + 1) * 8])
        np.testing.assert_allclose(outs[p], ref.detach().numpy(), rtol=1e-12, atol=1e-12)
        loss = loss + (ref * torch.tensor(douts[p])).sum()
    loss.backward()
    dx, dW, db = oracle.linear_backward(x, W, douts)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW, Wt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)
    y, _, _ = oracle.layernorm_forward(x, lw, lb, 1e-5)
    for a, c in zip(oracle.linear_forward(y, W, b, n_proj=3), oracle.ln_proj_forward(x, lw, lb, W, b, n_proj=3)):
        np.testing.assert_allclose(a, c, rtol=1e-13, atol=1e-13)

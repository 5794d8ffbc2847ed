"""Pins for the oracle of the pair-bias projection (LayerNorm of each pair
entry, then a bias-free linear map to one value per head).

* a library routine: torch-CPU fp64 layer_norm + linear + permute;
* special cases: a one-hot weight row returns that channel of the
  normalised pair entry; a zero weight returns zeros; constant pair entries
  give the LayerNorm bias projected;
* structure: the transposed layout is the plain one with (i, j) swapped;
  batches are independent; the result is linear in the weight.
* backward: torch-CPU fp64 autograd through layer_norm + linear + permute,
  for both layouts; central finite differences; zero upstream gradient,
  linearity in it, per-entry channel sums of dz vanish, a gradient on one
  head touches only that head's weight row, and the transposed layout is the
  plain one with (i, j) swapped.
"""
import numpy as np
import torch
import torch.nn.functional as F

import oracle


def _case(seed, B=2, Li=5, Lj=7, C=12, H=3):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((B, Li, Lj, C)) * 1.5 - 0.3
    lw = 1.0 + 0.2 * rng.standard_normal(C)
    lb = 0.2 * rng.standard_normal(C)
    W = rng.standard_normal((H, C)) / np.sqrt(C)
    return z, lw, lb, W


def test_matches_torch():
    z, lw, lb, W = _case(1)
    out = oracle.pair_bias_forward(z, lw, lb, W, 1e-5)
    y = F.layer_norm(torch.tensor(z), (z.shape[-1],), torch.tensor(lw), torch.tensor(lb), 1e-5)
    ref = F.linear(y, torch.tensor(W)).permute(0, 3, 1, 2)
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-12, atol=1e-12)
    outT = oracle.pair_bias_forward(z, lw, lb, W, 1e-5, transpose=True)
    np.testing.assert_allclose(outT, ref.transpose(2, 3).numpy(), rtol=1e-12, atol=1e-12)


def test_special_weights():
    z, lw, lb, _ = _case(2, C=6, H=2)
    y, _, _ = oracle.layernorm_forward(z, lw, lb, 1e-5)
    W = np.zeros((2, 6))
    W[0, 4] = 1.0
    W[1, 1] = 1.0
    out = oracle.pair_bias_forward(z, lw, lb, W)
    np.testing.assert_allclose(out[:, 0], y[..., 4], rtol=0, atol=1e-15)
    np.testing.assert_allclose(out[:, 1], y[..., 1], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(oracle.pair_bias_forward(z, lw, lb, np.zeros((2, 6))), 0.0)
    zc = np.full((1, 3, 4, 6), 2.5)
    Wr = np.random.default_rng(3).standard_normal((2, 6))
    out = oracle.pair_bias_forward(zc, lw, lb, Wr)
    np.testing.assert_allclose(out, np.broadcast_to((Wr @ lb)[None, :, None, None], out.shape), rtol=1e-14)


def test_transpose_batches_linearity():
    z, lw, lb, W = _case(4, Li=6, Lj=6)
    out = oracle.pair_bias_forward(z, lw, lb, W)
    outT = oracle.pair_bias_forward(z, lw, lb, W, transpose=True)
    np.testing.assert_array_equal(outT, np.swapaxes(out, 2, 3))
    # transposing the pair representation instead gives the same tensor
    zt = np.ascontiguousarray(np.swapaxes(z, 1, 2))
    np.testing.assert_allclose(oracle.pair_bias_forward(zt, lw, lb, W), outT, rtol=1e-14, atol=1e-14)
    for b in range(z.shape[0]):
        np.testing.assert_allclose(oracle.pair_bias_forward(z[b:b + 1], lw, lb, W)[0], out[b],
                                   rtol=1e-14, atol=1e-14)
    W2 = np.random.default_rng(5).standard_normal(W.shape)
    np.testing.assert_allclose(oracle.pair_bias_forward(z, lw, lb, 3 * W + W2),
                               3 * out + oracle.pair_bias_forward(z, lw, lb, W2), rtol=1e-12, atol=1e-12)


def _torch_grads(z, lw, lb, W, g, transpose):
    zt = torch.tensor(z, requires_grad=True)
    lwt = torch.tensor(lw, requires_grad=True)
    lbt = torch.tensor(lb, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    y = F.layer_norm(zt, (z.shape[-1],), lwt, lbt, 1e-5)
    out = F.linear(y, Wt).permute(0, 3, 1, 2)   # [B, H, Li, Lj]
    if transpose:
        out = out.transpose(2, 3)
    (out * torch.tensor(g)).sum().backward()
    return zt.grad.numpy(), lwt.grad.numpy(), lbt.grad.numpy(), Wt.grad.numpy()


def test_backward_matches_torch_autograd():
    for transpose in (False, True):
        z, lw, lb, W = _case(21)
        B, Li, Lj, _ = z.shape
        H = W.shape[0]
        g = np.random.default_rng(22).standard_normal((B, H, Lj, Li) if transpose else (B, H, Li, Lj))
        got = oracle.pair_bias_backward(z, lw, lb, W, g, 1e-5, transpose=transpose)
        ref = _torch_grads(z, lw, lb, W, g, transpose)
        for a, r in zip(got, ref):
            np.testing.assert_allclose(a, r, rtol=1e-10, atol=1e-12)


def test_backward_finite_differences():
    z, lw, lb, W = _case(23, B=1, Li=2, Lj=3, C=5, H=2)
    g = np.random.default_rng(24).standard_normal((1, 2, 2, 3))

    def loss(z_, W_):
        return float((oracle.pair_bias_forward(z_, lw, lb, W_) * g).sum())

    dz, _, _, dW = oracle.pair_bias_backward(z, lw, lb, W, g)
    h = 1e-6
    for arr, grad, which in ((z, dz, 0), (W, dW, 1)):
        num = np.zeros_like(arr)
        for i in np.ndindex(arr.shape):
            a1, a2 = arr.copy(), arr.copy()
            a1[i] += h
            a2[i] -= h
            num[i] = ((loss(a1, W) - loss(a2, W)) if which == 0 else (loss(z, a1) - loss(z, a2))) / (2 * h)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-7)


def test_backward_structure():
    z, lw, lb, W = _case(25)
    B, Li, Lj, C = z.shape
    H = W.shape[0]
    rng = np.random.default_rng(26)
    g1 = rng.standard_normal((B, H, Li, Lj))
    g2 = rng.standard_normal((B, H, Li, Lj))
    for a in oracle.pair_bias_backward(z, lw, lb, W, np.zeros_like(g1)):
        assert np.abs(a).max() == 0.0
    r1 = oracle.pair_bias_backward(z, lw, lb, W, g1)
    r2 = oracle.pair_bias_backward(z, lw, lb, W, g2)
    r12 = oracle.pair_bias_backward(z, lw, lb, W, 2.0 * g1 - 3.0 * g2)
    for a, c, ac in zip(r1, r2, r12):
        np.testing.assert_allclose(ac, 2.0 * a - 3.0 * c, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(r1[0].sum(axis=-1), 0.0, atol=1e-12)
    one = np.zeros_like(g1)
    one[:, 1] = g1[:, 1]
    dW = oracle.pair_bias_backward(z, lw, lb, W, one)[3]
    assert np.abs(dW[0]).max() == 0.0 and np.abs(dW[2:]).max() == 0.0 and np.abs(dW[1]).max() > 0.0
    # the transposed layout: the same gradients from dbias with (i, j) swapped
    rt = oracle.pair_bias_backward(z, lw, lb, W, np.ascontiguousarray(np.swapaxes(g1, 2, 3)), transpose=True)
    for a, c in zip(r1, rt):
        np.testing.assert_allclose(a, c, rtol=1e-13, atol=1e-13)

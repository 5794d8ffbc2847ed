"""Pins for the oracle of the pair-bias projection (LayerNorm of each pair
entry, then a bias-free linear map to one value per head).

* a library routine: torch-CPU fp64 layer_norm + linear + permute;
* special cases: a one-hot weight row returns that channel of the
  normalised pair entry; a zero weight returns zeros; constant pair entries
  give the LayerNorm bias projected;
* structure: the transposed layout is the plain one with (i, j) swapped;
  batches are independent; the result is linear in the weight.
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

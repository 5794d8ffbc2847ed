"""Pins for the optimizer-step oracle (clipping, Adam, SWA).

* library routines: torch.optim.Adam (fp64, several steps, with and without
  weight decay) and torch.nn.utils.clip_grad_norm_;
* closed forms: at the first step from zero moments the Adam update is
  lr * g / (|g| + eps); SWA with decay n/(n+1) gives the running mean; a
  gradient norm below the threshold leaves the scale at 1.
"""
import numpy as np
import pytest
import torch

from oracle import optim_oracle as oo


def _tensors(seed, shapes=((7,), (3, 5), (4, 2, 3))):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(s) for s in shapes]


@pytest.mark.parametrize("wd", [0.0, 0.01])
def test_matches_torch_adam_over_steps(wd):
    ps = _tensors(1)
    gs_steps = [_tensors(10 + k) for k in range(3)]
    tp = [torch.tensor(p, requires_grad=True) for p in ps]
    opt = torch.optim.Adam(tp, lr=1e-2, betas=(0.9, 0.999), eps=1e-6, weight_decay=wd)
    m = [np.zeros_like(p) for p in ps]
    v = [np.zeros_like(p) for p in ps]
    w = [p.copy() for p in ps]
    cur = [p.copy() for p in ps]
    for t, gs in enumerate(gs_steps, start=1):
        for x, g in zip(tp, gs):
            x.grad = torch.tensor(g)
        opt.step()
        cur, m, v, w = oo.adam_swa_step(cur, gs, m, v, w, lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-6,
                                        weight_decay=wd, step=t, swa_decay=0.5)
        for a, b in zip(cur, tp):
            np.testing.assert_allclose(a, b.detach().numpy(), rtol=1e-12, atol=1e-14)
        for a, x in zip(m, tp):
            np.testing.assert_allclose(a, opt.state[x]["exp_avg"].numpy(), rtol=1e-12, atol=1e-15)
        for a, x in zip(v, tp):
            np.testing.assert_allclose(a, opt.state[x]["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-15)


def test_first_step_closed_form():
    ps, gs = _tensors(2), _tensors(3)
    z = [np.zeros_like(p) for p in ps]
    newp, m, v, _ = oo.adam_swa_step(ps, gs, z, z, ps, lr=0.1, beta1=0.8, beta2=0.99, eps=1e-3,
                                     weight_decay=0.0, step=1, swa_decay=0.0)
    for p0, g, p1 in zip(ps, gs, newp):
        np.testing.assert_allclose(p1, p0 - 0.1 * g / (np.abs(g) + 1e-3), rtol=1e-13, atol=1e-15)


def test_swa_running_mean_and_ema():
    ps = _tensors(4)
    zero = [np.zeros_like(p) for p in ps]
    w = [np.zeros_like(p) for p in ps]
    iterates = []
    cur = [p.copy() for p in ps]
    for n in range(4):
        gs = _tensors(20 + n)
        cur, m_, v_, w = oo.adam_swa_step(cur, gs, zero, zero, w, lr=0.05, beta1=0.0, beta2=0.0, eps=1.0,
                                          weight_decay=0.0, step=1, swa_decay=n / (n + 1.0))
        iterates.append(cur)
    for k in range(len(ps)):
        np.testing.assert_allclose(w[k], np.mean([it[k] for it in iterates], axis=0), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("max_norm", [0.1, 1e6])
def test_clip_scale_matches_torch(max_norm):
    gs = _tensors(5)
    tp = [torch.zeros(g.shape, dtype=torch.float64, requires_grad=True) for g in gs]
    for x, g in zip(tp, gs):
        x.grad = torch.tensor(g)
    total = torch.nn.utils.clip_grad_norm_(tp, max_norm)
    norm, scale = oo.grad_norm_scale(gs, max_norm)
    assert abs(norm - float(total)) <= 1e-12 * norm
    for x, g in zip(tp, gs):
        np.testing.assert_allclose(x.grad.numpy(), g * scale, rtol=1e-12, atol=1e-15)
    if max_norm > norm:
        assert scale == 1.0

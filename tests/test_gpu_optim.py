"""GPU parity of the fused optimizer step (gradient-norm clipping, Adam, SWA;
through the C ABI) against the fp64 oracle, over several steps.

* a parity-size subset of the AlphaFold-shaped parameter list (136 tensors,
  2.7M elements) and hand-picked sizes around the chunk length (1, 3, 4095,
  4096, 4097, 10001 elements), one tensor misaligned (a view offset by one
  element, which takes the element-by-element path), one without SWA;
* clipping active (max_norm below the gradient norm) and inactive;
* weight decay on and off; repeatable results.

Tolerance: the kernel works in fp32 from the same fp32 inputs as the fp64
oracle, so each value is off by a few fp32 roundings of itself:
|x - ref| <= 2e-6 |ref| element-wise for p, m, v and SWA after 3
steps, plus 8 fp32 roundings (8 * 2^-24) of the tensor's largest magnitude
for values that passed through larger intermediates; norm and scale within
1e-5 relative (fp32 per-chunk sums).
"""
import numpy as np
import pytest
import torch

from oracle import optim_oracle as oo
from paper_2404_11068_amd import optim as op
from paper_2404_11068_amd import workloads as W

pytestmark = pytest.mark.gpu


def _close(name, got, ref, rtol=2e-6):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref)
    # a value that passed through larger intermediates (a parameter crossing
    # zero) carries their fp32 roundings: allow 8 roundings at the tensor's
    # largest magnitude on top of the relative bound
    atol = 8 * 2.0 ** -24 * (float(np.abs(ref).max()) if ref.size else 0.0)
    bound = atol + rtol * np.abs(ref)
    i = int(np.argmax(err - bound)) if err.size else 0
    assert (err <= bound).all(), (name, "err %.3g at ref %.3g" % (err.flat[i], ref.flat[i]))


def _run(d, *, steps, max_norm, wd, swa_decay, misalign=None, no_swa=None):
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    P = [dev(a) for a in d["params"]]
    G = [dev(a) for a in d["grads"]]
    M = [dev(a) for a in d["exp_avg"]]
    V = [dev(a) for a in d["exp_avg_sq"]]
    S = [dev(a) for a in d["swa"]]
    if misalign is not None:  # same values, stored one element into a fresh allocation
        for lst in (P, G, M, V, S):
            base = torch.empty(lst[misalign].numel() + 1, dtype=torch.float32, device="cuda")
            base[1:].copy_(lst[misalign].reshape(-1))
            lst[misalign] = base[1:].view(lst[misalign].shape)
            assert lst[misalign].data_ptr() % 16 != 0
    opt = op.FusedAdamSWA(P, G, M, V, S, lr=1e-3, betas=(0.9, 0.999), eps=1e-6, weight_decay=wd,
                          swa_decay=swa_decay)
    if no_swa is not None:  # rebuild with that tensor's SWA pointer removed from the table
        import ctypes
        tab = (op.evo_mt_tensor * len(P)).from_buffer_copy(bytes(opt.tensor_table.cpu().numpy()))
        tab[no_swa].swa = None
        opt.tensor_table = torch.frombuffer(bytearray(bytes(tab)), dtype=torch.uint8).cuda()
    p = [a.astype(np.float64) for a in d["params"]]
    m = [a.astype(np.float64) for a in d["exp_avg"]]
    v = [a.astype(np.float64) for a in d["exp_avg_sq"]]
    w = [a.astype(np.float64) for a in d["swa"]]
    for t in range(1, steps + 1):
        opt.step(max_norm=max_norm, step=t + 4)
        torch.cuda.synchronize()
        scale = 1.0
        if max_norm is not None:
            norm, scale = oo.grad_norm_scale(d["grads"], max_norm)
            assert abs(opt.norm.item() - norm) <= 1e-5 * norm
            assert abs(opt.scale.item() - scale) <= 1e-5 * scale
            scale = float(opt.scale.item())  # the kernel's own fp32 scale, as the step used it
        w_prev = w
        p, m, v, w = oo.adam_swa_step(p, d["grads"], m, v, w, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-6,
                                      weight_decay=wd, step=t + 4, swa_decay=swa_decay, grad_scale=scale)
        if no_swa is not None:
            w[no_swa] = w_prev[no_swa]
    for k in range(len(P)):
        _close("p%d" % k, P[k].cpu().numpy(), p[k])
        _close("m%d" % k, M[k].cpu().numpy(), m[k])
        _close("v%d" % k, V[k].cpu().numpy(), v[k])
        _close("w%d" % k, S[k].cpu().numpy(), w[k])
    return opt


@pytest.mark.parametrize("max_norm,wd", [(0.01, 0.0), (None, 0.01), (1e9, 0.0)])
def test_alphafold_subset(max_norm, wd):
    w = W.optim_by_name("adam_swa_small")
    print("\n[case] adam_swa_small max_norm=%s wd=%s" % (max_norm, wd), flush=True)
    _run(W.generate_optim(w), steps=3, max_norm=max_norm, wd=wd, swa_decay=0.999)


def test_chunk_edges_misaligned_and_no_swa():
    rng = np.random.default_rng(3)
    sizes = [1, 3, 4095, 4096, 4097, 10001, 8192, 7]
    d = {"params": [rng.standard_normal(n).astype(np.float32) for n in sizes],
         "grads": [rng.standard_normal(n).astype(np.float32) * np.float32(1e-2) for n in sizes],
         "exp_avg": [np.zeros(n, np.float32) for n in sizes],
         "exp_avg_sq": [np.zeros(n, np.float32) for n in sizes],
         "swa": [rng.standard_normal(n).astype(np.float32) for n in sizes]}
    print("\n[case] chunk edges", flush=True)
    _run(d, steps=3, max_norm=0.05, wd=0.0, swa_decay=0.5, misalign=5, no_swa=2)


def test_repeatable():
    w = W.optim_by_name("adam_swa_small")
    d = W.generate_optim(w)
    outs = []
    for _ in range(2):
        P = [torch.from_numpy(a).cuda() for a in d["params"]]
        opt = op.FusedAdamSWA(P, [torch.from_numpy(a).cuda() for a in d["grads"]])
        opt.step(max_norm=0.01)
        torch.cuda.synchronize()
        outs.append((torch.cat([p.reshape(-1) for p in P]).cpu(), opt.norm.item()))
    assert torch.equal(outs[0][0], outs[1][0]) and outs[0][1] == outs[1][1]

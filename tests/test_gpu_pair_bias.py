"""GPU parity of the pair-bias kernel (LayerNorm of pair entries projected to
per-head logit biases, through the C ABI) against the fp64 oracle.

* every pair-bias workload at full size (plain and transposed layouts);
* every compiled channel count and head count, non-square and ragged
  (non-multiple-of-32) lengths, batches, with and without statistics;
* the output feeds the attention's bias argument directly.

Tolerance: |x - ref| <= 1e-2 + 1e-2 |ref| and ||x - ref|| <= 5e-3 ||ref||
(the normalised entry is rounded to bf16 before the dot products, and the
result once more; see the projection tests for the budget).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2404_11068_amd import proj as pj
from paper_2404_11068_amd import workloads as W
from tests.parity_util import to_device, to_f64

pytestmark = pytest.mark.gpu


def run(w, d, label, stats=False):
    print("\n[case]", label, flush=True)
    z = to_device(d["z"], "bf16")
    res = pj.ln_pair_bias_fwd(z, torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda(),
                              to_device(d["weight"], "bf16"), w.eps, w.transpose, need_stats=stats)
    out = res[0] if stats else res
    torch.cuda.synchronize()
    zf = W.as_float64(d["z"], "bf16")
    ref = oracle.pair_bias_forward(zf, d["ln_weight"], d["ln_bias"], W.as_float64(d["weight"], "bf16"), w.eps,
                                   transpose=w.transpose)
    got = to_f64(out)
    assert got.shape == ref.shape
    err = np.abs(got - ref)
    assert (err <= 1e-2 + 1e-2 * np.abs(ref)).all(), (label, float(err.max()))
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rel <= 5e-3, (label, rel)
    if stats:
        _, rm, rr = oracle.layernorm_forward(zf, None, None, w.eps)
        np.testing.assert_allclose(to_f64(res[1]), rm, rtol=1e-5, atol=1e-5 * max(np.abs(zf).max(), 1.0))
        np.testing.assert_allclose(to_f64(res[2]), rr, rtol=1e-5)
    print("  normwise rel err %.2e" % rel, flush=True)
    return out


@pytest.mark.parametrize("name", [w.name for w in W.PAIR_BIAS_WORKLOADS])
def test_full_workload(name):
    w = W.pair_bias_by_name(name)
    run(w, W.generate_pair_bias(w), name, stats=True)


CASES = [
    # B, Li, Lj (via seq_len square unless noted), C, H, transpose
    (1, 8, 8, 64, 1, False),
    (2, 40, 72, 128, 2, True),
    (1, 24, 16, 256, 16, False),
    (3, 16, 48, 64, 4, True),
    (1, 104, 8, 128, 8, False),
    (1, 8, 104, 256, 8, True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "B%d_%dx%d_C%d_H%d_T%d" % c)
def test_shapes(case):
    B, Li, Lj, C, H, tr = case
    w = W.PairBiasWorkload("adhoc", B, Li, C, H, transpose=tr, seed=Li * 7 + Lj)
    rng = np.random.default_rng(Li + 3 * Lj + C + H)
    z = rng.standard_normal((B, Li, Lj, C)) * 1.7 + 0.4
    d = {"z": W._store(z, "bf16"), "ln_weight": (1 + 0.2 * rng.standard_normal(C)).astype(np.float32),
         "ln_bias": (0.2 * rng.standard_normal(C)).astype(np.float32),
         "weight": W._store(rng.standard_normal((H, C)) / np.sqrt(C), "bf16")}
    run(w, d, str(case), stats=(H % 2 == 0))


def test_feeds_attention():
    from paper_2404_11068_amd import evo_attn as ea
    w = W.pair_bias_by_name("pb_tri_start_bf16")
    d = W.generate_pair_bias(w)
    bias = pj.ln_pair_bias_fwd(to_device(d["z"], "bf16"), torch.from_numpy(d["ln_weight"]).cuda(),
                               torch.from_numpy(d["ln_bias"]).cuda(), to_device(d["weight"], "bf16"))
    N, L, H, dh = 4, 256, 4, 32
    q = torch.randn(N, L, H, dh, device="cuda", dtype=torch.bfloat16)
    out, lse = ea.evo_attn_fwd(q, q, q, None, bias, None, rows_per_bias=N)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()

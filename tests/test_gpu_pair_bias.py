"""GPU parity of the pair-bias kernel (LayerNorm of pair entries projected to
per-head logit biases, through the C ABI) against the fp64 oracle.

* every pair-bias workload at full size (plain and transposed layouts);
* every compiled channel count and head count, non-square and ragged
  (non-multiple-of-32) lengths, batches, with and without statistics;
* the output feeds the attention's bias argument directly;
* the backward (dz, dweight, dln_weight, dln_bias from an fp32 dbias in either
  layout) on the same workloads and shapes, repeatable to the bit, and fed by
  the attention backward's dbias.

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



# ---- backward ---------------------------------------------------------------
# Tolerances: dweight, dln_weight, dln_bias are fp32 sums over every pair
# entry of products of fp32 values (normalised input recomputed in fp32):
# normwise 1e-4 and element-wise 1e-4 max|ref| + 1e-3 |ref|.  dz is fp32 up
# to the final bf16 rounding (2^-9 relative): element-wise 2^-8 |ref| + 1e-3
# max|ref| of its entry's channels, normwise 5e-3.

def run_bwd(B, Li, Lj, C, H, transpose, d, label, eps=1e-5):
    print("\n[case] bwd", label, flush=True)
    rng = np.random.default_rng(B * 131 + Li * 17 + Lj * 3 + C + H)
    shape = (B, H, Lj, Li) if transpose else (B, H, Li, Lj)
    g = rng.standard_normal(shape).astype(np.float32)
    z = to_device(d["z"], "bf16")
    lw, lb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    Wt = to_device(d["weight"], "bf16")
    dz, dW, dlw, dlb = pj.ln_pair_bias_bwd(z, lw, lb, Wt, torch.from_numpy(g).cuda(), eps, transpose)
    torch.cuda.synchronize()
    zf = W.as_float64(d["z"], "bf16")
    rdz, rdlw, rdlb, rdW = oracle.pair_bias_backward(zf, d["ln_weight"], d["ln_bias"],
                                                    W.as_float64(d["weight"], "bf16"), g.astype(np.float64), eps,
                                                    transpose=transpose)
    for nm, got, ref in (("dW", to_f64(dW), rdW), ("dln_w", to_f64(dlw), rdlw), ("dln_b", to_f64(dlb), rdlb)):
        assert got.shape == ref.shape, nm
        err = np.abs(got - ref)
        m = np.abs(ref).max()
        assert (err <= 1e-4 * m + 1e-3 * np.abs(ref)).all(), (label, nm, float(err.max()), float(m))
        rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
        assert rel <= 1e-4, (label, nm, rel)
    gdz = to_f64(dz).reshape(rdz.shape)
    err = np.abs(gdz - rdz)
    bound = 2.0 ** -8 * np.abs(rdz) + 1e-3 * np.abs(rdz).max(axis=-1, keepdims=True)
    assert (err <= bound + 1e-30).all(), (label, "dz", float((err - bound).max()))
    rel = np.linalg.norm(gdz - rdz) / np.linalg.norm(rdz)
    assert rel <= 5e-3, (label, "dz", rel)
    print("  dz normwise rel err %.2e" % rel, flush=True)
    return dz, dW, dlw, dlb


@pytest.mark.parametrize("name", [w.name for w in W.PAIR_BIAS_WORKLOADS])
def test_backward_full_workload(name):
    w = W.pair_bias_by_name(name)
    d = W.generate_pair_bias(w)
    B, Li, Lj, C = d["z"].shape
    run_bwd(B, Li, Lj, C, w.n_heads, w.transpose, d, name, w.eps)


BWD_CASES = [
    # B, Li, Lj, C, H, transpose
    (1, 8, 8, 64, 1, False),
    (2, 40, 72, 128, 2, True),
    (3, 16, 48, 64, 4, True),
    (1, 104, 8, 128, 8, False),
    (1, 8, 104, 256, 8, True),
    (1, 24, 40, 256, 4, False),
    (2, 16, 200, 64, 8, False),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: "B%d_%dx%d_C%d_H%d_T%d" % c)
def test_backward_shapes(case):
    B, Li, Lj, C, H, tr = case
    rng = np.random.default_rng(Li + 5 * Lj + C + H)
    z = rng.standard_normal((B, Li, Lj, C)) * 1.7 + 0.4
    d = {"z": W._store(z, "bf16"), "ln_weight": (1 + 0.2 * rng.standard_normal(C)).astype(np.float32),
         "ln_bias": (0.2 * rng.standard_normal(C)).astype(np.float32),
         "weight": W._store(rng.standard_normal((H, C)) / np.sqrt(C), "bf16")}
    run_bwd(B, Li, Lj, C, H, tr, d, str(case))


def test_backward_repeatable():
    w = W.pair_bias_by_name("pb_msa_row_bf16")
    d = W.generate_pair_bias(w)
    z = to_device(d["z"], "bf16")
    lw, lb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    Wt = to_device(d["weight"], "bf16")
    B, Li, Lj, _ = d["z"].shape
    g = torch.randn(B, w.n_heads, Li, Lj, generator=torch.Generator().manual_seed(3)).cuda()
    a = pj.ln_pair_bias_bwd(z, lw, lb, Wt, g, w.eps)
    b = pj.ln_pair_bias_bwd(z, lw, lb, Wt, g, w.eps)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)


def test_backward_fed_by_attention():
    """The attention backward's dbias [B, H, L, L] (fp32) is the pair-bias
    backward's input as it stands; the chained result matches the oracle's
    pair-bias backward of that same dbias."""
    from paper_2404_11068_amd import evo_attn as ea
    w = W.pair_bias_by_name("pb_tri_start_bf16")
    d = W.generate_pair_bias(w)
    z = to_device(d["z"], "bf16")
    lw, lb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    Wt = to_device(d["weight"], "bf16")
    bias = pj.ln_pair_bias_fwd(z, lw, lb, Wt, w.eps)
    N, L, H, dh = 4, 256, w.n_heads, 32
    gen = torch.Generator().manual_seed(5)
    q, k, v, do = [torch.randn(N, L, H, dh, generator=gen).to(torch.bfloat16).cuda() for _ in range(4)]
    out, lse = ea.evo_attn_fwd(q, k, v, None, bias, None, rows_per_bias=N)
    dbias = ea.evo_attn_bwd(q, k, v, None, bias, None, out, lse, do, rows_per_bias=N)[4]
    assert dbias.dtype == torch.float32 and tuple(dbias.shape) == (1, H, L, L)
    dz, dW, dlw, dlb = pj.ln_pair_bias_bwd(z, lw, lb, Wt, dbias, w.eps)
    torch.cuda.synchronize()
    rdz, rdlw, rdlb, rdW = oracle.pair_bias_backward(W.as_float64(d["z"], "bf16"), d["ln_weight"], d["ln_bias"],
                                                    W.as_float64(d["weight"], "bf16"), to_f64(dbias), w.eps)
    for nm, got, ref in (("dW", to_f64(dW), rdW), ("dz", to_f64(dz).reshape(rdz.shape), rdz)):
        rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert rel <= 5e-3, (nm, rel)

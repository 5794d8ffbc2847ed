"""GPU parity of the fused LayerNorm + batched projections (through the C ABI)
against the fp64 oracle (LayerNorm then one matmul per projection).

* every projection workload at full size, all outputs, all elements;
* every compiled input width with ragged token counts, several projection
  widths and counts, with and without bias and statistics;
* the outputs feed the attention directly ([R, HD] == [N, L, H, d]).

Tolerance (bf16 outputs): |x - ref| <= 1e-2 + 1e-2 |ref| element-wise and
||x - ref|| <= 5e-3 ||ref||.  The kernel rounds the normalised input to bf16
before the products (relative 2^-9 per element, about 2e-3 of the output
norm after the sum over C) and rounds the outputs once more (2^-9); 5e-3
leaves room for both and still fails on any real slip.
Statistics: as for the stand-alone LayerNorm (rtol 1e-5).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2404_11068_amd import proj as pj
from paper_2404_11068_amd import workloads as W
from tests.parity_util import to_device, to_f64

pytestmark = pytest.mark.gpu


def _check(name, got, ref, atol=1e-2, rtol=1e-2, norm=5e-3):
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), name
    err = np.abs(got - ref)
    bound = atol + rtol * np.abs(ref)
    i = int(np.argmax(err - bound))
    assert (err <= bound).all(), (name, "max err %.3g at ref %.3g" % (err.flat[i], ref.flat[i]))
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    assert rel <= norm, (name, "normwise rel err %.3g" % rel)
    return rel


def run_case(w, d, label, stats=True):
    print("\n[case]", label, flush=True)
    x = to_device(d["x"], "bf16")
    Wt = to_device(d["weight"], "bf16")
    lnw, lnb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    b = None if d["bias"] is None else torch.from_numpy(d["bias"]).cuda()
    res = pj.ln_proj_fwd(x, lnw, lnb, Wt, b, n_proj=w.n_proj, eps=w.eps, need_stats=stats)
    outs, mean, rstd = res if stats else (res, None, None)
    torch.cuda.synchronize()
    xf = W.as_float64(d["x"], "bf16")
    ref = oracle.ln_proj_forward(xf, d["ln_weight"], d["ln_bias"], W.as_float64(d["weight"], "bf16"),
                                 d["bias"], n_proj=w.n_proj, eps=w.eps)
    worst = 0.0
    for p in range(w.n_proj):
        worst = max(worst, _check("%s out%d" % (label, p), to_f64(outs[p]), ref[p]))
    if stats:
        _, rm, rr = oracle.layernorm_forward(xf, None, None, w.eps)
        np.testing.assert_allclose(to_f64(mean), rm, rtol=1e-5, atol=1e-5 * max(np.abs(xf).max(), 1.0))
        np.testing.assert_allclose(to_f64(rstd), rr, rtol=1e-5)
    print("  worst normwise rel err %.2e" % worst, flush=True)


@pytest.mark.parametrize("name", [w.name for w in W.PROJ_WORKLOADS])
def test_full_workload(name):
    w = W.proj_by_name(name)
    run_case(w, W.generate_proj(w), name)


CASES = [
    # R, C, HD, P, bias, stats
    (1, 64, 32, 1, False, True),
    (33, 64, 64, 4, True, True),
    (100, 128, 96, 3, True, False),
    (1000, 128, 128, 4, False, True),
    (77, 256, 256, 4, True, True),
    (513, 256, 32, 2, True, True),
    (64, 256, 1024, 1, False, False),
    (129, 64, 160, 4, True, True),
    (4096, 256, 256, 4, True, True),    # fewer token tiles than CUs: features split over workgroups
    (300, 128, 128, 4, False, True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "R%d_C%d_HD%d_P%d_b%d_s%d" % c)
def test_shapes(case):
    R, C, HD, P, bias, stats = case
    w = W.ProjWorkload("adhoc", R, C, HD, n_proj=P, bias=bias, seed=R + C + HD)
    run_case(w, W.generate_proj(w), str(case), stats=stats)


def test_feeds_attention_layout():
    # q, k, v, g for an MSA-row shaped attention come out as [N, L, H, d]
    from paper_2404_11068_amd import evo_attn as ea
    N, L, H, d, C = 4, 64, 8, 32, 256
    w = W.ProjWorkload("adhoc", N * L, C, H * d, seed=5)
    dd = W.generate_proj(w)
    x = to_device(dd["x"], "bf16").view(N, L, C)
    q, k, v, g = pj.ln_proj_fwd(x, torch.from_numpy(dd["ln_weight"]).cuda(),
                                torch.from_numpy(dd["ln_bias"]).cuda(), to_device(dd["weight"], "bf16"),
                                torch.from_numpy(dd["bias"]).cuda(), n_proj=4)
    assert q.shape == (N, L, H * d)
    out, lse = ea.evo_attn_fwd(*(t.view(N, L, H, d) for t in (q, k, v, g)))
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()


def test_empty():
    x = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    Wt = torch.zeros((4 * 64, 128), dtype=torch.bfloat16, device="cuda")
    one, zero = torch.ones(128, device="cuda"), torch.zeros(128, device="cuda")
    outs = pj.ln_proj_fwd(x, one, zero, Wt, None, n_proj=4)
    assert all(o.shape == (0, 64) for o in outs)


# ---- backward ---------------------------------------------------------------
# Tolerances: dx (bf16): per element 4 x the shift the bf16 rounding of dY
# can cause (2^-9 rstd times |w dY| plus the row means of |w dY| and
# |w dY xhat| |xhat|) plus 2^-8 |ref|, and 1e-2 normwise; dweight (fp32 sums over R
# tokens of products whose y factor was rounded to bf16): normwise 5e-3 and
# element-wise 5e-3|ref| + 5e-3 max|ref|; dbias (exact bf16 inputs, fp32
# sums): 1e-5 relative + 1e-5 max; dln_weight, dln_bias (sums of bf16-rounded
# dY terms): normwise 5e-3, element-wise 1e-2|ref| + 5e-3 max|ref|.


def run_bwd(w, d, label, seed=0):
    print("\n[case] bwd", label, flush=True)
    x = to_device(d["x"], "bf16")
    Wt = to_device(d["weight"], "bf16")
    lnw, lnb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    b = None if d["bias"] is None else torch.from_numpy(d["bias"]).cuda()
    y = torch.empty_like(x)
    outs, mean, rstd = pj.ln_proj_fwd(x, lnw, lnb, Wt, b, n_proj=w.n_proj, eps=w.eps, need_stats=True, y_norm=y)
    rng = np.random.default_rng(seed + 17)
    douts_np = [W._store(rng.standard_normal((w.n_rows, w.proj_dim)), "bf16") for _ in range(w.n_proj)]
    douts = [to_device(a, "bf16") for a in douts_np]
    dx, dW, db, dlw, dlb = pj.ln_proj_bwd(x, lnw, mean, rstd, y, Wt, douts, eps=w.eps, has_bias=b is not None)
    torch.cuda.synchronize()
    ref = oracle.ln_proj_backward(W.as_float64(d["x"], "bf16"), d["ln_weight"], d["ln_bias"],
                                  W.as_float64(d["weight"], "bf16"), [W.as_float64(a, "bf16") for a in douts_np],
                                  w.eps)
    rdx, rdlw, rdlb, rdW, rdb = ref
    # dx: the kernel rounds dY to bf16 before the LayerNorm backward, which
    # moves dx[r, c] by up to rstd_r |w_c| |dY_rc| 2^-9 whatever the size of
    # dx itself; allow 4x that per element plus the output's own rounding
    xf = W.as_float64(d["x"], "bf16")
    _, _, rrstd = oracle.layernorm_forward(xf, None, None, w.eps)
    Wf = W.as_float64(d["weight"], "bf16")
    HD = w.proj_dim
    dY = sum(W.as_float64(douts_np[p_], "bf16") @ Wf[p_ * HD:(p_ + 1) * HD] for p_ in range(w.n_proj))
    # (the row means of g = w dY and g xhat in the LayerNorm backward carry
    # the same relative rounding, averaged over the row)
    _, rmean, _ = oracle.layernorm_forward(xf, None, None, w.eps)
    xhat = (xf - rmean[:, None]) * rrstd[:, None]
    g = np.abs(d["ln_weight"])[None, :] * np.abs(dY)
    row = g.mean(axis=1)[:, None] + np.abs(xhat) * (g * np.abs(xhat)).mean(axis=1)[:, None]
    bound = 4 * 2.0 ** -9 * rrstd[:, None] * (g + row) + 2.0 ** -8 * np.abs(rdx)
    gdx = to_f64(dx).reshape(rdx.shape)
    err = np.abs(gdx - rdx)
    i = int(np.argmax(err - bound - 1e-6))
    assert (err <= bound + 1e-6).all(), (label, "dx err %.3g at ref %.3g (bound %.3g)" %
                                         (err.flat[i], rdx.flat[i], bound.flat[i]))
    rel = np.linalg.norm(gdx - rdx) / np.linalg.norm(rdx)
    assert rel <= 1e-2, (label, "dx normwise %.3g" % rel)
    m = np.abs(rdW).max()
    _check(label + " dW", to_f64(dW), rdW, atol=5e-3 * m, rtol=5e-3, norm=5e-3)
    if db is not None:
        _check(label + " dbias", to_f64(db), rdb, atol=1e-5 * np.abs(rdb).max(), rtol=1e-5, norm=1e-5)
    for nm, g, r in (("dln_w", dlw, rdlw), ("dln_b", dlb, rdlb)):
        _check(label + " " + nm, to_f64(g), r, atol=5e-3 * np.abs(r).max(), rtol=1e-2, norm=5e-3)
    # the saved normalised input is the forward's bf16 LayerNorm
    yref, _, _ = oracle.layernorm_forward(W.as_float64(d["x"], "bf16"), d["ln_weight"], d["ln_bias"], w.eps)
    _check(label + " y", to_f64(y), yref, norm=5e-3)


@pytest.mark.parametrize("name", [w.name for w in W.PROJ_WORKLOADS])
def test_backward_full_workload(name):
    w = W.proj_by_name(name)
    run_bwd(w, W.generate_proj(w), name)


BWD_CASES = [
    # R, C, HD, P, bias
    (1, 64, 32, 1, False),
    (77, 256, 256, 4, True),
    (300, 128, 96, 3, True),
    (1000, 64, 64, 4, True),
    (129, 64, 160, 2, False),
    (4100, 256, 32, 4, True),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: "R%d_C%d_HD%d_P%d_b%d" % c)
def test_backward_shapes(case):
    R, C, HD, P, bias = case
    w = W.ProjWorkload("adhoc", R, C, HD, n_proj=P, bias=bias, seed=R + 3 * C + HD)
    run_bwd(w, W.generate_proj(w), str(case), seed=R)


def test_backward_repeatable():
    w = W.ProjWorkload("adhoc", 3000, 128, 128, seed=4)
    d = W.generate_proj(w)
    x = to_device(d["x"], "bf16")
    Wt = to_device(d["weight"], "bf16")
    lnw, lnb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    y = torch.empty_like(x)
    _, mean, rstd = pj.ln_proj_fwd(x, lnw, lnb, Wt, None, n_proj=4, need_stats=True, y_norm=y)
    douts = [torch.randn(3000, 128, device="cuda").to(torch.bfloat16) for _ in range(4)]
    a = pj.ln_proj_bwd(x, lnw, mean, rstd, y, Wt, douts)
    b = pj.ln_proj_bwd(x, lnw, mean, rstd, y, Wt, douts)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


# ---- linear layers without the LayerNorm (the output projection) -------------
# Tolerances: forward as the LayerNorm variant (bf16 inputs are exact, the
# output is rounded once); dx is dY rounded to bf16 once: |err| <= 2^-8 |ref|
# + 1e-3 max|ref| of its row, 5e-3 normwise; dweight and dbias are fp32 sums of
# exact bf16 products: 1e-4 normwise, 1e-4 max|ref| + 1e-4 |ref| per element.

LINEAR_CASES = [
    # R, C, HD, P, bias  (the first three: the output projections of the MSA
    # row, triangle and extra-MSA attention workloads: C = H * d -> c_out)
    (32768, 256, 256, 1, True),
    (65536, 128, 128, 1, True),
    (262144, 64, 64, 1, True),
    (77, 256, 64, 2, False),
    (1000, 128, 96, 3, True),
    (4100, 64, 32, 4, True),
]


@pytest.mark.parametrize("case", LINEAR_CASES, ids=lambda c: "R%d_C%d_HD%d_P%d_b%d" % c)
def test_linear_forward_backward(case):
    R, C, HD, P, bias = case
    print("\n[case] linear", case, flush=True)
    rng = np.random.default_rng(R + C + HD + P)
    x_np = W._store(rng.standard_normal((R, C)), "bf16")
    w_np = W._store(rng.standard_normal((P * HD, C)) / np.sqrt(C), "bf16")
    b_np = rng.standard_normal(P * HD).astype(np.float32) if bias else None
    x, Wt = to_device(x_np, "bf16"), to_device(w_np, "bf16")
    b = torch.from_numpy(b_np).cuda() if bias else None
    outs = pj.linear_fwd(x, Wt, b, n_proj=P)
    douts_np = [W._store(rng.standard_normal((R, HD)), "bf16") for _ in range(P)]
    douts = [to_device(a, "bf16") for a in douts_np]
    dx, dW, db = pj.linear_bwd(x, Wt, douts, has_bias=bias)
    torch.cuda.synchronize()
    xf, wf = W.as_float64(x_np, "bf16"), W.as_float64(w_np, "bf16")
    # the full-size cases are checked on a sample of 2048 rows (the oracle's
    # cost grows with R; the rows cover every workgroup position and the tail)
    rows = np.unique(np.concatenate([np.linspace(0, R - 1, 1024).astype(int),
                                     rng.integers(0, R, 1024)])) if R > 8192 else np.arange(R)
    ref = oracle.linear_forward(xf[rows], wf, b_np, n_proj=P)
    for p in range(P):
        _check("linear out%d" % p, to_f64(outs[p])[rows], ref[p])
    dfs = [W.as_float64(a, "bf16") for a in douts_np]
    rdx, rdW, rdb = oracle.linear_backward(xf, wf, dfs)
    gdx = to_f64(dx)
    err = np.abs(gdx[rows] - rdx[rows])
    bound = 2.0 ** -8 * np.abs(rdx[rows]) + 1e-3 * np.abs(rdx[rows]).max(axis=1, keepdims=True)
    assert (err <= bound + 1e-30).all(), ("dx", float((err - bound).max()))
    assert np.linalg.norm(gdx - rdx) / np.linalg.norm(rdx) <= 5e-3
    _check("linear dW", to_f64(dW), rdW, atol=1e-4 * np.abs(rdW).max(), rtol=1e-4, norm=1e-4)
    if bias:
        _check("linear db", to_f64(db), rdb, atol=1e-5 * np.abs(rdb).max(), rtol=1e-5, norm=1e-5)
    else:
        assert db is None

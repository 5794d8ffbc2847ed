"""End-to-end check of one whole MSA-row attention module step on the GPU
(the graphed step: LayerNorm + q/k/v/g projections, LayerNorm(z) + pair bias,
gated attention with the pair bias, output projection, and the backward of
every stage) against the fp64 oracles composed the same way.

Each stage has its own parity tests; this one checks the interfaces between
them: the projection outputs read as [N, L, H, d] tokens, the pair bias in
the attention's bias layout, the attention's dbias fed to the pair-bias
backward, the output projection's input gradient fed to the attention
backward.  The oracle chain rounds to bf16 where the GPU step stores bf16
(the projection outputs, the bias, the attention output and every
gradient handed from one stage to the next), so the remaining differences
are fp32-versus-fp64 arithmetic; a wrong layout or hand-off gives errors of
order one.  Tolerance: 2e-2 normwise on every output and gradient, except
the LayerNorm(z) bias gradient, which the chain makes zero (see below).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2404_11068_amd import graph as gr
from paper_2404_11068_amd import workloads as W
from tests.parity_util import to_f64

pytestmark = pytest.mark.gpu


def _bf(x):
    """Round to bf16 (nearest even) and back, as the GPU stores it."""
    return W.as_float64(W._store(np.asarray(x, dtype=np.float64), "bf16"), "bf16")


def _rel(got, ref):
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))


@pytest.mark.parametrize("N,L", [(4, 64), (2, 96)])
def test_module_step_matches_oracle_chain(N, L):
    print("\n[case] module N=%d L=%d" % (N, L), flush=True)
    step = gr.MSARowAttentionStep(N=N, L=L, seed=21)
    s = torch.cuda.Stream()
    cache = gr.GraphCache(capacity=2)
    cache.run(step.key(), step.record, s)
    torch.cuda.synchronize()
    got = {k: to_f64(v) for k, v in step.outputs().items()}

    H, d = step.H, step.d
    HD = H * d
    f = lambda t: to_f64(t)
    m, z = f(step.m), f(step.z)
    ln_m_w, ln_m_b, ln_z_w, ln_z_b = f(step.ln_m_w), f(step.ln_m_b), f(step.ln_z_w), f(step.ln_z_b)
    w_qkvg, b_qkvg, w_bias = f(step.w_qkvg), f(step.b_qkvg), f(step.w_bias)
    w_out, b_out, d_m_out = f(step.w_out), f(step.b_out), f(step.d_m_out)
    mask = np.ones((N, L), np.uint8)

    # forward
    q, k, v, g = (_bf(o).reshape(N, L, H, d) for o in oracle.ln_proj_forward(m, ln_m_w, ln_m_b, w_qkvg, b_qkvg,
                                                                             n_proj=4))
    bias = _bf(oracle.pair_bias_forward(z, ln_z_w, ln_z_b, w_bias))
    o, _ = oracle.forward(q, k, v, g, bias, mask, rows_per_bias=N)
    o = _bf(o)
    (m_out,) = oracle.linear_forward(o.reshape(N, L, HD), w_out, b_out)
    # backward
    d_o, dw_out, db_out = oracle.linear_backward(o.reshape(N, L, HD), w_out, [d_m_out])
    d_o = _bf(d_o).reshape(N, L, H, d)
    dq, dk, dv, dg, dbias = oracle.backward(q, k, v, d_o, g, bias, mask, rows_per_bias=N)
    douts = [_bf(t).reshape(N, L, HD) for t in (dq, dk, dv, dg)]
    dm, dln_m_w, dln_m_b, dw_qkvg, db_qkvg = oracle.ln_proj_backward(m, ln_m_w, ln_m_b, w_qkvg, douts)
    dz, dln_z_w, dln_z_b, dw_bias = oracle.pair_bias_backward(z, ln_z_w, ln_z_b, w_bias, dbias)

    ref = {"q": q, "k": k, "v": v, "gate": g, "bias": bias, "out": o, "m_out": m_out, "dout": d_o,
           "dw_out": dw_out, "db_out": db_out, "dq": dq, "dk": dk, "dv": dv, "dg": dg, "dbias": dbias,
           "dm": dm, "dw_qkvg": dw_qkvg, "db_qkvg": db_qkvg, "dln_m_w": dln_m_w, "dln_m_b": dln_m_b,
           "dz": dz, "dw_bias": dw_bias, "dln_z_w": dln_z_w, "dln_z_b": dln_z_b}
    # dln_z_b is zero in exact arithmetic: each row of the attention's dS sums
    # to zero over the keys, so dbias sums to zero over each plane, and
    # dln_z_b = sum over entries of dY = W^T (those sums).  It is checked
    # against the size of the terms it sums instead of its own (rounding-level)
    # size.  On the GPU the row sums of dS vanish only to ~2^-9 of Dsum (which
    # it forms from the bf16 attention output), so the bound is 1e-3 of the
    # terms' magnitude; layouts are checked by dz and dw_bias, not by this sum.
    dY = np.moveaxis(dbias, 1, 3) @ w_bias                       # [1, L, L, c_z]
    scale = np.abs(dY).reshape(-1, dY.shape[-1]).sum(axis=0)
    assert np.abs(got["dln_z_b"] - ref["dln_z_b"]).max() <= 1e-3 * scale.max(), "dln_z_b"
    assert np.abs(ref["dln_z_b"]).max() <= 1e-9 * scale.max()
    worst = 0.0
    for name, r in ref.items():
        if name == "dln_z_b":
            continue
        gv = got[name].reshape(r.shape)
        assert np.isfinite(gv).all(), name
        e = _rel(gv, r)
        worst = max(worst, e)
        assert e <= 2e-2, (name, e)
    print("  worst normwise rel err %.2e" % worst, flush=True)

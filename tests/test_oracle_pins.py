"""Pins for the fp64 oracle: checks against things other than the oracle itself.

* library routines: torch-CPU fp64 scaled_dot_product_attention (forward, with
  bias and key mask folded into a float attn_mask) and torch autograd through
  that routine (every gradient, including the pair bias);
* a closed form at L=2 worked by hand (tests/golden/closed_form_l2.json);
* central finite differences of a random projection of the output;
* invariants that the definition implies (normalisation, permutation of keys,
  single kept key, bias row shifts, gradient sums, masked keys, row
  independence, fully masked rows).

Each is chosen so that a plausible slip in the oracle (dropped bias or scale,
wrong sign, transposed operand, mask applied to queries, wrong bias plane,
dBias not summed over rows) fails at least one of them.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2404_11068_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_case(seed, N=3, L=5, H=2, d=3, rpb=3, gate=True, bias=True, mask_p=0.3):
    rng = np.random.default_rng(seed)
    q, k, v, g, do = (rng.standard_normal((N, L, H, d)) for _ in range(5))
    b = rng.standard_normal((N // rpb, H, L, L)) if bias else None
    m = None
    if mask_p:
        m = (rng.random((N, L)) >= mask_p).astype(np.uint8)
        m[m.sum(1) == 0, 0] = 1
    return dict(q=q, k=k, v=v, gate=g if gate else None, bias=b, mask=m, dout=do, rpb=rpb)


def _torch_reference(c, need_grad=True):
    """Forward and gradients from torch's SDPA + autograd (fp64, CPU)."""
    N, L, H, d = c["q"].shape
    t = {n: torch.tensor(c[n], dtype=torch.float64, requires_grad=need_grad)
         for n in ("q", "k", "v") }
    # SDPA wants [batch, heads, seq, dim]
    qh, kh, vh = (t[n].permute(0, 2, 1, 3) for n in ("q", "k", "v"))
    add = torch.zeros(N, H, L, L, dtype=torch.float64)
    bias_t = None
    if c["bias"] is not None:
        bias_t = torch.tensor(c["bias"], dtype=torch.float64, requires_grad=need_grad)
        plane = torch.arange(N) // c["rpb"]
        add = add + bias_t[plane]
    if c["mask"] is not None:
        keep = torch.tensor(c["mask"], dtype=torch.bool)
        add = add.masked_fill(~keep[:, None, None, :], float("-inf"))
    a = F.scaled_dot_product_attention(qh, kh, vh, attn_mask=add).permute(0, 2, 1, 3)
    g_t = None
    if c["gate"] is not None:
        g_t = torch.tensor(c["gate"], dtype=torch.float64, requires_grad=need_grad)
        o = torch.sigmoid(g_t) * a
    else:
        o = a
    res = {"out": o.detach().numpy()}
    if need_grad:
        o.backward(torch.tensor(c["dout"], dtype=torch.float64))
        res.update(dq=t["q"].grad.numpy(), dk=t["k"].grad.numpy(), dv=t["v"].grad.numpy(),
                   dgate=None if g_t is None else g_t.grad.numpy(),
                   dbias=None if bias_t is None else bias_t.grad.numpy())
    return res


def _oracle_all(c):
    o, lse = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], c["mask"], c["rpb"])
    dq, dk, dv, dg, db = oracle.backward(c["q"], c["k"], c["v"], c["dout"], c["gate"], c["bias"],
                                         c["mask"], c["rpb"])
    return dict(out=o, lse=lse, dq=dq, dk=dk, dv=dv, dgate=dg, dbias=db)


CASES = [
    dict(seed=1),
    dict(seed=2, gate=False),
    dict(seed=3, bias=False),
    dict(seed=4, mask_p=0.0),
    dict(seed=5, N=4, L=7, H=3, d=4, rpb=2),        # two bias planes
    dict(seed=6, N=2, L=9, H=1, d=8, rpb=1, mask_p=0.6),
    dict(seed=7, N=1, L=1, H=1, d=1, rpb=1, mask_p=0.0),  # degenerate L=1
    dict(seed=8, N=2, L=6, H=2, d=64, rpb=1),        # the largest head dim the library takes
]


@pytest.mark.parametrize("kw", CASES)
def test_matches_torch_sdpa_and_autograd(kw):
    c = _rand_case(**kw)
    ref = _torch_reference(c)
    got = _oracle_all(c)
    for name in ("out", "dq", "dk", "dv", "dgate", "dbias"):
        if ref[name] is None:
            assert got[name] is None
            continue
        np.testing.assert_allclose(got[name], ref[name], rtol=1e-10, atol=1e-12, err_msg=name)


def test_lse_matches_torch_logsumexp():
    c = _rand_case(11, N=3, L=6, H=2, d=5, rpb=3)
    N, L, H, d = c["q"].shape
    q = torch.tensor(c["q"]).permute(0, 2, 1, 3)
    k = torch.tensor(c["k"]).permute(0, 2, 1, 3)
    logits = q @ k.transpose(-1, -2).contiguous() / np.sqrt(d) + torch.tensor(c["bias"])[0]
    keep = torch.tensor(c["mask"], dtype=torch.bool)
    logits = logits.masked_fill(~keep[:, None, None, :], float("-inf"))
    _, lse = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], c["mask"], 3)
    np.testing.assert_allclose(lse, torch.logsumexp(logits, -1).numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("variant", ["ungated", "gated"])
def test_closed_form_l2(variant):
    gold = json.load(open(os.path.join(GOLDEN, "closed_form_l2.json")))
    sh = gold["shape"]
    shape4 = (sh["n_rows"], sh["seq_len"], 1, 1)
    q, k, v, do = (np.array(gold[n], np.float64).reshape(shape4) for n in ("q", "k", "v", "dout"))
    exp = gold[variant]
    g = np.array(exp["gate"], np.float64).reshape(shape4) if "gate" in exp else None
    bias = np.zeros((1, 1, 2, 2))
    o, lse = oracle.forward(q, k, v, g, bias, None, sh["rows_per_bias"])
    dq, dk, dv, dg, db = oracle.backward(q, k, v, do, g, bias, None, sh["rows_per_bias"])
    tol = dict(rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(o.reshape(2, 2), exp["out"], **tol)
    np.testing.assert_allclose(lse.reshape(2, 2), exp["lse"], **tol)
    np.testing.assert_allclose(dq.reshape(2, 2), exp["dq"], **tol)
    np.testing.assert_allclose(dk.reshape(2, 2), exp["dk"], **tol)
    np.testing.assert_allclose(dv.reshape(2, 2), exp["dv"], **tol)
    np.testing.assert_allclose(db.reshape(2, 2), exp["dbias"], **tol)
    if g is not None:
        np.testing.assert_allclose(dg.reshape(2, 2), exp["dgate"], **tol)


def test_finite_differences():
    """Central differences (step 1e-6) of <W, o> against every analytic gradient."""
    c = _rand_case(21, N=3, L=5, H=2, d=3, rpb=3, mask_p=0.3)
    rng = np.random.default_rng(99)
    W = rng.standard_normal(c["q"].shape)
    c["dout"] = W
    dq, dk, dv, dg, db = oracle.backward(c["q"], c["k"], c["v"], W, c["gate"], c["bias"], c["mask"], 3)
    analytic = dict(q=dq, k=dk, v=dv, gate=dg, bias=db)

    def f(**over):
        args = {n: over.get(n, c[n]) for n in ("q", "k", "v", "gate", "bias")}
        o, _ = oracle.forward(args["q"], args["k"], args["v"], args["gate"], args["bias"], c["mask"], 3)
        return float(np.sum(W * o))

    eps = 1e-6
    for name in ("q", "k", "v", "gate", "bias"):
        x = c[name]
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            num[idx] = (f(**{name: xp}) - f(**{name: xm})) / (2 * eps)
        scale = max(1.0, np.abs(num).max())
        err = np.abs(num - analytic[name]).max() / scale
        assert err < 1e-6, (name, err)


def test_probability_rows_normalised_and_masked():
    c = _rand_case(31, N=2, L=8, H=2, d=4, rpb=2, mask_p=0.4)
    for r in range(2):
        for h in range(2):
            P = oracle.probs(c["q"], c["k"], c["bias"], c["mask"], r, h, 2)
            assert (P >= 0).all()
            np.testing.assert_allclose(P.sum(1), 1.0, atol=1e-14)
            masked = c["mask"][r] == 0
            assert (P[:, masked] == 0).all()


def test_lse_reproduces_probabilities():
    """exp(s - lse) sums to one: checked through P's denominators at L=1 per key."""
    c = _rand_case(32, N=1, L=6, H=1, d=2, rpb=1, mask_p=0.0)
    _, lse = oracle.forward(c["q"], c["k"], c["v"], None, c["bias"], None, 1)
    # adding a constant to a whole bias row shifts that query's lse by the constant
    b2 = c["bias"].copy()
    b2[0, 0, 3, :] += 2.5
    _, lse2 = oracle.forward(c["q"], c["k"], c["v"], None, b2, None, 1)
    np.testing.assert_allclose(lse2[0, 0, 3] - lse[0, 0, 3], 2.5, atol=1e-13)
    keep = np.delete(np.arange(6), 3)
    np.testing.assert_allclose(lse2[0, 0, keep], lse[0, 0, keep], atol=1e-15)


def test_ones_values_give_gate():
    """V = 1 everywhere: softmax weights sum to one, so o = sigmoid(g)."""
    c = _rand_case(41, N=2, L=7, H=3, d=4, rpb=2)
    v = np.ones_like(c["v"])
    o, _ = oracle.forward(c["q"], c["k"], v, c["gate"], c["bias"], c["mask"], 2)
    np.testing.assert_allclose(o, 1.0 / (1.0 + np.exp(-c["gate"])), atol=1e-14)


def test_gate_open_zero_bias_is_standard_attention():
    c = _rand_case(42, N=2, L=6, H=2, d=4, rpb=2, mask_p=0.0)
    zero_bias = np.zeros_like(c["bias"])
    open_gate = np.full_like(c["gate"], 60.0)   # sigmoid(60) == 1 in fp64
    o1, _ = oracle.forward(c["q"], c["k"], c["v"], open_gate, zero_bias, None, 2)
    o2, _ = oracle.forward(c["q"], c["k"], c["v"], None, None, None, 2)
    np.testing.assert_allclose(o1, o2, atol=1e-15)
    q = torch.tensor(c["q"]).permute(0, 2, 1, 3)
    k = torch.tensor(c["k"]).permute(0, 2, 1, 3)
    v = torch.tensor(c["v"]).permute(0, 2, 1, 3)
    ref = F.scaled_dot_product_attention(q, k, v).permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(o2, ref, rtol=1e-12, atol=1e-13)


def test_key_permutation_invariance():
    c = _rand_case(51, N=2, L=7, H=2, d=3, rpb=2)
    perm = np.random.default_rng(5).permutation(7)
    o1, lse1 = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], c["mask"], 2)
    o2, lse2 = oracle.forward(c["q"], c["k"][:, perm], c["v"][:, perm], c["gate"],
                              c["bias"][..., perm], c["mask"][:, perm], 2)
    np.testing.assert_allclose(o1, o2, atol=1e-13)
    np.testing.assert_allclose(lse1, lse2, atol=1e-13)


def test_single_kept_key_returns_its_value():
    c = _rand_case(61, N=3, L=6, H=2, d=4, rpb=3)
    mask = np.zeros((3, 6), np.uint8)
    kept = [4, 0, 5]
    for r, j in enumerate(kept):
        mask[r, j] = 1
    o, lse = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], mask, 3)
    sg = 1.0 / (1.0 + np.exp(-c["gate"]))
    d = c["q"].shape[-1]
    for r, j in enumerate(kept):
        np.testing.assert_allclose(o[r], sg[r] * c["v"][r, j][None], atol=1e-14)
        # lse of a single kept key is that key's logit
        s = np.einsum("ihc,hc->hi", c["q"][r], c["k"][r, j]) / np.sqrt(d) + c["bias"][0, :, :, j]
        np.testing.assert_allclose(lse[r], s, atol=1e-13)


def test_bias_row_shift_invariance_and_gradient_sums():
    c = _rand_case(71, N=4, L=6, H=2, d=3, rpb=2)
    o1, _ = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], c["mask"], 2)
    b2 = c["bias"] + np.random.default_rng(3).standard_normal(c["bias"].shape[:3])[..., None]
    o2, _ = oracle.forward(c["q"], c["k"], c["v"], c["gate"], b2, c["mask"], 2)
    np.testing.assert_allclose(o1, o2, atol=1e-13)
    dq, dk, dv, dg, db = oracle.backward(c["q"], c["k"], c["v"], c["dout"], c["gate"], c["bias"],
                                         c["mask"], 2)
    # shift invariance => each dBias row sums to zero
    np.testing.assert_allclose(db.sum(-1), 0.0, atol=1e-13)
    # invariance to shifting every key by the same vector => sum_j dK_j = 0
    np.testing.assert_allclose(dk.sum(1), 0.0, atol=1e-13)
    # sum_j dV_j = sum_i dA_i with dA = dO * sigmoid(g)
    dA = c["dout"] / (1.0 + np.exp(-c["gate"]))
    np.testing.assert_allclose(dv.sum(1), dA.sum(1), atol=1e-12)
    # masked keys receive no gradient at all
    masked = c["mask"] == 0
    assert (dk[masked] == 0).all() and (dv[masked] == 0).all()


def test_rows_independent_and_dbias_sums_rows():
    c = _rand_case(81, N=4, L=5, H=2, d=3, rpb=4)
    o, lse = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], c["mask"], 4)
    full = oracle.backward(c["q"], c["k"], c["v"], c["dout"], c["gate"], c["bias"], c["mask"], 4)
    db_sum = np.zeros_like(c["bias"])
    for r in range(4):
        sl = slice(r, r + 1)
        o1, lse1 = oracle.forward(c["q"][sl], c["k"][sl], c["v"][sl], c["gate"][sl], c["bias"],
                                  c["mask"][sl], 1)
        np.testing.assert_allclose(o1[0], o[r], atol=1e-15)
        np.testing.assert_allclose(lse1[0], lse[r], atol=1e-15)
        g1 = oracle.backward(c["q"][sl], c["k"][sl], c["v"][sl], c["dout"][sl], c["gate"][sl],
                             c["bias"], c["mask"][sl], 1)
        for a, b in zip(g1[:4], full[:4]):
            np.testing.assert_allclose(a[0], b[r], atol=1e-15)
        db_sum += g1[4]
    np.testing.assert_allclose(full[4], db_sum, atol=1e-13)


def test_bias_planes_follow_rows_per_bias():
    """With two planes, rows 0-1 use plane 0 and rows 2-3 plane 1 (not interleaved)."""
    c = _rand_case(82, N=4, L=5, H=1, d=2, rpb=2, mask_p=0.0)
    o, _ = oracle.forward(c["q"], c["k"], c["v"], None, c["bias"], None, 2)
    for r in range(4):
        o1, _ = oracle.forward(c["q"][r:r + 1], c["k"][r:r + 1], c["v"][r:r + 1], None,
                               c["bias"][r // 2:r // 2 + 1], None, 1)
        np.testing.assert_allclose(o1[0], o[r], atol=1e-15)


def test_fully_masked_row_is_zero():
    c = _rand_case(91, N=2, L=4, H=2, d=3, rpb=2)
    mask = np.ones((2, 4), np.uint8)
    mask[1] = 0
    o, lse = oracle.forward(c["q"], c["k"], c["v"], c["gate"], c["bias"], mask, 2)
    assert (o[1] == 0).all() and np.isneginf(lse[1]).all()
    assert np.isfinite(o).all()
    dq, dk, dv, dg, db = oracle.backward(c["q"], c["k"], c["v"], c["dout"], c["gate"], c["bias"], mask, 2)
    for x in (dq, dk, dv, dg):
        assert np.isfinite(x).all() and (x[1] == 0).all()
    # dbias comes from row 0 only
    one = oracle.backward(c["q"][:1], c["k"][:1], c["v"][:1], c["dout"][:1], c["gate"][:1],
                          c["bias"], mask[:1], 1)
    np.testing.assert_allclose(db, one[4], atol=1e-15)


def test_empty_inputs():
    q = np.zeros((0, 4, 2, 3))
    o, lse = oracle.forward(q, q, q, None, None, None, 1)
    assert o.shape == (0, 4, 2, 3) and lse.shape == (0, 2, 4)
    q = np.zeros((2, 0, 2, 3))
    o, lse = oracle.forward(q, q, q, None, np.zeros((1, 2, 0, 0)), None, 2)
    assert o.shape == (2, 0, 2, 3)


def test_workload_generator_shapes_and_masks():
    for w in workloads.WORKLOADS:
        small = w.with_rows(min(w.n_rows, 4))
        x = workloads.generate(small)
        N, L, H, d = small.n_rows, small.seq_len, small.n_heads, small.head_dim
        assert x["q"].shape == (N, L, H, d)
        assert (x["bias"] is not None) == w.bias
        if x["mask"] is not None:
            assert x["mask"].shape == (N, L)
            assert (x["mask"].sum(1) >= 1).all()
        if w.dtype == "bf16":
            assert x["q"].dtype == np.uint16
    # same seed -> identical bits
    a = workloads.generate(workloads.WORKLOADS[0])
    b = workloads.generate(workloads.WORKLOADS[0])
    for n in a:
        if a[n] is not None:
            assert np.array_equal(a[n], b[n])


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], np.float32)
    bits = workloads.f32_to_bf16_bits(x)
    back = workloads.as_float64(bits, "bf16")
    # 1+2^-8 is a tie between 1 and 1+2^-7: even mantissa (1.0) wins;
    # 1+3*2^-8 ties between 1+2^-7 and 1+2^-6: even (1+2^-6) wins
    np.testing.assert_array_equal(back, [1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0])
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(back, ref)

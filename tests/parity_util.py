"""Shared helpers of the GPU parity tests: run one input set through the HIP
library (via its C ABI binding) and through the fp64 oracle, and compare.

Tolerances (element-wise |x - ref| <= atol + rtol*|ref|):
  fp32 path: atol = rtol = 1e-5;   bf16 path: atol = rtol = 2e-2.
Because several gradients have small magnitudes (where an absolute 2e-2 would
pass almost anything), the bf16 path must also meet a normwise bound,
||x - ref||_2 <= 1e-2 * ||ref||_2, which is about 4x the error that rounding
every MFMA input and every output to bf16 (relative 2^-9 each) produces.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import workloads as W

TOL = {"f32": dict(atol=1e-5, rtol=1e-5, norm=1e-5), "bf16": dict(atol=2e-2, rtol=2e-2, norm=1e-2)}


def to_device(arr, dtype: str, device="cuda"):
    if arr is None:
        return None
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to(device)


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def gpu_run(x: dict, dtype: str, rows_per_bias: int, view=None, stream=None):
    """Forward + backward on the GPU.  `view` optionally maps each token tensor
    (e.g. to a transposed view) before the call; results are returned as fp64
    numpy arrays in the [N, L, H, d] logical layout."""
    dev = {n: to_device(x[n], dtype) for n in ("q", "k", "v", "gate", "bias", "dout")}
    mask = None if x["mask"] is None else torch.from_numpy(x["mask"]).cuda()
    if view is not None:
        for n in ("q", "k", "v", "gate", "dout"):
            if dev[n] is not None:
                dev[n] = view(dev[n])
    out, lse = ea.evo_attn_fwd(dev["q"], dev["k"], dev["v"], dev["gate"], dev["bias"], mask,
                               rows_per_bias=rows_per_bias, stream=stream)
    dq, dk, dv, dg, db = ea.evo_attn_bwd(dev["q"], dev["k"], dev["v"], dev["gate"], dev["bias"], mask,
                                         out, lse, dev["dout"], rows_per_bias=rows_per_bias,
                                         stream=stream)
    torch.cuda.synchronize()
    res = dict(out=out, lse=lse, dq=dq, dk=dk, dv=dv, dgate=dg, dbias=db)
    return {k: (None if v is None else to_f64(v)) for k, v in res.items()}


def oracle_run(x: dict, dtype: str, rows_per_bias: int):
    f = {n: (None if x[n] is None else W.as_float64(x[n], dtype))
         for n in ("q", "k", "v", "gate", "bias", "dout")}
    out, lse = oracle.forward(f["q"], f["k"], f["v"], f["gate"], f["bias"], x["mask"], rows_per_bias)
    dq, dk, dv, dg, db = oracle.backward(f["q"], f["k"], f["v"], f["dout"], f["gate"], f["bias"],
                                         x["mask"], rows_per_bias)
    return dict(out=out, lse=lse, dq=dq, dk=dk, dv=dv, dgate=dg, dbias=db)


def compare(got: dict, ref: dict, dtype: str, names=None, label=""):
    tol = TOL[dtype]
    report = {}
    for name in names or ref.keys():
        r, g = ref[name], got[name]
        if r is None:
            assert g is None, (label, name)
            continue
        assert g.shape == r.shape, (label, name, g.shape, r.shape)
        # -inf lse (fully masked queries) must match exactly
        inf = np.isinf(r)
        assert np.array_equal(np.isinf(g), inf), (label, name, "infinite entries differ")
        if inf.any():
            assert np.array_equal(g[inf], r[inf]), (label, name)
        gf, rf = g[~inf], r[~inf]
        assert np.isfinite(gf).all(), (label, name, "non-finite output")
        err = np.abs(gf - rf)
        bound = tol["atol"] + tol["rtol"] * np.abs(rf)
        worst = np.argmax(err - bound) if err.size else 0
        rn = np.linalg.norm(rf)
        rel_norm = np.linalg.norm(gf - rf) / rn if rn > 0 else np.linalg.norm(gf - rf)
        report[name] = dict(max_abs=float(err.max()) if err.size else 0.0, rel_norm=float(rel_norm))
        assert (err <= bound).all(), (label, name, "max err %.3g at ref %.3g (bound %.3g)" %
                                      (err.flat[worst], rf.flat[worst], bound.flat[worst]))
        assert rel_norm <= tol["norm"] or rn == 0, (label, name, "normwise rel err %.3g" % rel_norm)
    return report


def make_inputs(N, L, H, d, dtype, *, bias=True, rpb=None, gate=True, mask="bernoulli", p=0.1,
                seed=0, qkv_scale=1.0):
    w = W.Workload("adhoc", N, L, H, d, dtype, bias, rpb or N, gate=gate, mask=mask, mask_p=p,
                   pad_max=max(L // 4, 0), len_lo=max(1, (3 * L) // 4), len_hi=L,
                   qkv_scale=qkv_scale, seed=seed)
    return w, W.generate(w)

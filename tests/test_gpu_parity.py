"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle,
element by element on identical seeded inputs.

* every workload at its full size (all outputs, all elements);
* small shapes that span several 32-key tiles with ragged tails, every head
  dim, fp32 and bf16, with and without gate / bias / mask, several bias planes;
* the ending-node layout (a transposed view, no copy);
* edge cases: one key, fully masked rows, empty problems, maximum seq_len;
* properties: exact zeros at masked keys, bitwise-repeatable backward,
  non-default stream, rows independent.
"""
import numpy as np
import pytest
import torch

from paper_2404_11068_amd import evo_attn as ea
from paper_2404_11068_amd import workloads as W
from tests.parity_util import compare, gpu_run, make_inputs, oracle_run, to_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", [w.name for w in W.WORKLOADS])
def test_full_workload_parity(name):
    w = W.by_name(name)
    x = W.generate(w)
    print("\n[case] full workload", name, flush=True)
    got = gpu_run(x, w.dtype, w.rows_per_bias)
    ref = oracle_run(x, w.dtype, w.rows_per_bias)
    rep = compare(got, ref, w.dtype, label=name)
    for k, v in rep.items():
        print("  %-6s max_abs %.3e  rel_norm %.3e" % (k, v["max_abs"], v["rel_norm"]))


SMALL = [
    # N, L, H, d, dtype, kwargs
    (3, 1, 2, 8, "bf16", dict(mask="none")),
    (4, 5, 2, 16, "bf16", dict()),
    (4, 33, 3, 32, "bf16", dict(rpb=2)),
    (2, 63, 2, 8, "bf16", dict(gate=False)),
    (3, 100, 2, 32, "bf16", dict(bias=False, mask="tail_pad")),
    (2, 129, 1, 16, "bf16", dict(mask="length")),
    (2, 200, 2, 32, "bf16", dict(rpb=1)),
    (2, 255, 1, 8, "bf16", dict(p=0.3)),
    (2, 256, 2, 32, "bf16", dict(mask="none", gate=False, bias=False)),
    (3, 7, 2, 8, "f32", dict()),
    (2, 37, 2, 16, "f32", dict(rpb=1)),
    (2, 96, 2, 32, "f32", dict(mask="length")),
    (2, 128, 1, 32, "f32", dict(gate=False)),
    (2, 250, 1, 16, "f32", dict(p=0.2)),
    # head_dim 64: two workgroups per (row, head), each with 32 output channels
    (2, 100, 2, 64, "bf16", dict()),
    (2, 256, 1, 64, "bf16", dict(rpb=1)),
    (2, 45, 2, 64, "bf16", dict(mask="length")),          # bias through the transpose kernel
    (3, 64, 2, 64, "bf16", dict(gate=False, bias=False, mask="none")),
    (2, 96, 1, 64, "f32", dict()),
    (2, 128, 2, 64, "f32", dict(rpb=1, mask="tail_pad")),
    # single-pass backward (bf16, head_dim <= 32; with a bias up to 128 keys, or
    # head_dim 8 at 256): several rows per chunk with partial dBias planes and
    # their reduction, one chunk per plane (dBias written directly), no bias
    (96, 256, 8, 8, "bf16", dict()),
    (128, 128, 8, 32, "bf16", dict(rpb=16, mask="length")),
    # the dQ sum's wave split: one key tile at head_dim 32 (four summing steps
    # per thread), two at head_dim 16 (both waves sum), four at head_dim 8
    # (one of the four sums)
    (4, 20, 2, 32, "bf16", dict()),
    (4, 50, 2, 16, "bf16", dict(rpb=2)),
    (4, 110, 2, 8, "bf16", dict(mask="tail_pad")),
    (64, 96, 2, 16, "bf16", dict(p=0.2)),
    (3, 200, 2, 8, "bf16", dict(rpb=1)),
    (5, 256, 3, 8, "bf16", dict(bias=False, gate=False)),
    (4, 256, 2, 32, "bf16", dict(bias=False, mask="length")),
    # 257..512 keys (bf16, head_dim <= 32): 16-wave workgroups, two-pass backward
    (3, 384, 2, 32, "bf16", dict()),
    (2, 512, 2, 32, "bf16", dict(mask="length")),
    (3, 512, 2, 8, "bf16", dict(p=0.2)),
    (2, 333, 3, 16, "bf16", dict(rpb=1)),
    (2, 460, 2, 8, "bf16", dict(bias=False, mask="tail_pad")),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "N%dL%dH%dd%d_%s_%s" % (c[:5] + (
    "-".join("%s=%s" % kv for kv in sorted(c[5].items())) or "default",)))
def test_small_ragged_parity(case):
    N, L, H, d, dtype, kw = case
    w, x = make_inputs(N, L, H, d, dtype, seed=7 + L, **kw)
    print("\n[case]", case, flush=True)
    got = gpu_run(x, dtype, w.rows_per_bias)
    ref = oracle_run(x, dtype, w.rows_per_bias)
    compare(got, ref, dtype, label=str(case))


# Shapes that select the row-walking forward (all rows under one bias plane,
# bf16, L a multiple of 8, at most 256 keys, at least two (row, head) units
# per resident workgroup: 256 * 8 / (key tiles) workgroups): it must produce
# the bits of the one-unit kernel, which the environment switch
# EVO_ATTN_FWD_ROWS=0 selects.  The full-size workloads with a shared bias
# (MSA row, triangle, extra-MSA) run it against the oracle in
# test_full_workload_parity.
ROWS = [
    # N, L, H, d, kwargs
    (128, 256, 4, 32, dict()),                      # 8 key tiles, 512 units: the threshold
    (512, 256, 4, 32, dict()),                      # 2048 units
    (256, 200, 8, 8, dict(p=0.2)),                  # ragged last key tile
    (256, 248, 8, 16, dict(gate=False, mask="length")),
    (1024, 104, 4, 16, dict(mask="none")),          # 4 key tiles
    (2048, 40, 4, 8, dict(mask="tail_pad")),        # 2 key tiles
    (4096, 24, 4, 32, dict()),                      # 1 key tile
    (700, 256, 3, 16, dict(mask="length")),         # 3 heads: a grid of 240 workgroups
]


def test_forward_with_several_bias_planes_at_scale():
    """Enough units for the row-walking forward but rows under several bias
    planes: the one-unit kernel runs; oracle parity of the whole call."""
    w, x = make_inputs(512, 256, 4, 8, "bf16", rpb=256, seed=23)
    print("\n[case] several planes at scale", flush=True)
    got = gpu_run(x, "bf16", w.rows_per_bias)
    ref = oracle_run(x, "bf16", w.rows_per_bias)
    compare(got, ref, "bf16", label="several planes")


@pytest.mark.parametrize("case", ROWS, ids=lambda c: "N%dL%dH%dd%d" % c[:4])
def test_row_walking_forward_matches_one_unit_kernel(case, monkeypatch):
    N, L, H, d, kw = case
    w, x = make_inputs(N, L, H, d, "bf16", seed=11 + L, **kw)
    print("\n[case] row-walking forward", case, flush=True)
    dev = {n: to_device(x[n], "bf16") for n in ("q", "k", "v", "gate", "bias")}
    mask = None if x["mask"] is None else torch.from_numpy(x["mask"]).cuda()
    args = (dev["q"], dev["k"], dev["v"], dev["gate"], dev["bias"], mask)
    monkeypatch.setenv("EVO_ATTN_FWD_ROWS", "0")
    out0, lse0 = ea.evo_attn_fwd(*args, rows_per_bias=w.rows_per_bias)
    monkeypatch.setenv("EVO_ATTN_FWD_ROWS", "1")
    out1, lse1 = ea.evo_attn_fwd(*args, rows_per_bias=w.rows_per_bias)
    torch.cuda.synchronize()
    assert torch.equal(out0.view(torch.int16), out1.view(torch.int16))
    assert torch.equal(lse0, lse1)


# dBias sums dS over the R rows that share a plane.  Each row's term carries
# the bf16 rounding of D (formed from the saved bf16 output) and of dA, and
# where the softmax puts its mass on one key the exact term nearly cancels,
# so those elements keep an absolute error that grows like sqrt(R) while
# their reference stays near zero.  The normwise error does not grow
# (measured 1.9e-3 from R = 64 to 2048); the element bound is met up to the
# workloads' 256 rows per plane at head_dim 32 and 2048 at head_dim 8.
_MANY_ROWS = [(1024, 32), (2048, 8)]


@pytest.mark.parametrize("R,d", _MANY_ROWS, ids=lambda v: str(v))
def test_dbias_over_many_rows_normwise(R, d):
    w, x = make_inputs(R, 256, 4, d, "bf16", seed=77)
    print("\n[case] dbias over rows", R, d, flush=True)
    got = gpu_run(x, "bf16", w.rows_per_bias)
    ref = oracle_run(x, "bf16", w.rows_per_bias)
    compare(got, ref, "bf16", names=[n for n in ref if n != "dbias"], label="R%d d%d" % (R, d))
    rel = np.linalg.norm(got["dbias"] - ref["dbias"]) / np.linalg.norm(ref["dbias"])
    assert rel <= 1e-2, rel


@pytest.mark.xfail(reason="bf16 dBias over 1024 rows at head_dim 32: near-cancelling elements keep a "
                          "sqrt(R)-growing absolute error past the element bound (stated in evo_attn.h)",
                   strict=False)
def test_dbias_over_many_rows_elementwise():
    w, x = make_inputs(1024, 256, 4, 32, "bf16", seed=77)
    print("\n[case] dbias over rows, element bound", flush=True)
    compare(gpu_run(x, "bf16", w.rows_per_bias), oracle_run(x, "bf16", w.rows_per_bias), "bf16",
            names=["dbias"], label="R1024 d32")


@pytest.mark.parametrize("d", [32, 64])
def test_ending_node_transposed_view(d):
    """Triangle attention around the ending node: rows are the columns of the
    pair representation, passed as a strided view without a copy."""
    L, H = 64, 4
    w, x = make_inputs(L, L, H, d, "bf16", seed=11, mask="length")
    print("\n[case] ending-node view d=%d" % d, flush=True)
    # the pair representation z[i, j] holds row j, token i: build it so that
    # z.transpose(0, 1) is the [N=L, L, H, d] logical tensor of x
    def view(t):
        z = t.transpose(0, 1).contiguous()      # physical [L(token), L(row), H, d]
        v = z.transpose(0, 1)                   # logical [row, token, H, d], strided
        assert not v.is_contiguous()
        return v
    got = gpu_run(x, "bf16", w.rows_per_bias, view=view)
    ref = oracle_run(x, "bf16", w.rows_per_bias)
    compare(got, ref, "bf16", label="ending-node")


# head_dim 64, bf16: the backward forms D_i = sum_c dO_ic o_ic from the
# bf16-rounded output, so D carries about 2^-9 * ||dO_i o_i|| (sqrt(d) * 2^-9
# for unit entries) of rounding, and dS = P (dP - D) inherits all of it where
# P puts its mass on one key -- which is what this ramp does.  At d = 64 one
# dBias element misses the element bound by about 5%; the limit is stated in
# include/evo_attn.h.
_D64_RAMP = pytest.mark.xfail(reason="bf16 head_dim 64: D is formed from the bf16 output; a peaked softmax "
                                     "leaves dBias ~5% past the element bound (stated in evo_attn.h)",
                              strict=False)


@pytest.mark.parametrize("dtype,d,L", [("bf16", 32, 256), ("bf16", 8, 256), ("f32", 16, 256),
                                       ("bf16", 32, 512), ("bf16", 8, 448),
                                       pytest.param("bf16", 64, 256, marks=_D64_RAMP)])
@pytest.mark.parametrize("sign", [1, -1])
def test_running_max_moves(dtype, d, L, sign):
    """A bias ramp of 40 along the keys makes the logits of every query grow
    (sign 1: the running max is raised at many key tiles, each time by more
    than the 2^8 rescale threshold) or fall (sign -1: set by the first tile)."""
    N, H = 2, 2
    w, x = make_inputs(N, L, H, d, dtype, seed=21, mask="none")
    ramp = sign * np.linspace(0.0, 40.0, L)
    b = W.as_float64(x["bias"], dtype) + ramp[None, None, None, :]
    x = dict(x)
    x["bias"] = W.f32_to_bf16_bits(b.astype(np.float32)) if dtype == "bf16" else b.astype(np.float32)
    print("\n[case] running max", dtype, d, sign, flush=True)
    got = gpu_run(x, dtype, w.rows_per_bias)
    ref = oracle_run(x, dtype, w.rows_per_bias)
    compare(got, ref, dtype, label="ramp %s d%d %+d" % (dtype, d, sign))


def test_fully_masked_rows_are_zero():
    N, L, H, d = 4, 40, 2, 16
    w, x = make_inputs(N, L, H, d, "bf16", seed=3)
    x["mask"][1] = 0
    x["mask"][3] = 0
    print("\n[case] fully masked rows", flush=True)
    got = gpu_run(x, "bf16", w.rows_per_bias)
    assert (got["out"][[1, 3]] == 0).all()
    assert np.isneginf(got["lse"][[1, 3]]).all()
    for n in ("dq", "dk", "dv", "dgate"):
        assert (got[n][[1, 3]] == 0).all(), n
    ref = oracle_run(x, "bf16", w.rows_per_bias)
    compare(got, ref, "bf16", label="fully-masked")


def test_masked_keys_get_exact_zero_gradients():
    w, x = make_inputs(3, 90, 2, 32, "bf16", seed=5, p=0.3)
    got = gpu_run(x, "bf16", w.rows_per_bias)
    masked = x["mask"] == 0
    assert masked.any()
    assert (got["dk"][masked] == 0).all() and (got["dv"][masked] == 0).all()


# 90 keys: the single-pass backward for bf16, the two-pass one for fp32; 256
# keys at head_dim 16 and 32: the two-pass backward for bf16 (kv's masked-key
# term on the matrix unit); 256 keys at head_dim 8: the single pass with the
# masked-key term and -Dsum in the logit and dP products' spare k-slots
@pytest.mark.parametrize("dtype,d,L", [("bf16", 8, 90), ("bf16", 32, 90), ("f32", 16, 90),
                                       ("bf16", 32, 256), ("bf16", 16, 256), ("bf16", 8, 256)])
def test_masked_keys_with_huge_logits(dtype, d, L):
    """Masked keys whose logits sit more than 100 above every kept key's are
    still excluded: exp of such a logit against the saved lse (which leaves
    masked keys out) overflows to +inf, so any multiply-by-zero masking would
    turn it into NaN.  One bias plane per row carries +120 at that row's
    masked keys; dK, dV and dBias must be exactly 0 there, and every output
    must match the oracle."""
    N, H = 3, 2
    w, x = make_inputs(N, L, H, d, dtype, seed=55 + d, rpb=1, p=0.3)
    masked = x["mask"] == 0
    assert masked.any()
    b = W.as_float64(x["bias"], dtype) + 120.0 * masked[:, None, None, :]
    x = dict(x)
    x["bias"] = W.f32_to_bf16_bits(b.astype(np.float32)) if dtype == "bf16" else b.astype(np.float32)
    print("\n[case] masked keys, huge logits", dtype, d, L, flush=True)
    got = gpu_run(x, dtype, w.rows_per_bias)
    for n in ("dk", "dv"):
        assert (got[n][masked] == 0).all(), n
    db = got["dbias"]  # [N, H, L, L]: plane r belongs to row r, its last axis is the key
    assert (db[np.broadcast_to(masked[:, None, None, :], db.shape)] == 0).all()
    ref = oracle_run(x, dtype, w.rows_per_bias)
    compare(got, ref, dtype, label="huge masked logits %s d%d L%d" % (dtype, d, L))


def test_empty_problems_are_noops():
    for shape in [(0, 16, 2, 32), (3, 0, 2, 32)]:
        q = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
        out, lse = ea.evo_attn_fwd(q, q, q)
        dq, dk, dv, dg, db = ea.evo_attn_bwd(q, q, q, None, None, None, out, lse, q)
        torch.cuda.synchronize()
        assert out.numel() == 0 and dq.numel() == 0


@pytest.mark.parametrize("name,rows", [("msa_row_bias_bf16", 16), ("extra_msa_bf16", 64)])
def test_backward_is_bitwise_repeatable_and_stream_ordered(name, rows):
    """Two calls on a non-default stream give identical bits: every sum in the
    backward (over keys, queries and rows) runs in a fixed order (two-pass
    backward at head_dim 32 with 256 keys, single pass at head_dim 8)."""
    w = W.by_name(name).with_rows(rows)
    x = W.generate(w)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        a = gpu_run(x, w.dtype, w.rows_per_bias, stream=s)
        b = gpu_run(x, w.dtype, w.rows_per_bias, stream=s)
    for n in a:
        if a[n] is not None:
            assert np.array_equal(a[n], b[n], equal_nan=True), n


def test_rows_are_independent():
    w, x = make_inputs(6, 70, 2, 16, "bf16", seed=9, rpb=6)
    full = gpu_run(x, "bf16", 6)
    sub = {k: (None if v is None else (v[2:4] if k not in ("bias",) else v)) for k, v in x.items()}
    part = gpu_run(sub, "bf16", 2)
    for n in ("out", "lse", "dq", "dk", "dv", "dgate"):
        np.testing.assert_array_equal(part[n], full[n][2:4])


def test_unsupported_shapes_raise():
    q = torch.zeros((2, 520, 2, 32), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ea.EvoAttnError) as e:
        ea.evo_attn_fwd(q, q, q)
    assert e.value.status == 2
    q = torch.zeros((2, 300, 2, 32), dtype=torch.float32, device="cuda")
    with pytest.raises(ea.EvoAttnError) as e:
        ea.evo_attn_fwd(q, q, q)
    assert e.value.status == 2
    q = torch.zeros((2, 16, 2, 24), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ea.EvoAttnError):
        ea.evo_attn_fwd(q, q, q)


@pytest.mark.parametrize("dtype,L", [("bf16", 96), ("bf16", 90), ("f32", 64)])
def test_traced_backward_matches_plain(dtype, L):
    """The profiling entry point gives the same bits as the plain backward, on
    both bias paths (a bf16 bias of whole 16-byte rows is read directly; fp32
    and other lengths go through the transpose kernel), and its events bracket
    non-negative intervals."""
    w, x = make_inputs(3, L, 2, 32, dtype, seed=31 + L)
    print("\n[case] traced backward", dtype, L, flush=True)
    dev = {n: to_device(x[n], dtype) for n in ("q", "k", "v", "gate", "bias", "dout")}
    mask = torch.from_numpy(x["mask"]).cuda()
    args = (dev["q"], dev["k"], dev["v"], dev["gate"], dev["bias"], mask)
    out, lse = ea.evo_attn_fwd(*args, rows_per_bias=w.rows_per_bias)
    plain = ea.evo_attn_bwd(*args, out, lse, dev["dout"], rows_per_bias=w.rows_per_bias)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(ea.evo_attn_bwd_kernel_count(True) + 1)]
    traced = ea.evo_attn_bwd(*args, out, lse, dev["dout"], rows_per_bias=w.rows_per_bias, events=ev)
    torch.cuda.synchronize()
    for a, b in zip(plain, traced):
        assert torch.equal(a, b)
    assert all(ev[j].elapsed_time(ev[j + 1]) >= 0.0 for j in range(len(ev) - 1))


@pytest.mark.parametrize("dtype,bound", [("bf16", 1e-2), ("f32", 1e-5)])
def test_gradient_sums_over_keys_vanish(dtype, bound):
    """Every row of dS sums to zero over the keys (sum_j P_ij (dP_ij - D_i) =
    D_i - D_i), so dK summed over the keys vanishes for every (row, head,
    channel) and dBias summed over the keys vanishes for every (plane, head,
    query).  Checked against the size of the summed terms: the bf16 path forms
    D from the bf16 output, which leaves row sums of about 2^-9 of the terms."""
    w, x = make_inputs(4, 96, 2, 32, dtype, seed=41, rpb=2)
    print("\n[case] gradient sums", dtype, flush=True)
    got = gpu_run(x, dtype, w.rows_per_bias)
    for name, axis in (("dk", 1), ("dbias", -1)):
        g = got[name]
        total = np.abs(g.sum(axis=axis))
        terms = np.abs(g).sum(axis=axis)
        ratio = float((total / np.maximum(terms, 1e-30)).max())
        print("  %-6s max |sum| / sum|.| = %.2e" % (name, ratio), flush=True)
        assert (total <= bound * terms + 1e-7).all(), (name, ratio)

"""bench.py's host-side model of the attention step, on the CPU.

* Its algorithmic bytes for the five scope-table workloads equal the sums of
  the tensors the method reads and writes (the table's own per-tensor sizes:
  one [N, L, H, d] token tensor, the bias plane(s), the fp32 LSE and dBias, the
  key-mask bytes), written out here tensor by tensor.
* Its mirror of the library's launch rules (which forward kernel, single-pass
  or two-pass backward) names, for every attention workload, the kernels that
  the rocprofv3 traces in profiles/ show running.
* The per-kernel model adds up to the step's algorithmic bytes wherever each
  tensor is touched by one kernel (forward; single-pass backward + reduction).
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2404_11068_amd import workloads as W  # noqa: E402


def _tensors(N, L, H, d, es, bias_planes, gate=True, mask=True):
    tok = N * L * H * d * es
    return dict(tok=tok, lse=N * H * L * 4, bias=bias_planes * H * L * L * es, dbias=bias_planes * H * L * L * 4,
                mask=N * L if mask else 0, gates=1 if gate else 0)


# name: (N, L, H, d, bytes per element, bias planes)
SCOPE = {
    "tri_tiny_f32": (32, 32, 4, 32, 4, 1),
    "msa_col_bf16": (256, 128, 8, 32, 2, 0),
    "msa_row_bias_bf16": (128, 256, 8, 32, 2, 1),
    "tri_start_bf16": (256, 256, 4, 32, 2, 1),
    "extra_msa_bf16": (1024, 256, 8, 8, 2, 1),
}


@pytest.mark.parametrize("name", sorted(SCOPE))
def test_algorithmic_bytes_are_the_tensors_of_the_method(name):
    N, L, H, d, es, planes = SCOPE[name]
    w = W.by_name(name)
    assert (w.n_rows, w.seq_len, w.n_heads, w.head_dim) == (N, L, H, d)
    t = _tensors(N, L, H, d, es, planes, gate=w.gate, mask=w.mask != "none")
    # forward: read Q, K, V, G, bias, mask; write O, LSE
    fwd = 3 * t["tok"] + t["gates"] * t["tok"] + t["bias"] + t["mask"] + t["tok"] + t["lse"]
    # backward: read Q, K, V, G, O, dO, LSE, bias, mask; write dQ, dK, dV, dG, dBias (fp32)
    bwd = (5 + t["gates"]) * t["tok"] + t["lse"] + t["bias"] + t["mask"] + (3 + t["gates"]) * t["tok"] + t["dbias"]
    assert bench.algorithmic_bytes(w, es) == (fwd, bwd)


def test_headline_byte_counts():
    """The triangle workload: 85.52 MB forward and 170.46 MB backward."""
    fwd, bwd = bench.algorithmic_bytes(W.by_name("tri_start_bf16"), 2)
    assert (fwd, bwd) == (85_524_480, 170_459_136)


# the kernels each workload runs, as the kernel traces in profiles/ show them
TRACED = {
    "tri_tiny_f32": ("fwd_kernel", False),
    "msa_col_bf16": ("fwd_kernel", True),
    "msa_row_bias_bf16": ("fwd_rows_kernel", False),
    "tri_start_bf16": ("fwd_rows_kernel", False),
    "extra_msa_bf16": ("fwd_rows_kernel", True),
    "msa_row_bias_bf16_share8": ("fwd_kernel", False),
    "extra_msa_bf16_share8": ("fwd_rows_kernel", True),
}


@pytest.mark.parametrize("name", sorted(TRACED))
def test_launch_rules_match_the_traces(name):
    w = W.by_name(name)
    es = 2 if w.dtype == "bf16" else 4
    fwd_name, fused = TRACED[name]
    assert bench.forward_kernel(w, es) == fwd_name
    assert bench.fused_backward(w, es) == fused
    prof = open(os.path.join(ROOT, "profiles", "kernels_%s.md" % name)).read()
    assert fwd_name + "<" in prof
    assert ("bwd_fused_kernel<" in prof) == fused
    assert ("qbias_kernel<" in prof) == (not fused)


@pytest.mark.parametrize("name", sorted(TRACED))
def test_kernel_model_adds_up(name):
    w = W.by_name(name)
    es = 2 if w.dtype == "bf16" else 4
    fwd, bwd = bench.algorithmic_bytes(w, es)
    ks = bench.kernel_model(w, es, ws_bytes=1 << 26)
    assert ks[0][1] == fwd
    if bench.fused_backward(w, es):
        assert sum(k[1] for k in ks[1:]) == bwd
    else:
        # the two passes both read Q, K, V, LSE, bias and mask: at least the step's bytes
        assert sum(k[1] for k in ks[1:]) >= bwd

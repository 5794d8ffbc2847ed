"""The oracle's pins catch plausible mistakes in it.

Each case plants one slip in a copy of oracle/evo_attn_oracle.c (a dropped
scale, a transposed operand, a wrong sign or index, the mask applied to the
wrong axis, ...) or of oracle/layernorm_oracle.c (biased/unbiased variance,
eps placement, a dropped term of the input gradient, ...), compiles the copy
with gcc, and runs the pin suites that rest on that file against it in a
subprocess: at least one pin must fail.  The unmutated sources, built the same
way, must pass them all, so that a failure means the planted slip and not the
harness.  CPU only.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "evo_attn_oracle.c")
LN_SRC = os.path.join(ROOT, "oracle", "layernorm_oracle.c")
PINS = [os.path.join(HERE, "test_oracle_pins.py")]
LN_PINS = [os.path.join(HERE, f) for f in ("test_layernorm_oracle_pins.py", "test_proj_oracle_pins.py",
                                         "test_pair_bias_oracle_pins.py")]

# (name, text in the oracle, replacement): each text occurs exactly once
MUTATIONS = [
    ("logit scale dropped", "double s = scale * dot;", "double s = dot;"),
    ("bias transposed", "bias[((b * dm->n_heads + h) * L + i) * L + j]", "bias[((b * dm->n_heads + h) * L + j) * L + i]"),
    ("wrong bias plane", "const int64_t b = r / dm->rows_per_bias;\n    for (int64_t i = 0; i < L; ++i) {",
     "const int64_t b = r % (dm->n_rows / dm->rows_per_bias);\n    for (int64_t i = 0; i < L; ++i) {"),
    ("mask applied to queries", "int keep = mask ? (mask[r * L + j] != 0) : 1;", "int keep = mask ? (mask[r * L + i] != 0) : 1;"),
    ("mask inverted", "int keep = mask ? (mask[r * L + j] != 0) : 1;", "int keep = mask ? (mask[r * L + j] == 0) : 1;"),
    ("fully masked row uniform", "for (int64_t j = 0; j < L; ++j) row[j] = 0.0;", "for (int64_t j = 0; j < L; ++j) row[j] = 1.0 / (double)L;"),
    ("lse without log", "if (lse) lse[i] = m + log(sum);", "if (lse) lse[i] = m + sum;"),
    ("gate not through sigmoid", "out[x] = g ? sigmoid(g[x]) * a : a;", "out[x] = g ? g[x] * a : a;"),
    ("dG sign", "dg[x] = dout[x] * acc * sg * (1.0 - sg);", "dg[x] = -dout[x] * acc * sg * (1.0 - sg);"),
    ("dV from transposed P", "for (int64_t i = 0; i < L; ++i) acc += P[i * L + j] * dA[i * d + c];",
     "for (int64_t i = 0; i < L; ++i) acc += P[j * L + i] * dA[i * d + c];"),
    ("softmax Jacobian sign", "dPi[j] = P[i * L + j] * (dPi[j] - pdp);", "dPi[j] = P[i * L + j] * (dPi[j] + pdp);"),
    ("dQ from q instead of k", "for (int64_t j = 0; j < L; ++j) acc += dS[i * L + j] * k[tok_index(dm, r, j, h, c)];",
     "for (int64_t j = 0; j < L; ++j) acc += dS[i * L + j] * q[tok_index(dm, r, j, h, c)];"),
    ("dK scale dropped", "dk[tok_index(dm, r, j, h, c)] = scale * acc;", "dk[tok_index(dm, r, j, h, c)] = acc;"),
    ("dBias not summed over rows", "for (int64_t x = 0; x < L * L; ++x) plane[x] += dS[x];",
     "for (int64_t x = 0; x < L * L; ++x) plane[x] = dS[x];"),
]


LN_MUTATIONS = [
    ("unbiased variance", "v /= (double)C;", "v /= (double)(C - 1);"),
    ("eps outside the square root", "*rstd = 1.0 / sqrt(v + eps);", "*rstd = 1.0 / (sqrt(v) + eps);"),
    ("weight and bias swapped", "y[r * C + c] = xh * (w ? w[c] : 1.0) + (b ? b[c] : 0.0);",
     "y[r * C + c] = xh * (b ? b[c] : 1.0) + (w ? w[c] : 0.0);"),
    ("dx mean term dropped", "dx[r * C + c] = rs * (g - sg - xh * sgx);", "dx[r * C + c] = rs * (g - xh * sgx);"),
    ("dx projection sign", "dx[r * C + c] = rs * (g - sg - xh * sgx);", "dx[r * C + c] = rs * (g - sg + xh * sgx);"),
    ("dx sums without the weight", "const double g = gr[c] * (w ? w[c] : 1.0);\n            sg += g;",
     "const double g = gr[c];\n            sg += g;"),
    ("dw without the normalisation", "if (dw) dw[c] += gr[c] * (xr[c] - mu) * rs;", "if (dw) dw[c] += gr[c] * (xr[c] - mu);"),
]


def _read(path):
    with open(path) as f:
        return f.read()


def _build(attn_text, ln_text, out_dir):
    srcs = []
    for name, text in (("attn", attn_text), ("ln", ln_text)):
        srcs.append(os.path.join(out_dir, name + ".c"))
        with open(srcs[-1], "w") as f:
            f.write(text)
    lib = os.path.join(out_dir, "liboracle.so")
    subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", lib] + srcs + ["-lm"],
                   check=True, capture_output=True)
    return lib


def _pins_pass(lib, pins):
    env = dict(os.environ, EVO_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] + pins,
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return res.returncode == 0, res.stdout[-2000:]


def test_unmutated_copy_passes_the_pins(tmp_path):
    ok, log = _pins_pass(_build(_read(SRC), _read(LN_SRC), str(tmp_path)), PINS + LN_PINS)
    assert ok, log


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new):
    source = _read(SRC)
    assert source.count(old) == 1, "the text to mutate must occur exactly once: %r" % old
    ok, log = _pins_pass(_build(source.replace(old, new), _read(LN_SRC), str(tmp_path)), PINS)
    assert not ok, "no pin caught the planted mistake %r" % name


@pytest.mark.parametrize("name,old,new", LN_MUTATIONS, ids=[m[0] for m in LN_MUTATIONS])
def test_planted_layernorm_mistake_fails_a_pin(tmp_path, name, old, new):
    source = _read(LN_SRC)
    assert source.count(old) == 1, "the text to mutate must occur exactly once: %r" % old
    ok, log = _pins_pass(_build(_read(SRC), source.replace(old, new), str(tmp_path)), LN_PINS)
    assert not ok, "no pin caught the planted mistake %r" % name

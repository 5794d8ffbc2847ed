"""Benchmark of the Evoformer gated attention with pair bias on one MI355X.

One step = one evo_attn_fwd + one evo_attn_bwd over a whole synthetic batch
(the complete hot path: logits, bias, mask, softmax, PV, gate, and the
recompute backward with dQ/dK/dV/dG and the cross-row dBias reduction).
Inputs are resident in HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

Prints ONE JSON line.  `value` is fwd+bwd TFLOP/s (dense count
14*N*H*L^2*d).  `roofline` is measured for the dominant kernel with HIP
events on the stream it runs on; `cpu_baseline` times the fp64 oracle on a
bounded sample of the same workload on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
MFMA_F32_PEAK_TFLOPS = 157.3


def algorithmic_bytes(w, es: int):
    """Bytes each call must move at least once (bias counted once)."""
    tok = w.n_rows * w.seq_len * w.n_heads * w.head_dim * es
    lse = w.n_rows * w.n_heads * w.seq_len * 4
    bias = (w.n_rows // w.rows_per_bias) * w.n_heads * w.seq_len ** 2 * es if w.bias else 0
    dbias = bias // es * 4 if w.bias else 0
    mask = w.n_rows * w.seq_len if w.mask != "none" else 0
    n_gate = 1 if w.gate else 0
    fwd = (3 + n_gate) * tok + bias + mask + tok + lse              # Q K V G bias mask -> O lse
    bwd = (5 + n_gate) * tok + lse + bias + mask + (3 + n_gate) * tok + dbias  # Q K V G O dO lse bias mask -> dQ dK dV dG dBias
    return fwd, bwd


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="tri_start_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-baseline duration")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(rows shard across GPUs with no communication in the forward and one dBias "
              "all-reduce in the backward; see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2404_11068_amd import evo_attn as ea
    from paper_2404_11068_amd import workloads as W

    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, max(args.steps, 1))
        return

    w = W.by_name(args.workload)
    x = W.generate(w)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    es = 2 if w.dtype == "bf16" else 4

    def dev(a):
        if a is None:
            return None
        if w.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

    q, k, v, g, bias, dout = (dev(x[n]) for n in ("q", "k", "v", "gate", "bias", "dout"))
    mask = None if x["mask"] is None else torch.from_numpy(x["mask"]).cuda()
    rpb = w.rows_per_bias
    N, L, H, d = w.n_rows, w.seq_len, w.n_heads, w.head_dim
    out = torch.empty_like(q)
    lse = torch.empty((N, H, L), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    dg = torch.empty_like(q) if g is not None else None
    dbias = torch.empty(bias.shape, dtype=torch.float32, device="cuda") if bias is not None else None
    ws = torch.empty(max(ea.evo_attn_bwd_workspace_size(q, rpb), 1), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def fwd():
        ea.evo_attn_fwd(q, k, v, g, bias, mask, rows_per_bias=rpb, out=out, lse=lse, stream=stream)

    def bwd():
        ea.evo_attn_bwd(q, k, v, g, bias, mask, out, lse, dout, rows_per_bias=rpb, dq=dq, dk=dk,
                        dv=dv, dgate=dg, dbias=dbias, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()

    # timed region: K steps, events around every call on the launch stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for e0, e1, e2 in ev:
        e0.record(stream)
        fwd()
        e1.record(stream)
        bwd()
        e2.record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(stop)
    ms_step = total_ms / args.steps
    fwd_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in ev]))
    bwd_ms = float(np.mean([b.elapsed_time(c) for _, b, c in ev]))

    flops = w.flops_fwd() + w.flops_bwd()
    tflops = flops / (ms_step * 1e-3) / 1e12
    fwd_bytes, bwd_bytes = algorithmic_bytes(w, es)

    # roofline of the forward kernel (one kernel per evo_attn_fwd call, so the
    # event pair around the call brackets exactly that kernel)
    fwd_gbs = fwd_bytes / (fwd_ms * 1e-3) / 1e9
    roofline = {"kernel": "fwd_kernel", "bound": "hbm", "achieved": round(fwd_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(fwd_gbs / HBM_PEAK_GBS, 4),
                "traffic": None, "avg_ms": round(fwd_ms, 5),
                "algorithmic_bytes": fwd_bytes,
                "mfma_tflops": round(w.flops_fwd() / (fwd_ms * 1e-3) / 1e12, 1)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, x, args.cpu_seconds)

    line = {
        "metric": "Evoformer attention fwd+bwd TFLOP/s (bf16) and % MFMA/HBM roofline on 1 MI355X",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "n_rows": N, "seq_len": L, "n_heads": H, "head_dim": d,
                   "rows_per_bias": rpb, "bias": w.bias, "gate": w.gate, "mask": w.mask,
                   "parallelism": "single-gpu"},
        "fwd_ms": round(fwd_ms, 5), "bwd_ms": round(bwd_ms, 5),
        "fwd_bwd_frac_of_mfma_peak": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "fwd_bwd_hbm_gbs": round((fwd_bytes + bwd_bytes) / (ms_step * 1e-3) / 1e9, 1),
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def copy_calibration(torch, mib: int, steps: int):
    """A plain copy of known size: its FETCH_SIZE / WRITE_SIZE counter readings
    turn the counters of the attention kernels into bytes."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        dst.copy_(src)
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    print(json.dumps({"copy_mib": mib, "bytes_read": n * 4, "bytes_written": n * 4, "ms": round(ms, 5),
                      "gbs_read_plus_write": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}))


def cpu_baseline(w, x, target_s: float):
    """The fp64 oracle (forward + backward) on a bounded sample of the workload's
    rows, timed on the host cores; scaled to TFLOP/s of the full row count."""
    import oracle
    from paper_2404_11068_amd import workloads as W

    f = lambda a: None if a is None else W.as_float64(a, w.dtype)

    def run(rows):
        sl = slice(0, rows)
        rpb = min(w.rows_per_bias, rows)
        args = [f(x[n][sl]) for n in ("q", "k", "v")]
        g = None if x["gate"] is None else f(x["gate"][sl])
        b = None if x["bias"] is None else f(x["bias"])[: max(rows // rpb, 1)]
        m = None if x["mask"] is None else x["mask"][sl]
        t = time.perf_counter()
        oracle.forward(*args, g, b, m, rpb)
        oracle.backward(*args, f(x["dout"][sl]), g, b, m, rpb)
        return time.perf_counter() - t

    rows = max(1, min(w.n_rows, 4))
    t = run(rows)
    # grow the sample to roughly target_s of CPU work (bounded by the workload)
    want = int(rows * target_s / max(t, 1e-3))
    want = max(1, min(w.n_rows, want))
    # a sample of at least one whole bias plane keeps whole planes
    if w.bias and want >= w.rows_per_bias:
        want = (want // w.rows_per_bias) * w.rows_per_bias
    t = run(want)
    reps = 1
    if want == w.n_rows and t < target_s:  # the whole workload is short: repeat it
        reps = max(1, int(target_s / max(t, 1e-3)))
        t = sum(run(want) for _ in range(reps)) / reps
    flops = (w.flops_fwd() + w.flops_bwd()) * want / w.n_rows
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds_per_run": round(t, 3), "runs": reps,
            "sample": "%d of %d rows of %s, forward + backward in fp64 (OpenMP), mean of %d run(s)"
                      % (want, w.n_rows, w.name, reps)}


if __name__ == "__main__":
    main()

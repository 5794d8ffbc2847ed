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


def _align(x: int) -> int:
    return (x + 255) // 256 * 256


def kernel_model(w, es: int, ws_bytes: int):
    """Per-launch algorithmic traffic (each input and output of the kernel
    counted once, the shared bias plane once) and MFMA flops of every kernel
    of one step, in launch order.  T = one [N, L, H, d] token tensor."""
    N, L, H, d = w.n_rows, w.seq_len, w.n_heads, w.head_dim
    T = N * L * H * d * es
    lse = N * H * L * 4
    B = N // w.rows_per_bias if w.bias else 0
    bias = B * H * L * L * es
    mask = N * L if w.mask != "none" else 0
    g = 1 if w.gate else 0
    S = N * H * L * L  # logits
    parts = max(0, ws_bytes - _align(T) - _align(lse) - (_align(bias) if w.bias else 0))
    ks = [("fwd_kernel", (3 + g) * T + bias + mask + T + lse, 4.0 * S * d)]
    if w.bias:
        ks.append(("bias_transpose", 2 * bias, 0.0))
    # dK/dV pass: reads Q K V O dO [G] lse bias^T mask, writes dK dV dA [dG] Dsum
    ks.append(("kv_kernel", (5 + g) * T + lse + bias + mask + (3 + g) * T + lse, 8.0 * S * d))
    # dQ/dBias pass: reads Q K V dA lse Dsum bias mask, writes dQ and the partial dBias planes
    ks.append(("qbias_kernel", 4 * T + 2 * lse + bias + mask + T + parts, 6.0 * S * d))
    if w.bias:
        ks.append(("dbias_reduce", parts + B * H * L * L * 4, 0.0))
    return ks


def algorithmic_bytes(w, es: int):
    """Bytes the forward and the backward must move at least once."""
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
    ap.add_argument("--source-hash", action="store_true", help="print the kernel-source hash and exit")
    args = ap.parse_args()
    if args.source_hash:
        print(kernel_source_hash())
        return
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

    def bwd(events=None):
        ea.evo_attn_bwd(q, k, v, g, bias, mask, out, lse, dout, rows_per_bias=rpb, dq=dq, dk=dk,
                        dv=dv, dgate=dg, dbias=dbias, workspace=ws, stream=stream, events=events)

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()

    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, stop = mk(), mk()

    # timed region: K plain steps bracketed by events on the launch stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        fwd()
        bwd()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start.elapsed_time(stop)
    ms_step = total_ms / args.steps

    # per-kernel timing: K more steps with events on the launch stream around
    # the forward kernel and (through evo_attn_bwd_traced) around every
    # backward kernel; recording them adds a few microseconds per event, which
    # is why the headline time above comes from plain steps
    nk = ea.evo_attn_bwd_kernel_count(bias is not None)
    fev = [(mk(), mk()) for _ in range(args.steps)]
    bev = [[mk() for _ in range(nk + 1)] for _ in range(args.steps)]
    for e in [x for p_ in fev for x in p_] + [x for l_ in bev for x in l_]:
        e.record(stream)  # create the HIP events before timing
    torch.cuda.synchronize()
    for (e0, e1), evs in zip(fev, bev):
        e0.record(stream)
        fwd()
        e1.record(stream)
        bwd(evs)
    torch.cuda.synchronize()
    fwd_ms = float(np.mean([a.elapsed_time(b) for a, b in fev]))
    bwd_ms = float(np.mean([l_[0].elapsed_time(l_[-1]) for l_ in bev]))
    kern_ms = [fwd_ms] + [float(np.mean([l_[j].elapsed_time(l_[j + 1]) for l_ in bev])) for j in range(nk)]

    flops = w.flops_fwd() + w.flops_bwd()
    tflops = flops / (ms_step * 1e-3) / 1e12
    fwd_bytes, bwd_bytes = algorithmic_bytes(w, es)
    model = kernel_model(w, es, ws.numel())
    assert len(model) == len(kern_ms), (len(model), len(kern_ms))
    kernels = {}
    for (name, nbytes, kflops), ms in zip(model, kern_ms):
        kernels[name] = {"avg_ms": round(ms, 5), "algorithmic_bytes": int(nbytes),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "mfma_tflops": round(kflops / (ms * 1e-3) / 1e12, 1)}
    dom = max(range(len(model)), key=lambda i: kern_ms[i])
    dname, dbytes, dflops = model[dom]
    dms = kern_ms[dom]
    peak_mfma = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
    ridge = peak_mfma * 1e12 / (HBM_PEAK_GBS * 1e9)          # flop per byte
    if dflops / max(dbytes, 1) >= ridge:
        ach = dflops / (dms * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(ach, 2), "peak": peak_mfma, "unit": "TFLOP/s",
                    "frac": round(ach / peak_mfma, 4)}
    else:
        ach = dbytes / (dms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(ach / HBM_PEAK_GBS, 4)}
    roofline.update({"traffic": measured_traffic(dname, w.name), "kernel": dname, "avg_ms": round(dms, 5),
                     "algorithmic_bytes": int(dbytes), "flops": dflops,
                     "intensity_flop_per_byte": round(dflops / max(dbytes, 1), 1)})

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
        "fwd_ms": round(fwd_ms, 5), "bwd_ms": round(bwd_ms, 5), "kernels": kernels,
        "fwd_bwd_frac_of_mfma_peak": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "fwd_bwd_hbm_gbs": round((fwd_bytes + bwd_bytes) / (ms_step * 1e-3) / 1e9, 1),
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary
    (profiles/traffic.json: FETCH_SIZE and WRITE_SIZE scaled by a plain copy
    kernel's readings), or None when there is none for this kernel and
    workload or the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            entries = json.load(f)
    except (OSError, ValueError):
        return None
    for e in entries.get("entries", []):
        if e.get("kernel") == kernel and e.get("workload") == workload:
            if e.get("source_sha256") != kernel_source_hash():
                return None
            return e.get("bytes_per_launch")
    return None


def kernel_source_hash() -> str:
    """sha256 over the HIP sources and headers that define the kernels."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2404_11068_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


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

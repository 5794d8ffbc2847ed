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
import ctypes
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


def bias_transposed(w, es: int) -> bool:
    """The backward transposes the bias in a kernel of its own only for fp32
    or a seq_len that is not a multiple of 8 (bf16 rows of whole 16-byte
    groups are read as they are by the dK/dV pass)."""
    return bool(w.bias) and not (es == 2 and w.seq_len % 8 == 0)


def fused_backward(w, es: int) -> bool:
    """Whether the library runs the single-pass backward for this workload:
    bf16 with head_dim <= 32; with a bias only where the chunk's dBias
    accumulators fit (up to 128 keys, or head_dim 8 with rows of whole
    16-byte groups)."""
    if es != 2 or w.head_dim > 32:
        return False
    if not w.bias:
        return True
    nkt = (w.seq_len + 31) // 32
    return nkt <= 4 or (w.head_dim == 8 and w.seq_len % 8 == 0)


def forward_kernel(w, es: int) -> str:
    """The forward kernel the library runs for this workload: the row-walking
    kernel (bias rows held in registers across the rows of one head) for bf16
    at head_dim <= 32 and at most 256 keys in 16-byte rows, when all rows
    share one bias plane and there are at least two (row, head) units per
    resident workgroup; the one-unit kernel otherwise."""
    if es != 2 or w.head_dim > 32 or not w.bias or w.seq_len % 8 or w.seq_len > 256:
        return "fwd_kernel"
    if w.rows_per_bias < w.n_rows:
        return "fwd_kernel"
    nkt = 1
    while nkt * 32 < w.seq_len:
        nkt *= 2
    g0 = 256 * 8 // nkt
    g = g0 // 8 // w.n_heads * 8 * w.n_heads
    units = w.n_rows * w.n_heads
    return "fwd_rows_kernel" if g > 0 and units >= 2 * g0 else "fwd_kernel"


def kernel_model(w, es: int, ws_bytes: int):
    """Per-launch traffic and MFMA flops of every kernel of one step, in launch
    order, as (name, algorithmic bytes, workspace bytes, flops).

    Algorithmic bytes count only the method's own tensors that the kernel
    reads or writes, each once (Q, K, V, G, O, dO, LSE, bias, mask, dQ, dK, dV,
    dG, fp32 dBias; the shared bias plane once per launch).  The kernel's own
    scratch traffic -- dA and Dsum handed between the backward passes, the
    transposed bias, the partial dBias planes -- is workspace, reported apart.
    T = one [N, L, H, d] token tensor."""
    N, L, H, d = w.n_rows, w.seq_len, w.n_heads, w.head_dim
    T = N * L * H * d * es
    lse = N * H * L * 4
    B = N // w.rows_per_bias if w.bias else 0
    bias = B * H * L * L * es
    dbias = B * H * L * L * 4
    mask = N * L if w.mask != "none" else 0
    g = 1 if w.gate else 0
    S = N * H * L * L  # logits
    fwd = (forward_kernel(w, es), (3 + g) * T + bias + mask + T + lse, 0, 4.0 * S * d)
    if fused_backward(w, es):
        # one pass: reads Q K V O dO [G] lse bias mask, writes dQ dK dV [dG]
        # (and dBias itself when each plane is one row chunk); workspace:
        # writes the partial dBias planes, which the reduction reads
        parts = ws_bytes if w.bias else 0
        ks = [fwd, ("bwd_fused_kernel", (5 + g) * T + lse + bias + mask + (3 + g) * T + (0 if parts else dbias),
                    parts, 10.0 * S * d)]
        if w.bias and parts:
            ks.append(("dbias_tiles_reduce", dbias, parts, 0.0))
        return ks
    transposed = bias_transposed(w, es)
    biast = bias if transposed else 0
    dsum = lse
    parts = max(0, ws_bytes - _align(T) - _align(dsum) - (_align(biast) if transposed else 0))
    ks = [fwd]
    if transposed:
        ks.append(("bias_transpose", bias, biast, 0.0))
    # dK/dV pass: reads Q K V O dO [G] lse bias mask, writes dK dV [dG];
    # workspace: writes dA and Dsum (and reads the transposed bias)
    ks.append(("kv_kernel", (5 + g) * T + lse + (0 if transposed else bias) + mask + (2 + g) * T,
               T + dsum + biast, 8.0 * S * d))
    # dQ/dBias pass: reads Q K V lse bias mask, writes dQ; workspace: reads dA
    # and Dsum, writes the partial dBias planes
    ks.append(("qbias_kernel", 3 * T + lse + bias + mask + T, T + dsum + parts, 6.0 * S * d))
    if w.bias:
        ks.append(("dbias_reduce", dbias, parts, 0.0))
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
    # the GPU's clock rises over the first ~30 ms of continuous work after an
    # idle period (a step of the triangle workload: ~140 us in its first 50
    # steps, ~116 us from about step 250 on), so the untimed warm-up runs 300
    # steps by default and the timed steps see the clock a training loop runs at
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--workload", default="tri_start_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-baseline duration")
    ap.add_argument("--rate-calibration", action="store_true",
                    help="only measure the vector ALU's exp2 and fma lane-op rates (evo_probe_rate)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (reference for HBM byte counters)")
    ap.add_argument("--source-hash", nargs="?", const="attn", default=None, choices=sorted(KERNEL_SOURCES),
                    help="print the source hash of a kernel family and exit")
    args = ap.parse_args()
    if args.source_hash:
        print(kernel_source_hash(args.source_hash))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(rows shard across GPUs with no communication in the forward and one dBias "
              "all-reduce in the backward; see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2404_11068_amd import evo_attn as ea
    from paper_2404_11068_amd import workloads as W

    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, max(args.steps, 1))
        return
    if args.rate_calibration:
        rate_calibration(torch, max(args.steps, 1))
        return

    if args.workload.startswith("ln_"):
        ln_bench(torch, args)
        return
    if args.workload.startswith("proj_"):
        proj_bench(torch, args)
        return
    if args.workload.startswith("pb_"):
        pair_bias_bench(torch, args)
        return
    if args.workload.startswith("adam_"):
        optim_bench(torch, args)
        return
    if args.workload.startswith("graph_"):
        graph_bench(torch, args)
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
    fwd_warm = [a.elapsed_time(b) for a, b in fev]
    bwd_warm = [l_[0].elapsed_time(l_[-1]) for l_ in bev]
    fwd_ms = float(np.mean(fwd_warm))
    bwd_ms = float(np.mean(bwd_warm))
    kern_ms = [fwd_ms] + [float(np.mean([l_[j].elapsed_time(l_[j + 1]) for l_ in bev])) for j in range(nk)]
    model = kernel_model(w, es, ws.numel())
    if fused_backward(w, es):
        kern_ms = kern_ms[:len(model)]  # the slots after the last kernel bracket nothing
    elif w.bias and not bias_transposed(w, es):
        del kern_ms[1]  # the transpose slot brackets no kernel

    # cold mode: a 512 MiB scratch buffer is written before every timed call
    # (outside the events), which evicts the inputs from L2 and the Infinity
    # Cache, so each call reads them from HBM
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cev = [[mk() for _ in range(4)] for _ in range(args.steps)]
    for e in [x for l_ in cev for x in l_]:
        e.record(stream)
    torch.cuda.synchronize()
    for e0, e1, e2, e3 in cev:
        flush.fill_(1)
        e0.record(stream)
        fwd()
        e1.record(stream)
        flush.fill_(2)
        e2.record(stream)
        bwd()
        e3.record(stream)
    torch.cuda.synchronize()
    fwd_cold = [l_[0].elapsed_time(l_[1]) for l_ in cev]
    bwd_cold = [l_[2].elapsed_time(l_[3]) for l_ in cev]
    del flush

    flops = w.flops_fwd() + w.flops_bwd()
    tflops = flops / (ms_step * 1e-3) / 1e12
    fwd_bytes, bwd_bytes = algorithmic_bytes(w, es)
    assert len(model) == len(kern_ms), (len(model), len(kern_ms))
    kernels = {}
    for (name, nbytes, wsb, kflops), ms in zip(model, kern_ms):
        tr = measured_traffic(name, w.name)
        kernels[name] = {"avg_ms": round(ms, 5), "algorithmic_bytes": int(nbytes),
                         "workspace_bytes": int(wsb),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         "mfma_tflops": round(kflops / (ms * 1e-3) / 1e12, 1),
                         "traffic": tr,
                         "traffic_over_algorithmic": None if tr is None or not nbytes else round(tr / nbytes, 3)}
    dom = max(range(len(model)), key=lambda i: kern_ms[i])
    dname, dbytes, _, dflops = model[dom]
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
    dtr = measured_traffic(dname, w.name)
    roofline.update({"traffic": dtr, "kernel": dname, "avg_ms": round(dms, 5),
                     "algorithmic_bytes": int(dbytes), "flops": dflops,
                     "intensity_flop_per_byte": round(dflops / max(dbytes, 1), 1),
                     "traffic_over_algorithmic": None if dtr is None else round(dtr / max(dbytes, 1), 3)})
    step_traffic = [measured_traffic(n, w.name) for n, _, _, _ in model]
    step_traffic = None if any(t is None for t in step_traffic) else int(sum(step_traffic))

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] GPU timing done; timing the CPU oracle (about %.0f s)" % args.cpu_seconds,
              file=sys.stderr, flush=True)
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
        "fwd_tflops": round(w.flops_fwd() / (fwd_ms * 1e-3) / 1e12, 2),
        "bwd_tflops": round(w.flops_bwd() / (bwd_ms * 1e-3) / 1e12, 2),
        "timing": {
            "warm": {"note": "calls back to back, inputs resident in HBM and partly in caches",
                     "fwd_ms": _pct(fwd_warm), "bwd_ms": _pct(bwd_warm)},
            "cold": {"note": "512 MiB scratch written before each call, outside the events",
                     "fwd_ms": _pct(fwd_cold), "bwd_ms": _pct(bwd_cold),
                     "fwd_bwd_tflops_median": round(flops / ((np.median(fwd_cold) + np.median(bwd_cold))
                                                             * 1e-3) / 1e12, 2)},
        },
        "kernels": kernels,
        "fwd_bwd_frac_of_mfma_peak": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "fwd_bwd_hbm_gbs": round((fwd_bytes + bwd_bytes) / (ms_step * 1e-3) / 1e9, 1),
        "step_hbm": {"algorithmic_bytes": int(fwd_bytes + bwd_bytes),
                     "frac": round((fwd_bytes + bwd_bytes) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": step_traffic,
                     "traffic_over_algorithmic": None if step_traffic is None
                     else round(step_traffic / (fwd_bytes + bwd_bytes), 3)},
        "wall_s": round(wall, 3),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def ln_bench(torch, args):
    """LayerNorm forward + backward on one of the LayerNorm workloads: one step
    is evo_layernorm_fwd + evo_layernorm_bwd over the whole [R, C] tensor.
    `value` is algorithmic HBM bytes of the step (each tensor touched once)
    per second; the roofline is the HBM bound of the dominant kernel."""
    from paper_2404_11068_amd import layernorm as ln
    from paper_2404_11068_amd import workloads as W

    w = W.ln_by_name(args.workload)
    x = W.generate_ln(w)
    es = 2 if w.dtype == "bf16" else 4

    def dev(a):
        if w.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

    xd, dyd = dev(x["x"]), dev(x["dy"])
    wt, bt = torch.from_numpy(x["weight"]).cuda(), torch.from_numpy(x["bias"]).cuda()
    R, C = w.n_rows, w.n_cols
    y = torch.empty_like(xd)
    dx = torch.empty_like(xd)
    mean = torch.empty(R, dtype=torch.float32, device="cuda")
    rstd = torch.empty(R, dtype=torch.float32, device="cuda")
    dw = torch.empty(C, dtype=torch.float32, device="cuda")
    db = torch.empty(C, dtype=torch.float32, device="cuda")
    ws_bytes = ln.workspace_size(xd, w.eps)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    n_part = ws_bytes // (2 * C * 4)
    stream = torch.cuda.current_stream()

    def fwd():
        ln.layernorm_fwd(xd, wt, bt, w.eps, y=y, mean=mean, rstd=rstd, stream=stream)

    def bwd(events=None):
        ln.layernorm_bwd(xd, wt, mean, rstd, dyd, dx=dx, dweight=dw, dbias=db, workspace=ws, eps=w.eps,
                         stream=stream, events=events)

    for _ in range(args.warmup):
        fwd()
        bwd()
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, stop = mk(), mk()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        fwd()
        bwd()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps

    fev = [(mk(), mk()) for _ in range(args.steps)]
    bev = [[mk() for _ in range(3)] for _ in range(args.steps)]
    for e in [e for p_ in fev for e in p_] + [e for l_ in bev for e in l_]:
        e.record(stream)
    torch.cuda.synchronize()
    for (e0, e1), evs in zip(fev, bev):
        e0.record(stream)
        fwd()
        e1.record(stream)
        bwd(evs)
    torch.cuda.synchronize()
    fwd_warm = [a.elapsed_time(b) for a, b in fev]
    bwd_warm = [l_[0].elapsed_time(l_[2]) for l_ in bev]
    k_ms = [float(np.mean(fwd_warm)), float(np.mean([l_[0].elapsed_time(l_[1]) for l_ in bev])),
            float(np.mean([l_[1].elapsed_time(l_[2]) for l_ in bev]))]

    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cev = [[mk() for _ in range(4)] for _ in range(args.steps)]
    for e in [e for l_ in cev for e in l_]:
        e.record(stream)
    torch.cuda.synchronize()
    for e0, e1, e2, e3 in cev:
        flush.fill_(1)
        e0.record(stream)
        fwd()
        e1.record(stream)
        flush.fill_(2)
        e2.record(stream)
        bwd()
        e3.record(stream)
    torch.cuda.synchronize()
    fwd_cold = [l_[0].elapsed_time(l_[1]) for l_ in cev]
    bwd_cold = [l_[2].elapsed_time(l_[3]) for l_ in cev]

    # context: a plain device copy x -> y moves the forward's bytes (read R*C,
    # write R*C); its time at this size shows what HBM delivers to a kernel
    # this short, launch and ramp included
    copy_ms = {}
    for mode in ("warm", "cold"):
        ev = [(mk(), mk()) for _ in range(args.steps)]
        for a, b in ev:
            if mode == "cold":
                flush.fill_(3)
            a.record(stream)
            y.copy_(xd)
            b.record(stream)
        torch.cuda.synchronize()
        copy_ms[mode] = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del flush

    tok = R * C * es
    part = n_part * 2 * C * 4
    model = [("ln_fwd_kernel", 2 * tok + 8 * R + 8 * C),
             ("ln_bwd_kernel", 3 * tok + 8 * R + 4 * C + part),
             ("ln_param_reduce", part + 8 * C)]
    kernels = {}
    for (name, nbytes), ms in zip(model, k_ms):
        kernels[name] = {"avg_ms": round(ms, 5), "algorithmic_bytes": int(nbytes),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1)}
    dom = max(range(len(model)), key=lambda i: k_ms[i])
    dname, dbytes = model[dom]
    ach = dbytes / (k_ms[dom] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic(dname, w.name),
                "kernel": dname, "avg_ms": round(k_ms[dom], 5), "algorithmic_bytes": int(dbytes)}
    step_bytes = w.bytes_fwd() + w.bytes_bwd()
    cpu = None if args.no_cpu_baseline else ln_cpu_baseline(w, x, args.cpu_seconds)
    line = {
        "metric": "LayerNorm fwd+bwd throughput (algorithmic HBM bytes per second) on 1 MI355X",
        "value": round(step_bytes / (ms_step * 1e-3) / 1e9, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "n_rows": R, "n_cols": C, "eps": w.eps, "parallelism": "single-gpu"},
        "fwd_ms": round(k_ms[0], 5), "bwd_ms": round(float(np.mean(bwd_warm)), 5),
        "fwd_gbs": round(w.bytes_fwd() / (k_ms[0] * 1e-3) / 1e9, 1),
        "bwd_gbs": round(w.bytes_bwd() / (float(np.mean(bwd_warm)) * 1e-3) / 1e9, 1),
        "timing": {
            "warm": {"note": "calls back to back, inputs resident in HBM and partly in caches",
                     "fwd_ms": _pct(fwd_warm), "bwd_ms": _pct(bwd_warm)},
            "cold": {"note": "512 MiB scratch written before each call, outside the events",
                     "fwd_ms": _pct(fwd_cold), "bwd_ms": _pct(bwd_cold),
                     "fwd_bwd_gbs_median": round(step_bytes / ((np.median(fwd_cold) + np.median(bwd_cold))
                                                               * 1e-3) / 1e9, 1)},
        },
        "reference_copy": {"note": "torch device copy of x (same bytes as the forward), event-timed median",
                           "bytes": 2 * tok, "warm_ms": round(copy_ms["warm"], 5),
                           "cold_ms": round(copy_ms["cold"], 5)},
        "kernels": kernels, "wall_s": round(wall, 3), "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def proj_bench(torch, args):
    """Fused LayerNorm + batched projections (forward) on one of the
    projection workloads: one step is one evo_ln_proj_fwd over all tokens.
    `value` is TFLOP/s of the products (2*R*C*P*HD); the roofline is the
    kernel's HBM bound (its intensity is below the bf16 ridge point)."""
    from paper_2404_11068_amd import proj as pj
    from paper_2404_11068_amd import workloads as W

    w = W.proj_by_name(args.workload)
    d = W.generate_proj(w)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    x, Wt = bf(d["x"]), bf(d["weight"])
    lnw, lnb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    b = None if d["bias"] is None else torch.from_numpy(d["bias"]).cuda()
    outs = [torch.empty((w.n_rows, w.proj_dim), dtype=torch.bfloat16, device="cuda") for _ in range(w.n_proj)]
    stream = torch.cuda.current_stream()

    def step():
        pj.ln_proj_fwd(x, lnw, lnb, Wt, b, n_proj=w.n_proj, eps=w.eps, outs=outs, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, stop = mk(), mk()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    res = {}
    for mode in ("warm", "cold"):
        ev = [(mk(), mk()) for _ in range(args.steps)]
        for a, b_ in ev:
            a.record(stream)
            b_.record(stream)
        torch.cuda.synchronize()
        for a, b_ in ev:
            if mode == "cold":
                flush.fill_(1)
            a.record(stream)
            step()
            b_.record(stream)
        torch.cuda.synchronize()
        res[mode] = [a.elapsed_time(b_) for a, b_ in ev]
    del flush
    # backward (training forward saves the normalised input): dY product,
    # LayerNorm backward, weight-gradient product and the partial sums
    y = torch.empty_like(x)
    _, mean, rstd = pj.ln_proj_fwd(x, lnw, lnb, Wt, b, n_proj=w.n_proj, eps=w.eps, need_stats=True, y_norm=y,
                                   stream=stream)
    gen = torch.Generator(device="cpu").manual_seed(w.seed + 1)
    douts = [torch.randn(w.n_rows, w.proj_dim, generator=gen).to(torch.bfloat16).cuda() for _ in range(w.n_proj)]
    bufs = dict(dx=torch.empty_like(x), dweight=torch.empty(w.n_proj * w.proj_dim, w.c_in, device="cuda"),
                dbias=torch.empty(w.n_proj * w.proj_dim, device="cuda") if b is not None else None,
                dln_weight=torch.empty(w.c_in, device="cuda"), dln_bias=torch.empty(w.c_in, device="cuda"))
    wsb = torch.empty(max(1, int(pj._lib().evo_ln_proj_bwd_workspace_size(ctypes.byref(
        pj.evo_proj_dims(1, w.c_in, w.n_proj, w.proj_dim, w.n_rows, w.eps, 0))))), dtype=torch.uint8, device="cuda")

    def bwd():
        pj.ln_proj_bwd(x, lnw, mean, rstd, y, Wt, douts, eps=w.eps, has_bias=b is not None, workspace=wsb,
                       stream=stream, **bufs)

    for _ in range(args.warmup):
        bwd()
    torch.cuda.synchronize()
    bev = [(mk(), mk()) for _ in range(args.steps)]
    for a_, b2 in bev:
        a_.record(stream)
        bwd()
        b2.record(stream)
    torch.cuda.synchronize()
    bwd_ms = [a_.elapsed_time(b2) for a_, b2 in bev]
    bwd_flops = 2.0 * w.flops()
    k_ms = float(np.mean(res["warm"]))
    nbytes = w.bytes()
    ach = nbytes / (k_ms * 1e-3) / 1e9
    flops = w.flops()
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic("ln_proj_kernel", w.name),
                "kernel": "ln_proj_kernel", "avg_ms": round(k_ms, 5), "algorithmic_bytes": int(nbytes),
                "flops": flops, "intensity_flop_per_byte": round(flops / nbytes, 1),
                "mfma_frac": round(flops / (k_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    cpu = None if args.no_cpu_baseline else proj_cpu_baseline(w, d, args.cpu_seconds)
    line = {
        "metric": "Fused LayerNorm + batched q/k/v/gate projections, TFLOP/s on 1 MI355X",
        "value": round(flops / (ms_step * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "n_rows": w.n_rows, "c_in": w.c_in, "n_proj": w.n_proj,
                   "proj_dim": w.proj_dim, "bias": w.bias, "parallelism": "single-gpu"},
        "gbs": round(nbytes / (ms_step * 1e-3) / 1e9, 1),
        "bwd_ms": _pct(bwd_ms),
        "bwd_tflops": round(bwd_flops / (float(np.median(bwd_ms)) * 1e-3) / 1e12, 2),
        "timing": {"warm": {"note": "calls back to back", "ms": _pct(res["warm"])},
                   "cold": {"note": "512 MiB scratch written before each call, outside the events",
                            "ms": _pct(res["cold"])}},
        "wall_s": round(wall, 3), "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def pair_bias_bench(torch, args):
    """Pair bias (LayerNorm of each pair entry + bias-free projection to the
    heads, written in the attention's bias layout) on one pair-bias workload.
    `value` is algorithmic HBM bytes per second (read z, write the bias)."""
    from paper_2404_11068_amd import proj as pj
    from paper_2404_11068_amd import workloads as W

    w = W.pair_bias_by_name(args.workload)
    d = W.generate_pair_bias(w)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    z, Wt = bf(d["z"]), bf(d["weight"])
    lnw, lnb = torch.from_numpy(d["ln_weight"]).cuda(), torch.from_numpy(d["ln_bias"]).cuda()
    L, H = w.seq_len, w.n_heads
    out = torch.empty((w.n_batch, H, L, L), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        pj.ln_pair_bias_fwd(z, lnw, lnb, Wt, w.eps, w.transpose, out=out, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, stop = mk(), mk()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    res = {}
    for mode in ("warm", "cold"):
        ev = [(mk(), mk()) for _ in range(args.steps)]
        for a, b_ in ev:
            a.record(stream)
            b_.record(stream)
        torch.cuda.synchronize()
        for a, b_ in ev:
            if mode == "cold":
                flush.fill_(1)
            a.record(stream)
            step()
            b_.record(stream)
        torch.cuda.synchronize()
        res[mode] = [a.elapsed_time(b_) for a, b_ in ev]
    del flush
    # backward from an fp32 dbias in the forward's layout: dz, dweight, dln
    gen = torch.Generator(device="cpu").manual_seed(w.seed + 1)
    gshape = (w.n_batch, H, L, L)  # square: the same shape in either layout
    g = torch.randn(gshape, generator=gen).cuda()
    C = w.c_in
    bbufs = dict(dz=torch.empty_like(z), dweight=torch.empty(H, C, device="cuda"),
                 dln_weight=torch.empty(C, device="cuda"), dln_bias=torch.empty(C, device="cuda"),
                 workspace=torch.empty(max(16, pj.pair_bias_bwd_workspace_size(w.n_batch, L, L, C, H, w.transpose)),
                                       dtype=torch.uint8, device="cuda"))

    def bwd():
        pj.ln_pair_bias_bwd(z, lnw, lnb, Wt, g, w.eps, w.transpose, stream=stream, **bbufs)

    for _ in range(args.warmup):
        bwd()
    torch.cuda.synchronize()
    bev = [(mk(), mk()) for _ in range(args.steps)]
    for a_, b2 in bev:
        a_.record(stream)
        bwd()
        b2.record(stream)
    torch.cuda.synchronize()
    bwd_ms = [a_.elapsed_time(b2) for a_, b2 in bev]
    # algorithmic bytes: read z and dbias, write dz, partial rows out and back
    n_ent = w.n_batch * L * L
    bwd_bytes = 4 * n_ent * C + 4 * n_ent * H + 2 * bbufs["workspace"].numel()
    k_ms = float(np.mean(res["warm"]))
    nbytes = w.bytes()
    ach = nbytes / (k_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic("pair_bias_kernel", w.name),
                "kernel": "pair_bias_kernel", "avg_ms": round(k_ms, 5), "algorithmic_bytes": int(nbytes)}
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        zf, Wf = W.as_float64(d["z"], "bf16"), W.as_float64(d["weight"], "bf16")
        run = lambda: oracle.pair_bias_forward(zf, d["ln_weight"], d["ln_bias"], Wf, w.eps, w.transpose)
        t1 = time.perf_counter()
        run()
        t = time.perf_counter() - t1
        reps = max(1, int(args.cpu_seconds / max(t, 1e-3)))
        ts = []
        for _ in range(reps):
            t1 = time.perf_counter()
            run()
            ts.append(time.perf_counter() - t1)
        t = float(np.median(ts))
        cpu = {"value": round(nbytes / t / 1e9, 3), "unit": "GB/s", "cores": oracle.threads(), "kind": "oracle",
               "cpu_model": _cpu_model(), "seconds_per_run": round(t, 4), "runs": reps,
               "sample": "whole workload, LayerNorm (C, OpenMP) + numpy fp64 matmul, median of %d runs" % reps}
    line = {
        "metric": "Pair bias (LayerNorm + projection to heads, attention layout), GB/s on 1 MI355X",
        "value": round(nbytes / (ms_step * 1e-3) / 1e9, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "bwd_ms": _pct(bwd_ms), "bwd_algorithmic_bytes": int(bwd_bytes),
        "bwd_gbs": round(bwd_bytes / (float(np.median(bwd_ms)) * 1e-3) / 1e9, 1),
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "n_batch": w.n_batch, "seq_len": L, "c_in": w.c_in, "n_heads": H,
                   "transpose": w.transpose, "parallelism": "single-gpu"},
        "timing": {"warm": {"note": "calls back to back", "ms": _pct(res["warm"])},
                   "cold": {"note": "512 MiB scratch written before each call, outside the events",
                            "ms": _pct(res["cold"])}},
        "wall_s": round(wall, 3), "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(line))


def optim_bench(torch, args):
    """Optimizer step over every parameter tensor of an AlphaFold-sized model:
    gradient-norm clipping (two kernels) then the fused Adam + SWA kernel.
    `value` is algorithmic HBM bytes per second of the whole step."""
    from paper_2404_11068_amd import optim as op
    from paper_2404_11068_amd import workloads as W

    w = W.optim_by_name(args.workload)
    d = W.generate_optim(w)
    dev = lambda lst: [torch.from_numpy(a).cuda() for a in lst]
    P, G, M, V, S = (dev(d[k]) for k in ("params", "grads", "exp_avg", "exp_avg_sq", "swa"))
    opt = op.FusedAdamSWA(P, G, M, V, S, lr=w.lr, betas=w.betas, eps=w.eps, swa_decay=w.swa_decay)
    stream = torch.cuda.current_stream()
    step_no = [w.step]

    def step():
        opt.step(max_norm=w.max_norm, stream=stream, step=step_no[0])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    start, stop = mk(), mk()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps
    # per phase: clipping (sum-of-squares + scale kernels), then the Adam + SWA kernel alone
    ev = [[mk() for _ in range(3)] for _ in range(args.steps)]
    for l_ in ev:
        for e in l_:
            e.record(stream)
    torch.cuda.synchronize()
    for e0, e1, e2 in ev:
        e0.record(stream)
        opt.clip(w.max_norm, stream)
        e1.record(stream)
        opt.step(max_norm=None, stream=stream, step=step_no[0])
        e2.record(stream)
    torch.cuda.synchronize()
    clip_ms = [a.elapsed_time(b) for a, b, _ in ev]
    adam_ms = [b.elapsed_time(c) for _, b, c in ev]
    k_ms = float(np.mean(adam_ms))
    nbytes = w.bytes_step()
    ach = nbytes / (k_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic("adam_swa_kernel", w.name),
                "kernel": "adam_swa_kernel", "avg_ms": round(k_ms, 5), "algorithmic_bytes": int(nbytes)}
    total = nbytes + w.bytes_clip()
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import optim_oracle as oo
        sub = slice(None, None, 10)
        f64 = {k: [a.astype(np.float64) for a in d[k][sub]] for k in d}
        n_sub = sum(a.size for a in f64["params"])
        reps, ts = 0, []
        while sum(ts) < args.cpu_seconds and reps < 50:
            t1 = time.perf_counter()
            _, sc = oo.grad_norm_scale(f64["grads"], w.max_norm)
            oo.adam_swa_step(f64["params"], f64["grads"], f64["exp_avg"], f64["exp_avg_sq"], f64["swa"], lr=w.lr,
                             beta1=w.betas[0], beta2=w.betas[1], eps=w.eps, weight_decay=0.0, step=w.step,
                             swa_decay=w.swa_decay, grad_scale=sc)
            ts.append(time.perf_counter() - t1)
            reps += 1
        t = float(np.median(ts))
        cpu = {"value": round(40 * n_sub / t / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
               "cpu_model": _cpu_model(), "seconds_per_run": round(t, 4), "runs": reps,
               "sample": "every 10th tensor (%d elements), clipping + Adam + SWA in numpy fp64, median of %d runs"
                         % (n_sub, reps)}
    line = {
        "metric": "Optimizer step (grad clipping + fused Adam + SWA over all parameters), GB/s on 1 MI355X",
        "value": round(total / (ms_step * 1e-3) / 1e9, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "tensors": len(P), "elements": w.numel(), "chunks": opt.n_chunks,
                   "max_norm": w.max_norm, "parallelism": "single-gpu"},
        "clip_ms": _pct(clip_ms), "adam_swa_ms": _pct(adam_ms),
        "wall_s": round(wall, 3), "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(line))


GRAPH_WORKLOADS = {
    # MSA row attention with pair bias at one GPU's share under 8-way dynamic axial parallelism
    # (128 MSA rows / 8 = 16 rows of 256 residues), and the whole 128-row module; one step is the
    # projections, the pair bias, attention forward and backward and the projections' backward
    "graph_msa_row_dap8": dict(N=16, L=256),
    "graph_msa_row_full": dict(N=128, L=256),
    # a launch-bound size: 4 rows of 64 residues (GPU work well below the host's launch cost)
    "graph_msa_row_small": dict(N=4, L=64),
}


def graph_bench(torch, args):
    """One MSA-row-attention step (LayerNorm + q/k/v/g projections, pair bias,
    attention forward, output projection, and the backward of each: 8 C-ABI
    calls, 17 kernels) run eagerly through the Python binding and replayed
    from the HIP graph cache.
    `value` is graphed steps per second; the eager rate, the host time to
    enqueue one step and the speedup are reported beside it."""
    from paper_2404_11068_amd import graph as gr

    cfg = GRAPH_WORKLOADS[args.workload]
    step = gr.MSARowAttentionStep(N=cfg["N"], L=cfg["L"], seed=11)
    s = torch.cuda.Stream()
    cache = gr.GraphCache(capacity=4)
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def run(fn, n):
        torch.cuda.synchronize()
        e0, e1 = mk(), mk()
        t0 = time.perf_counter()
        e0.record(s)
        for _ in range(n):
            fn()
        t_enq = time.perf_counter() - t0
        e1.record(s)
        torch.cuda.synchronize()
        t_all = time.perf_counter() - t0
        return t_enq / n * 1e3, t_all / n * 1e3, e0.elapsed_time(e1) / n

    eager = lambda: step.record(s)
    graphed = lambda: cache.run(step.key(), step.record, s)
    for _ in range(args.warmup):
        eager()
        graphed()
    res = {}
    for name, fn in (("eager", eager), ("graph", graphed)):
        enq, wall, gpu = run(fn, args.steps)
        res[name] = {"host_enqueue_ms_per_step": round(enq, 5), "wall_ms_per_step": round(wall, 5),
                     "gpu_ms_per_step": round(gpu, 5)}
    g = res["graph"]["wall_ms_per_step"]
    N, L, H, d, c_m, c_z = cfg["N"], cfg["L"], 8, 32, 256, 128
    tok = N * L * H * d * 2
    nbytes = (2 * N * L * c_m + 4 * tok + 2 * 4 * H * d * c_m + 2 * N * L * c_m + 8 * N * L) + \
        (2 * L * L * c_z + 2 * H * L * L) + \
        (4 * tok + 2 * H * L * L + N * L + tok + 4 * N * H * L) + \
        (6 * tok + 4 * N * H * L + 2 * H * L * L + N * L + 4 * tok + 4 * H * L * L) + \
        (4 * tok + 3 * 2 * N * L * c_m + 8 * N * L + 2 * 4 * H * d * c_m + 4 * 4 * H * d * c_m)
    ach = nbytes / (res["graph"]["gpu_ms_per_step"] * 1e-3) / 1e9
    line = {
        "metric": "MSA row attention step (projections, pair bias, attention fwd+bwd) from the HIP graph cache, "
                  "steps/s on 1 MI355X",
        "value": round(1e3 / g, 1), "unit": "steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": g, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "n_rows": N, "seq_len": L, "n_heads": H, "head_dim": d, "c_m": c_m,
                   "c_z": c_z, "kernels_per_step": 17, "parallelism": "single-gpu"},
        "eager": res["eager"], "graph": res["graph"],
        "speedup_wall": round(res["eager"]["wall_ms_per_step"] / g, 3),
        "host_enqueue_reduction": round(res["eager"]["host_enqueue_ms_per_step"] /
                                        max(res["graph"]["host_enqueue_ms_per_step"], 1e-9), 1),
        "captures": cache.captures,
        "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "whole graphed step",
                     "avg_ms": res["graph"]["gpu_ms_per_step"], "algorithmic_bytes": int(nbytes)},
        "cpu_baseline": None,
    }
    print(json.dumps(line))


def proj_cpu_baseline(w, d, target_s: float):
    """The fp64 oracle (LayerNorm + one numpy matmul per projection) on the
    host, on a slice of rows sized for about target_s."""
    import oracle
    from paper_2404_11068_amd import workloads as W

    xf = W.as_float64(d["x"], "bf16")
    Wf = W.as_float64(d["weight"], "bf16")

    def run(rows):
        t0 = time.perf_counter()
        oracle.ln_proj_forward(xf[:rows], d["ln_weight"], d["ln_bias"], Wf, d["bias"], n_proj=w.n_proj, eps=w.eps)
        return time.perf_counter() - t0

    rows = min(w.n_rows, 4096)
    t = run(rows)
    rows = int(max(1, min(w.n_rows, rows * target_s / max(t, 1e-3))))
    reps = 1
    t = run(rows)
    if rows == w.n_rows and t < target_s:
        reps = max(1, int(target_s / max(t, 1e-3)))
        t = float(np.median([run(rows) for _ in range(reps)]))
    return {"value": round(w.flops() * rows / w.n_rows / t / 1e12, 6), "unit": "TFLOP/s",
            "cores": oracle.threads(), "kind": "oracle", "cpu_model": _cpu_model(),
            "seconds_per_run": round(t, 4), "runs": reps,
            "sample": "%d of %d rows, LayerNorm (C, OpenMP) + numpy fp64 matmuls" % (rows, w.n_rows)}


def ln_cpu_baseline(w, x, target_s: float):
    """The fp64 LayerNorm oracle (forward + backward) on the host cores, on
    the whole workload repeated (or a slice of rows) for about target_s."""
    import oracle
    from paper_2404_11068_amd import workloads as W

    xf = W.as_float64(x["x"], w.dtype)
    dyf = W.as_float64(x["dy"], w.dtype)
    wf, bf = x["weight"].astype(np.float64), x["bias"].astype(np.float64)

    def run(rows):
        t0 = time.perf_counter()
        oracle.layernorm_forward(xf[:rows], wf, bf, w.eps)
        oracle.layernorm_backward(xf[:rows], dyf[:rows], wf, w.eps)
        return time.perf_counter() - t0

    rows = w.n_rows
    t = run(rows)
    reps = max(1, int(target_s / max(t, 1e-3)))
    t = float(np.median([run(rows) for _ in range(reps)]))
    return {"value": round((w.bytes_fwd() + w.bytes_bwd()) / t / 1e9, 3), "unit": "GB/s",
            "cores": oracle.threads(), "kind": "oracle", "cpu_model": _cpu_model(),
            "seconds_per_run": round(t, 4), "runs": reps,
            "sample": "whole workload (%d x %d), forward + backward in fp64 (OpenMP rows), median of %d runs"
                      % (w.n_rows, w.n_cols, reps)}


def _pct(xs):
    """median and 10th/90th percentiles of per-call times in ms"""
    a = np.asarray(xs, dtype=np.float64)
    return {"median": round(float(np.median(a)), 5), "p10": round(float(np.percentile(a, 10)), 5),
            "p90": round(float(np.percentile(a, 90)), 5), "n": int(a.size)}


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
            if e.get("source_sha256") != kernel_source_hash(kernel_family(kernel)):
                return None
            return e.get("bytes_per_launch")
    return None


# device sources of each kernel family (a change to any of them invalidates
# the family's recorded counters)
KERNEL_SOURCES = {"attn": ("evo_frag.h", "evo_fwd.hip", "evo_bwd.hip", "evo_bwd_fused.hip"),
                  "ln": ("evo_frag.h", "evo_ln.hip"),
                  "proj": ("evo_frag.h", "evo_proj.hip"),
                  "proj_bwd": ("evo_frag.h", "evo_proj_bwd.hip"),
                  "pb": ("evo_frag.h", "evo_pair_bias.hip"),
                  "pb_bwd": ("evo_frag.h", "evo_pair_bias_bwd.hip"),
                  "optim": ("evo_frag.h", "evo_optim.hip")}


def kernel_family(kernel: str) -> str:
    if kernel.startswith("ln_proj"):
        return "proj"
    if kernel in ("dy_kernel", "dw_kernel", "colsum_kernel"):
        return "proj_bwd"
    if kernel in ("pair_bias_bwd_kernel", "pb_param_reduce_kernel"):
        return "pb_bwd"
    if kernel.startswith("pair_bias"):
        return "pb"
    if kernel in ("adam_swa_kernel", "sumsq_kernel", "clip_scale_kernel"):
        return "optim"
    return "ln" if kernel.startswith("ln_") else "attn"


def kernel_source_hash(family: str = "attn") -> str:
    """sha256 over the HIP sources that define one family's kernels."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2404_11068_amd", "csrc")
    for name in KERNEL_SOURCES[family]:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def rate_calibration(torch, steps: int):
    """Lane operations per second of v_exp_f32 and v_fma_f32 over the whole GPU
    (evo_probe_rate: 8 independent chains per lane, 2048 workgroups of 256
    threads), the unit rates behind the VALU bounds of the attention kernels."""
    from paper_2404_11068_amd import evo_attn as ea
    lib = ea.load_library()
    lib.evo_probe_rate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.evo_probe_rate.restype = ctypes.c_int
    blocks, iters = 2048, 4096
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {}
    for name, op in (("v_exp_f32", 0), ("v_fma_f32", 1)):
        for _ in range(2):  # warm-up
            assert lib.evo_probe_rate(op, blocks, iters, ctypes.c_void_p(sink.data_ptr()),
                                      ctypes.c_void_p(stream.cuda_stream)) == 0
        torch.cuda.synchronize()
        ts = []
        for _ in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            lib.evo_probe_rate(op, blocks, iters, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ms = float(np.median(ts))
        out[name] = {"tera_lane_ops_per_s": round(blocks * 256 * 8 * iters / (ms * 1e-3) / 1e12, 2), "ms": round(ms, 4)}
    assert bool(torch.isfinite(sink).all())
    print(json.dumps({"rate_calibration": out, "lane_ops_per_launch": blocks * 256 * 8 * iters,
                      "note": "8 independent chains per lane, one instruction per step; median of %d launches" % steps}))


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
        do = f(x["dout"][sl])
        t0 = time.perf_counter()
        oracle.forward(*args, g, b, m, rpb)
        t1 = time.perf_counter()
        oracle.backward(*args, do, g, b, m, rpb)
        t2 = time.perf_counter()
        split.append((t1 - t0, t2 - t1))
        return t2 - t0

    split = []
    rows = max(1, min(w.n_rows, 4))
    t = run(rows)
    # grow the sample to roughly target_s of CPU work (bounded by the workload)
    want = int(rows * target_s / max(t, 1e-3))
    want = max(1, min(w.n_rows, want))
    # a sample of at least one whole bias plane keeps whole planes
    if w.bias and want >= w.rows_per_bias:
        want = (want // w.rows_per_bias) * w.rows_per_bias
    # the same sample three times (more when one run is short, at most 25),
    # median taken; t_run estimates one run of the sample from the probe
    reps = 3
    t_run = t * want / rows
    if want == w.n_rows and 3 * t_run < target_s:  # the whole workload is short: repeat it
        reps = min(25, max(3, int(target_s / max(t_run, 1e-3))))
    elif t_run > target_s / 3:                    # keep three runs near the target
        want = max(1, int(want * target_s / (3 * t_run)))
        if w.bias and want >= w.rows_per_bias:
            want = (want // w.rows_per_bias) * w.rows_per_bias
    split.clear()
    times = [run(want) for _ in range(reps)]
    t = float(np.median(times))
    flops = (w.flops_fwd() + w.flops_bwd()) * want / w.n_rows
    tf = float(np.median([a for a, _ in split]))
    tb = float(np.median([b_ for _, b_ in split]))
    return {"value": round(flops / t / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "cpu_model": _cpu_model(), "seconds_per_run": round(t, 3), "runs": reps,
            "fwd_s_median": round(tf, 3), "bwd_s_median": round(tb, 3),
            "sample": "%d of %d rows of %s, forward + backward in fp64 (OpenMP), median of %d runs"
                      % (want, w.n_rows, w.name, reps)}


def _cpu_model() -> str:
    """The host CPU as /proc/cpuinfo names it, with its family / model /
    stepping numbers (some hosts report only a generic model name)."""
    info = {}
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ":" not in ln:
                    if info:
                        break  # first processor block only
                    continue
                key, val = (x.strip() for x in ln.split(":", 1))
                info.setdefault(key, val)
    except OSError:
        return "unknown"
    name = info.get("model name", "unknown")
    ids = ", ".join("%s %s" % (k, info[k]) for k in ("cpu family", "model", "stepping") if k in info)
    extra = [ids] if ids else []
    if "cpu MHz" in info:
        extra.append("%s MHz" % info["cpu MHz"])
    try:
        extra.append("%d logical CPUs on the host" % os.cpu_count())
    except TypeError:
        pass
    return "%s (%s)" % (name, "; ".join(extra)) if extra else name


if __name__ == "__main__":
    main()

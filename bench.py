#!/usr/bin/env python3
"""Throughput of 3D Deformable Slide Attention (forward + backward) on one MI355X.

One step = one pass of the whole operator over one batch of synthetic input: the forward
(coordinates, trilinear K gather, logits, softmax, V gather, output + LSE) and the backward
(recompute, dq, d_offsets, dK/dV scatter).  Inputs are generated on the host by the seeded
Philox generator, copied to HBM once, and are resident before timing starts.

Prints ONE JSON line:
  value          query tokens (all heads) per second over the timed steps, fwd + bwd
  roofline       the dominant kernel's algorithmic work per launch over its average HIP-event
                 duration, against the chip's peak for its bound
  cpu_baseline   the CPU oracle (plain C, fp64) timed on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "3D-DSA fwd+bwd queries/s and achieved HBM GB/s (% of peak) at 1 GPU"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
VALU_PEAK_TFLOPS = 157.3        # MI355X fp32 vector peak (2 FLOP/lane/clk: dot2 / dual issue)
DEFAULT_WORKLOAD = "fwdbwd_64x34x60"
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2607_22696_amd", "csrc")


def kernel_source_hash() -> str:
    """Hash of the HIP sources: counter figures taken from other sources are stale."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def kernel_family(name: str) -> str:
    """Which entry point a kernel of the library belongs to."""
    return "forward" if "fwd_kernel" in name else "backward"


def pmc_summary(workload, fetch_dir, write_dir, copyf_dir, copyw_dir, copy_mib):
    """Turn four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE of the bench command, and of
    a device copy of copy_mib MiB) into profiles/traffic_<workload>.json: HBM bytes per call of
    each entry point, each counter scaled by what it reads for the copy of known size."""
    import csv
    import re

    def per_kernel(d):
        path = [os.path.join(d, f) for f in os.listdir(d) if f.endswith("counter_collection.csv")][0]
        acc = {}
        for r in csv.DictReader(open(path)):
            m = re.search(r"(\w+_kernel)(<[^>]*>)?|(__amd_rocclr_copyBuffer)", r["Kernel_Name"])
            key = m.group(0) if m else r["Kernel_Name"][:60]
            acc.setdefault(key, []).append(float(r["Counter_Value"]) * 1024.0)  # KiB -> B
        return acc

    fetch, write = per_kernel(fetch_dir), per_kernel(write_dir)
    true_bytes = copy_mib * (1 << 20)
    cf = per_kernel(copyf_dir)["__amd_rocclr_copyBuffer"]
    cw = per_kernel(copyw_dir)["__amd_rocclr_copyBuffer"]
    fetch_scale = (sum(cf) / len(cf)) / true_bytes   # counter bytes per byte actually read
    write_scale = (sum(cw) / len(cw)) / true_bytes
    out = {"workload": workload, "kernel_source_hash": kernel_source_hash(),
           "fetch_scale": round(fetch_scale, 4), "write_scale": round(write_scale, 4),
           "kernels": {}, "per_call_bytes": {"forward": 0.0, "backward": 0.0}}
    for k in fetch:
        if k not in write or k == "__amd_rocclr_copyBuffer":
            continue
        f = sum(fetch[k]) / len(fetch[k]) / fetch_scale
        w = sum(write[k]) / len(write[k]) / write_scale
        out["kernels"][k] = {"fetch_bytes": round(f), "write_bytes": round(w)}
        out["per_call_bytes"][kernel_family(k)] += f + w
    os.makedirs(PROFILES, exist_ok=True)
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(path)


def measured_traffic(workload, kernel_name):
    """HBM bytes per call from profiles/traffic_<workload>.json, or None if absent or stale."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    return d["per_call_bytes"].get(kernel_name)


def algorithmic(w):
    """Per-launch algorithmic HBM bytes and FLOPs of the forward and backward kernels.

    Per query row (token, head), with s = bytes per q/k/v element:
      forward  bytes  q, k, v read + out written (4 D s) + offsets (12 P) + lse (4)
               flops  16 P D multiply-adds (8 corners x D for q.K, 8 x D for V) = 32 P D
      backward bytes  q, k, v, dout read (4 D s) + offsets (12 P) + lse (4)
                      + dq, dk, dv written (3 D 4) + d_offsets (12 P)
               flops  40 P D multiply-adds (q.K, dout.V, dq, dK scatter, dV scatter) = 80 P D
    """
    s = 2 if w.dtype == "bf16" else 4
    rows = w.queries
    P, D = w.P, w.head_dim
    return {
        "fwd_bytes": rows * (4 * D * s + 12 * P + 4),
        "fwd_flops": rows * 32 * P * D,
        "bwd_bytes": rows * (4 * D * s + 12 * P + 4 + 3 * D * 4 + 12 * P),
        "bwd_flops": rows * 80 * P * D,
    }


def cpu_baseline(w, host, budget_s, backward=True):
    """The oracle (forward rows, plus the backward slab with its dK/dV scatter when the step
    has a backward) on head 0, one frame at a time, until about budget_s seconds of CPU work;
    reported in query tokens per second."""
    import numpy as np

    import oracle
    q, k, v, off, dout = host
    shape = (w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw)
    HW = w.H * w.W
    dk = np.zeros((w.T, w.H, w.W, w.head_dim)) if backward else None
    dv = np.zeros_like(dk) if backward else None
    rows_done = 0
    frames = 0
    t0 = time.perf_counter()
    while frames < w.T and time.perf_counter() - t0 < budget_s:
        rows = (np.arange(HW, dtype=np.int64) + frames * HW) * w.heads  # head 0 of each token
        oracle.forward(shape, w.dtype, q, k, v, off, rows=rows)
        if backward:
            oracle.backward_slab(shape, w.dtype, q, k, v, off, dout, 0, 0, frames, frames + 1,
                                 dk=dk, dv=dv)
        rows_done += HW
        frames += 1
    dt = time.perf_counter() - t0
    # one query token carries all heads: rows / heads tokens
    return {"value": rows_done / w.heads / dt, "unit": "queries/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": f"head 0 of frames [0,{frames}) of {w.name}: {rows_done} (token, head) rows, "
                      + ("forward + backward incl. dK/dV scatter" if backward else "forward")
                      + f", fp64, {dt:.1f} s; "
                      f"scaled to query tokens (all {w.heads} heads)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--forward-only", action="store_true",
                    help="time the forward alone (workloads without a backward pass)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of CPU-oracle work for cpu_baseline (0 = skip)")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH", "WRITE", "COPYF", "COPYW"),
                    help="summarise four rocprofv3 --pmc output folders into "
                         "profiles/traffic_<workload>.json (no GPU needed)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 3 device-to-device copies of MIB MiB and exit (calibrates the "
                         "FETCH_SIZE / WRITE_SIZE counters against a known byte count)")
    args = ap.parse_args()

    if args.pmc_summary:
        pmc_summary(args.workload, *args.pmc_summary, copy_mib=args.copy_probe or 1024)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the operator's "
              "multi-GPU sharding is a design note, not part of this build", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_22696_amd as dsa
    import testgen
    from tests.util import to_device

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_probe:
        n = args.copy_probe * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        t = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t[0].record()
        for _ in range(3):
            dst.copy_(src)
        t[1].record()
        torch.cuda.synchronize()
        ms = t[0].elapsed_time(t[1]) / 3
        print(json.dumps({"copy_mib": args.copy_probe, "ms": round(ms, 4),
                          "gbs_read_plus_write": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}))
        return
    dsa.load()
    w = testgen.WORKLOADS[args.workload]
    do_bwd = w.backward and not args.forward_only
    t_gen = time.perf_counter()
    host = testgen.gen_inputs(w)
    if host[4] is None and do_bwd:
        host = host[:4] + (testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True),)
    q, k, v, off, dout = host
    bf = w.dtype == "bf16"
    qd, kd, vd = (to_device(a, bf) for a in (q, k, v))
    od = to_device(off, False)
    gd = to_device(dout, bf) if do_bwd else None
    t_gen = time.perf_counter() - t_gen
    kern = (w.kt, w.kh, w.kw)
    out, lse = dsa.forward(qd, kd, vd, od, kernel=kern)
    grads = None
    if do_bwd:
        f32 = dict(dtype=torch.float32, device=qd.device)
        grads = (torch.empty(q.shape, **f32), torch.empty(q.shape, **f32),
                 torch.empty(q.shape, **f32), torch.empty(off.shape, **f32))

    def step():
        dsa.forward(qd, kd, vd, od, kernel=kern, out=out, lse=lse)
        if do_bwd:
            dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern, grads=grads)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s in range(K):
        ev[s][0].record()
        dsa.forward(qd, kd, vd, od, kernel=kern, out=out, lse=lse)
        ev[s][1].record()
        if do_bwd:
            dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern, grads=grads)
        ev[s][2].record()
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    fwd_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / K
    bwd_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / K if do_bwd else 0.0
    ms_step = total_ms / K

    alg = algorithmic(w)
    step_bytes = alg["fwd_bytes"] + (alg["bwd_bytes"] if do_bwd else 0)
    tokens = w.B * w.N
    # dominant kernel: the longer of the two launches
    kname, kms = ("backward", bwd_ms) if do_bwd and bwd_ms >= fwd_ms else ("forward", fwd_ms)
    kbytes = alg["bwd_bytes"] if kname == "backward" else alg["fwd_bytes"]
    kflops = alg["bwd_flops"] if kname == "backward" else alg["fwd_flops"]
    t_hbm = kbytes / (HBM_PEAK_GBS * 1e9)
    t_alu = kflops / (VALU_PEAK_TFLOPS * 1e12)
    if t_alu >= t_hbm:
        ach = kflops / (kms * 1e-3) / 1e12
        roof = {"bound": "alu", "achieved": round(ach, 3), "peak": VALU_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / VALU_PEAK_TFLOPS, 4), "traffic": None}
    else:
        ach = kbytes / (kms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None}
    tr = measured_traffic(w.name, kname)
    roof["traffic"] = None if tr is None else round(tr)
    roof["kernel"] = f"dsa3d_{kname}"
    roof["avg_launch_ms"] = round(kms, 4)

    res = {
        "metric": METRIC,
        "value": round(tokens / (ms_step * 1e-3), 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded Philox inputs shaped like the paper's video-latent grids)",
        "config": {"workload": w.name, "grid_TxHxW": [w.T, w.H, w.W], "batch": w.B,
                   "heads": w.heads, "head_dim": w.head_dim, "kernel": [w.kt, w.kh, w.kw],
                   "points": w.P, "backward": do_bwd, "parallelism": "single GPU"},
        "fwd_ms": round(fwd_ms, 4),
        "bwd_ms": round(bwd_ms, 4),
        "hbm_gbs_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "token_head_rows_per_s": round(w.queries / (ms_step * 1e-3), 1),
        "roofline": roof,
        "input_gen_s": round(t_gen, 1),
    }
    if args.cpu_budget > 0:
        res["cpu_baseline"] = cpu_baseline(w, host, args.cpu_budget, backward=do_bwd)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

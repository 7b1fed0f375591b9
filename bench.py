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
DEFAULT_WORKLOAD = "wide_64x68x120_p75"
DEFAULT_CONV_WORKLOAD = "dwconv_1080p_256f"
DEFAULT_PW_WORKLOAD = "pw_64x34x60"
PW_METRIC = "3D-DSA predicted-weights fwd+bwd queries/s and achieved HBM GB/s (% of peak) at 1 GPU"
CONV_METRIC = "DWConv3D fwd+bwd tokens/s and achieved HBM GB/s (% of peak) at 1 GPU"
WIN_METRIC = "Swin-DiT shifted-window attention fwd+bwd queries/s and MFMA TFLOP/s (% of peak) at 1 GPU"
DEFAULT_WIN_WORKLOAD = "swin_1080p_256f"
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2607_22696_amd", "csrc")


# Device sources of each kernel family: counter figures taken from other sources are stale.
FAMILY_SOURCES = {
    "dsa": ["dsa3d_device.h", "tile_order.h", "dsa3d_forward.hip", "dsa3d_backward.hip"],
    "dwconv": ["dsa3d_device.h", "dwconv3d.hip"],
    "win": ["winattn.hip"],
}


def kernel_source_hash(family: str = "dsa") -> str:
    """Hash of the device sources of one kernel family, comments and layout left out (a
    change of a comment does not make counters taken on the same code stale)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in FAMILY_SOURCES[family]:
        with open(os.path.join(CSRC, name), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        text = " ".join(text.split())
        h.update(name.encode() + b"\0" + text.encode())
    return h.hexdigest()[:16]


def workload_family(workload: str) -> str:
    if workload.startswith("dwconv"):
        return "dwconv"
    return "win" if workload.startswith("swin") else "dsa"


def kernel_base(name: str) -> str:
    """Kernel function name without namespace, template arguments or parameters; the bf16
    dK/dV gather (bwd_gather_mfma_kernel) under the name of the backward phase it runs,
    bwd_gather_kernel."""
    import re
    m = re.search(r"(\w+_kernel)\b|(__amd_rocclr_copyBuffer)", name)
    base = m.group(0) if m else name[:60]
    return "bwd_gather_kernel" if base == "bwd_gather_mfma_kernel" else base


# Counters of the two rocprofv3 --pmc passes that give a kernel's traffic past the L2s
# (each pass within the 4 TCC counters one run can hold):
READ_COUNTERS = ("TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum",
                 "TCC_EA0_RDREQ_sum")
WRITE_COUNTERS = ("WRITE_SIZE", "TCC_ATOMIC_sum", "TCC_EA0_ATOMIC_sum")


def pmc_summary(workload, read_dir, write_dir, copyr_dir, copyw_dir, copy_mib):
    """Turn four rocprofv3 --pmc runs (READ_COUNTERS and WRITE_COUNTERS of the bench command,
    and of a device copy of copy_mib MiB) into profiles/traffic_<workload>.json: per launch of
    each kernel, the bytes read past the L2s (read requests to the memory side times their
    size: 32, 64 or 128 bytes), the bytes written (WRITE_SIZE), and the atomic requests at the
    L2s (TCC_ATOMIC) and past them (TCC_EA0_ATOMIC).  The copy checks the accounting: its read
    and write bytes per byte copied are stored beside the kernels' figures.  (The derived
    FETCH_SIZE counter counts 64 bytes per 128-byte read request on this GPU, half the bytes,
    which is why the request counters are read directly.)"""
    import csv

    def per_kernel(d):
        path = [os.path.join(d, f) for f in os.listdir(d) if f.endswith("counter_collection.csv")][0]
        acc = {}
        for r in csv.DictReader(open(path)):
            key = (kernel_base(r["Kernel_Name"]), r["Dispatch_Id"])
            acc.setdefault(key, {})[r["Counter_Name"]] = float(r["Counter_Value"])
        out = {}
        for (k, _), c in acc.items():
            out.setdefault(k, []).append(c)
        return out

    def read_bytes(c):
        return (32 * c["TCC_EA0_RDREQ_32B_sum"] + 64 * c["TCC_EA0_RDREQ_64B_sum"]
                + 128 * c["TCC_EA0_RDREQ_128B_sum"])

    def mean(xs):
        return sum(xs) / len(xs)

    reads, writes = per_kernel(read_dir), per_kernel(write_dir)
    true_bytes = copy_mib * (1 << 20)
    cr = per_kernel(copyr_dir)["__amd_rocclr_copyBuffer"]
    cw = per_kernel(copyw_dir)["__amd_rocclr_copyBuffer"]
    out = {"workload": workload, "kernel_source_hash": kernel_source_hash(workload_family(workload)),
           "counted_at": "past the L2s: read requests x size (TCC_EA0_RDREQ_32B/64B/128B), "
                         "WRITE_SIZE; memory-side-cache hits count too",
           "copy_check": {"mib": copy_mib,
                          "read_bytes_per_byte": round(mean([read_bytes(c) for c in cr]) / true_bytes, 4),
                          "write_bytes_per_byte": round(mean([c["WRITE_SIZE"] * 1024.0 for c in cw])
                                                        / true_bytes, 4)},
           "kernels": {}}
    for k in reads:
        # the operator's kernels only (not the copy, torch's own kernels or the gather
        # microbenchmark)
        if k not in writes or not k.endswith("_kernel") or "elementwise" in k:
            continue
        rd = mean([read_bytes(c) for c in reads[k]])
        req = mean([c["TCC_EA0_RDREQ_sum"] for c in reads[k]])
        sized = mean([c["TCC_EA0_RDREQ_32B_sum"] + c["TCC_EA0_RDREQ_64B_sum"]
                      + c["TCC_EA0_RDREQ_128B_sum"] for c in reads[k]])
        wr = mean([c["WRITE_SIZE"] * 1024.0 for c in writes[k]])
        out["kernels"][k] = {"fetch_bytes": round(rd), "write_bytes": round(wr),
                             "hbm_bytes": round(rd + wr),
                             "read_requests_of_known_size": round(sized / max(req, 1.0), 4),
                             "atomics_l2": round(mean([c["TCC_ATOMIC_sum"] for c in writes[k]])),
                             "atomics_past_l2": round(mean([c["TCC_EA0_ATOMIC_sum"]
                                                            for c in writes[k]]))}
    os.makedirs(PROFILES, exist_ok=True)
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(path)


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from profiles/traffic_<workload>.json, or None if
    absent or taken from other kernel sources."""
    path = os.path.join(PROFILES, f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        d = json.load(fh)
    if d.get("kernel_source_hash") != kernel_source_hash(workload_family(workload)):
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k["hbm_bytes"]


# kernels of one backward call of the main operator, in launch order (the bin scan is three
# small kernels after the fill of the counts)
BWD_KERNELS = ("fill_u32_kernel", "bwd_vpass_kernel", "scan_reduce_kernel", "scan_sums_kernel",
               "scan_apply_kernel", "bwd_kpass_kernel", "bwd_gather_kernel")
# the backward's four timed phases (dsa3d_backward_timed), main operator and predicted weights
BWD_PHASES = ("bwd_vpass_kernel", "bin_scan", "bwd_kpass_kernel", "bwd_gather_kernel")
PW_BWD_PHASES = ("bwd_sweep_kernel", "bin_scan", "bwd_finalize_kernel", "bwd_gather_kernel")


def measured_step_traffic(workload, backward):
    """HBM bytes of one step (forward, and the backward's kernels if `backward`) summed from
    profiles/traffic_<workload>.json, or None if the file is absent, was taken from other
    kernel sources, or lacks one of the step's kernels."""
    names = ("fwd_kernel",) + (BWD_KERNELS if backward else ())
    total = 0
    for n in names:
        b = measured_traffic(workload, n)
        if b is None:
            return None
        total += b
    return total


def hbm_rocprof(workload, backward, ms_step, alg_bytes):
    """The step's traffic past the L2s as rocprofv3 counted it (read requests x size plus
    WRITE_SIZE, profiles/traffic_<workload>.json) over the step time measured in this run:
    GB/s, fraction of the 8 TB/s HBM peak, and the ratio to the step's algorithmic bytes (what
    the counters see beyond the compulsory traffic: re-reads of corner rows that missed L2,
    workspace, atomics).  Rows served by the memory-side cache count too, so this is an upper
    bound on DRAM traffic.  None where no counters for the current kernel sources are
    committed."""
    b = measured_step_traffic(workload, backward)
    if b is None:
        return None
    gbs = b / (ms_step * 1e-3) / 1e9
    return {"counted_at": "L2 egress", "bytes_per_step": b, "GBps": round(gbs, 1),
            "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
            "ratio_to_algorithmic": round(b / alg_bytes, 2)}


def copy_ceiling(torch, mib=2048):
    """A device-to-device copy of `mib` MiB on the bench's device: read + write GB/s, the
    practical ceiling of HBM traffic on this machine."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t[0].record()
    for _ in range(5):
        dst.copy_(src)
    t[1].record()
    torch.cuda.synchronize()
    ms = t[0].elapsed_time(t[1]) / 5
    gbs = 2 * n * 4 / (ms * 1e-3) / 1e9
    del src, dst
    return {"what": f"device-to-device copy of {mib} MiB, read + write bytes",
            "GBps": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}


def host_info():
    """CPU model, logical CPUs and RAM of the machine the oracle runs on."""
    model, ram = "unknown", None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                ram = round(int(line.split()[1]) / (1 << 20), 1)
                break
    except OSError:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "ram_GiB": ram}


def algorithmic(w):
    """Algorithmic HBM bytes and FLOPs per launch of each kernel, and of the two entry points.

    Per query row (token, head), with s = bytes per q/k/v element, P points, head_dim D:
      fwd_kernel           bytes  q, k, v read + out written (4 D s), offsets (12 P), lse (4)
                           flops  16 P D multiply-adds: 8 corners x D for q.K, 8 x D for V
      bwd_vpass_kernel     bytes  v, dout read (2 D s), offsets (12 P)
                           flops  8 P D multiply-adds: dout.V_c at 8 corners
      bwd_kpass_kernel     bytes  q, k read (2 D s), offsets (12 P), lse (4), dq and
                                  d_offsets written (4 D + 12 P)
                           flops  16 P D multiply-adds: q.K_c at 8 corners and the 8-corner
                                  K interpolation that dq needs
      bwd_gather_kernel    bytes  q, dout read (2 D s), dk, dv written (8 D)
                           flops  16 P D multiply-adds: w_c ds_p q into dK and w_c alpha_p dout
                                  into dV at 8 corners
      backward (entry)     bytes  q, k, v, dout (4 D s), offsets (12 P), lse (4) read once;
                                  dq, dk, dv (12 D) and d_offsets (12 P) written once
                           flops  40 P D multiply-adds
    A multiply-add is 2 FLOPs.  The bin scan moves 4-byte counters only (no algorithmic work).
    """
    s = 2 if w.dtype == "bf16" else 4
    rows = w.queries
    P, D = w.P, w.head_dim
    per = {
        "fwd_kernel": (4 * D * s + 12 * P + 4, 32 * P * D),
        "bwd_vpass_kernel": (2 * D * s + 12 * P, 16 * P * D),
        "bwd_kpass_kernel": (2 * D * s + 12 * P + 4 + 4 * D + 12 * P, 32 * P * D),
        "bwd_gather_kernel": (2 * D * s + 8 * D, 32 * P * D),
        "forward": (4 * D * s + 12 * P + 4, 32 * P * D),
        "backward": (4 * D * s + 12 * P + 4 + 3 * D * 4 + 12 * P, 80 * P * D),
    }
    return {k: {"bytes": rows * b, "flops": rows * f} for k, (b, f) in per.items()}


def vmem_bytes(w):
    """Bytes that the vector-memory instructions (loads and stores through each compute
    unit's L1 path) of the query-owned kernels move per launch, per query row (s = bytes per
    q/k/v element):
      fwd_kernel        16 P D s (8 K and 8 V corner rows per point) + D s (q) + 12 P
                        (offsets) + D s (out) + 4 (lse)
      bwd_vpass_kernel  8 P D s (V corner rows) + D s (dout) + 12 P (offsets) + 16 P (the V
                        half of each point record) + 4 P (bin-count atomics)
      bwd_kpass_kernel  8 P D s (K corner rows) + D s (q) + 24 P (offsets, twice) + 4 (lse)
                        + 4 P (da_p) + 16 P (the V half of each record, read to finish the
                        points) + 32 P (the K half, written and read back, only for rows of
                        more than 5 chunks of L = D s / 16 points, whose K halves the kernel
                        cannot hold in registers) + 4 D (dq) + 12 P (d_offsets) + 8 P (ranks
                        and bin starts) + 24 P (bin entries)
    These, not the HBM bytes, are what bounds the kernels: the corner rows come from L2 and
    L1, and the per-unit gather path is busy most of the time (rocprofv3 TA/TD counters)."""
    s = 2 if w.dtype == "bf16" else 4
    P, D = w.P, w.head_dim
    lanes = D * s // 16
    kept = 32 * P if -(-P // lanes) > 5 else 0
    per = {
        "fwd_kernel": 16 * P * D * s + 2 * D * s + 12 * P + 4,
        "bwd_vpass_kernel": 8 * P * D * s + D * s + 12 * P + 16 * P + 4 * P,
        "bwd_kpass_kernel": 8 * P * D * s + D * s + 24 * P + 4 + 4 * P + 16 * P + kept + 4 * D
                            + 12 * P + 8 * P + 24 * P,
    }
    return {k: w.queries * b for k, b in per.items()}


PROBE_SRC = os.path.join(ROOT, "gather_probe.hip")
PROBE_LIB = os.path.join(ROOT, "libgather_probe.so")


def build_probe(verbose=False):
    """Compile the gather microbenchmark (gather_probe.hip, measurement only) beside this
    script."""
    from paper_2607_22696_amd import build as pkg_build
    pkg_build.compile_shared([PROBE_SRC], PROBE_LIB, verbose)
    return PROBE_LIB


def gather_ceiling(row_bytes):
    """The gather microbenchmark (libgather_probe.so): 16-byte lane loads, one contiguous row
    of row_bytes per lane group at pseudo-random addresses, every row already in L1 (the
    ceiling of the kernels' gather path), every row missing L1 and hitting L2, the same
    pattern from LDS, rows from a 512 MB region (missing L2: what comes from past the L2s),
    and the L1- and L2-resident rows through direct-to-LDS loads."""
    import ctypes
    if not os.path.exists(PROBE_LIB):
        raise RuntimeError(f"{PROBE_LIB} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(PROBE_LIB)
    lib.dsa3d_probe_gather.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_float),
                                       ctypes.POINTER(ctypes.c_double)]
    out = {"row_bytes": row_bytes}
    for src, name in ((0, "l1"), (2, "l2"), (1, "lds"), (3, "mem"), (4, "l1_to_lds"),
                      (5, "l2_to_lds")):
        ms, nb = ctypes.c_float(), ctypes.c_double()
        rc = lib.dsa3d_probe_gather(src, row_bytes, 2048, 4096, ctypes.byref(ms), ctypes.byref(nb))
        if rc != 0:
            raise RuntimeError(f"gather probe failed ({rc})")
        out[f"{name}_TBps"] = round(nb.value / (ms.value * 1e-3) / 1e12, 2)
    return out


def working_set_curve(sets_mib=(1, 2, 3, 4, 6, 8, 16, 32, 64, 128, 256, 512)):
    """Random gathers of whole rows (256 B, and 128 B) from working sets of growing size, the
    rows contiguous and 6 KB apart (one head of a 24-head x 256 B tensor): the rate as the
    working set outgrows an XCD's 4 MB L2 and the 256 MB memory-side cache.  One JSON line per
    point."""
    import ctypes
    lib = ctypes.CDLL(PROBE_LIB)
    fn = lib.dsa3d_probe_working_set
    fn.argtypes = [ctypes.c_int, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_int, ctypes.c_int,
                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]
    for rb in (256, 128):
        for stride in (rb, 6144):
            for mib in sets_mib:
                ms, nb = ctypes.c_float(), ctypes.c_double()
                set_bytes = mib << 20
                if set_bytes // rb * stride > (4 << 30):
                    continue
                rc = fn(rb, stride, set_bytes, 8192, 256, ctypes.byref(ms), ctypes.byref(nb))
                if rc != 0:
                    raise RuntimeError(f"working-set probe failed ({rc})")
                print(json.dumps({"row_bytes": rb, "stride_bytes": stride, "set_MiB": mib,
                                  "ms": round(ms.value, 4),
                                  "TBps": round(nb.value / (ms.value * 1e-3) / 1e12, 2)}),
                      flush=True)


def roofline(work, ms, peak=VALU_PEAK_TFLOPS, bound="alu"):
    """Roofline entry of one kernel: bound by whichever of HBM bytes and its flops takes
    longer at peak (fp32 vector peak; the dense bf16 matrix peak for a kernel whose
    multiply-adds run on the matrix cores); achieved = algorithmic work per launch / average
    launch time."""
    t_hbm = work["bytes"] / (HBM_PEAK_GBS * 1e9)
    t_alu = work["flops"] / (peak * 1e12)
    if t_alu >= t_hbm:
        ach = work["flops"] / (ms * 1e-3) / 1e12
        return {"bound": bound, "achieved": round(ach, 3), "peak": peak,
                "unit": "TFLOP/s", "frac": round(ach / peak, 4)}
    ach = work["bytes"] / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4)}


def kernel_roofline(w, alg, name, ms):
    """The bf16 dK/dV gather takes its multiply-adds on the matrix cores; the other kernels
    on the vector ALUs."""
    if name == "bwd_gather_kernel" and w.dtype == "bf16":
        return roofline(alg[name], ms, MFMA_BF16_PEAK_TFLOPS, "mfma")
    return roofline(alg[name], ms)


def cpu_baseline(w, host, budget_s, backward=True):
    """The oracle (forward rows, plus the backward slab with its dK/dV scatter when the step
    has a backward) one (head, frame) at a time, head 0 first, until about budget_s seconds
    of CPU work; reported in query tokens per second."""
    import numpy as np

    import oracle
    q, k, v, off, dout = host
    shape = (w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw)
    HW = w.H * w.W
    rows_done = 0
    done = []  # (head, frames) per head touched
    t0 = time.perf_counter()
    for m in range(w.heads):
        if time.perf_counter() - t0 >= budget_s:
            break
        dk = np.zeros((w.T, w.H, w.W, w.head_dim)) if backward else None
        dv = np.zeros_like(dk) if backward else None
        frames = 0
        while frames < w.T and time.perf_counter() - t0 < budget_s:
            rows = (np.arange(HW, dtype=np.int64) + frames * HW) * w.heads + m
            oracle.forward(shape, w.dtype, q, k, v, off, rows=rows)
            if backward:
                oracle.backward_slab(shape, w.dtype, q, k, v, off, dout, 0, m, frames,
                                     frames + 1, dk=dk, dv=dv)
            rows_done += HW
            frames += 1
        done.append((m, frames))
    dt = time.perf_counter() - t0
    what = ", ".join(f"head {m} frames [0,{f})" for m, f in done)
    # one query token carries all heads: rows / heads tokens
    return {"value": rows_done / w.heads / dt, "unit": "queries/s", "cores": oracle.threads(),
            "kind": "oracle", **host_info(),
            "sample": f"{what} of {w.name}: {rows_done} (token, head) rows, "
                      + ("forward + backward incl. dK/dV scatter" if backward else "forward")
                      + f", fp64, {dt:.1f} s; "
                      f"scaled to query tokens (all {w.heads} heads)"}


def conv_algorithmic(w):
    """Algorithmic HBM bytes and FLOPs per launch of the depthwise-conv kernels, per element
    (token, channel), s = bytes per x / y / dy element, taps = kt kh kw:
      dwconv_kernel (forward)   x read, y written: 2 s;         2 taps FLOPs
      dwconv_kernel (dx)        dy read, dx (fp32) written: s + 4; 2 taps FLOPs
      dwconv_wgrad_kernel       x and dy read: 2 s;              2 taps FLOPs
    (the filter, the bias and the per-slice partial sums are a few MB)."""
    s = 2 if w.dtype == "bf16" else 4
    n = w.tokens * w.C
    f = 2 * w.taps * n
    return {"dwconv_forward": {"bytes": n * 2 * s, "flops": f},
            "dwconv_dx": {"bytes": n * (s + 4), "flops": f},
            "dwconv_wgrad": {"bytes": n * 2 * s, "flops": f}}


def conv_cpu_baseline(w, host, budget_s):
    """The conv oracle (forward and dx of one frame at a time, fp64) for about budget_s
    seconds; tokens per second."""
    import oracle
    x, dy, wt, bias = host
    frames = 0
    t0 = time.perf_counter()
    while frames < w.T and time.perf_counter() - t0 < budget_s:
        oracle.dwconv_forward(w.shape8(), w.dtype, x, wt, bias, frames=(frames, frames + 1))
        oracle.dwconv_backward(w.shape8(), w.dtype, x, wt, dy, frames=(frames, frames + 1),
                               weight_grads=False)
        frames += 1
    dt = time.perf_counter() - t0
    toks = frames * w.H * w.W * w.B
    return {"value": toks / dt, "unit": "tokens/s", "cores": oracle.threads(), "kind": "oracle",
            **host_info(),
            "sample": f"frames [0,{frames}) of {w.name}: {toks} tokens x {w.C} channels, forward "
                      f"+ dx (no weight gradient), fp64, {dt:.1f} s"}


def bench_dwconv(args, torch, dsa, testgen, to_device):
    """One step = forward, dx, and the weight and bias gradients of the depthwise conv."""
    w = testgen.CONV_WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    host = testgen.gen_conv_inputs(w, progress=lambda m: print(m, file=sys.stderr, flush=True))
    x, dy, wt, bias = host
    bf = w.dtype == "bf16"
    xd, dyd = to_device(x, bf), to_device(dy, bf)
    wd, bd = to_device(wt, False), to_device(bias, False)
    t_gen = time.perf_counter() - t_gen
    y = torch.empty_like(xd)
    dx = torch.empty(xd.shape, dtype=torch.float32, device=xd.device)
    desc = dsa.make_conv_desc(w.B, w.T, w.H, w.W, w.C, w.kt, w.kh, w.kw, w.dtype)
    ws = torch.empty(dsa.dsa3d_dwconv3d_backward_workspace_size(desc), dtype=torch.uint8,
                     device=xd.device)
    dwt = torch.empty(wt.shape, dtype=torch.float32, device=xd.device)
    dbt = torch.empty(bias.shape, dtype=torch.float32, device=xd.device)
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]

    def step(s=None):
        if s is not None:
            ev[s][0].record()
        dsa.dwconv3d_forward(xd, wd, bd, out=y)
        if s is not None:
            ev[s][1].record()
        dsa.dwconv3d_backward(xd, wd, dyd, need_dweight=False, need_dbias=False, dx=dx)
        if s is not None:
            ev[s][2].record()
        dsa.dsa3d_dwconv3d_backward(desc, xd, wd, dyd, None, dwt, dbt, ws, ws.numel())
        if s is not None:
            ev[s][3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(K):
        step(s)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / K
    kernel_ms = {n: sum(e[i].elapsed_time(e[i + 1]) for e in ev) / K
                 for i, n in enumerate(["dwconv_forward", "dwconv_dx", "dwconv_wgrad"])}
    alg = conv_algorithmic(w)
    kname = max(kernel_ms, key=lambda n: kernel_ms[n])
    roof = roofline(alg[kname], kernel_ms[kname])
    roof["traffic"] = None
    roof["kernel"] = kname
    roof["avg_launch_ms"] = round(kernel_ms[kname], 4)
    step_bytes = sum(a["bytes"] for a in alg.values())
    res = {
        "metric": CONV_METRIC, "value": round(w.tokens / (ms_step * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded Philox inputs shaped like the paper's video-latent grids)",
        "config": {"workload": w.name, "grid_TxHxW": [w.T, w.H, w.W], "batch": w.B,
                   "channels": w.C, "kernel": [w.kt, w.kh, w.kw], "parallelism": "single GPU"},
        "kernel_ms": {n: round(t, 4) for n, t in kernel_ms.items()},
        "kernel_roofline": {n: roofline(alg[n], t) for n, t in kernel_ms.items()},
        "hbm_gbs_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "roofline": roof, "input_gen_s": round(t_gen, 1),
    }
    if args.cpu_budget > 0:
        res["cpu_baseline"] = conv_cpu_baseline(w, host, args.cpu_budget)
    print(json.dumps(res), flush=True)


def pw_algorithmic(w):
    """Per-launch algorithmic HBM bytes and FLOPs of the predicted-weights kernels, per query row
    (s = bytes per V element, P points, head_dim D):
      fwd_kernel           logits (4 P), offsets (12 P), V read and out written (2 D s), lse (4);
                           8 P D multiply-adds (V at 8 corners)
      bwd_sweep_kernel     logits, offsets, lse, V and dout read (2 D s + 16 P + 4);
                           8 P D multiply-adds (dout.V at 8 corners)
      bwd_finalize_kernel  offsets read, d_offsets and dlogits written (28 P)
      bwd_gather_kernel    dout read, dV written (D s + 4 D); 8 P D multiply-adds
    """
    s = 2 if w.dtype == "bf16" else 4
    rows, P, D = w.queries, w.P, w.head_dim
    per = {
        "fwd_kernel": (2 * D * s + 16 * P + 4, 16 * P * D),
        "bwd_sweep_kernel": (2 * D * s + 16 * P + 4, 16 * P * D),
        "bwd_finalize_kernel": (28 * P, 0),
        "bwd_gather_kernel": (D * s + 4 * D, 16 * P * D),
        "forward": (2 * D * s + 16 * P + 4, 16 * P * D),
        "backward": (2 * D * s + 16 * P + 4 + 4 * D + 16 * P, 32 * P * D),
    }
    return {k: {"bytes": rows * b, "flops": rows * f} for k, (b, f) in per.items()}


def bench_pw(args, torch, dsa, testgen, to_device):
    """One step = forward and backward of the predicted-weights variant."""
    w = testgen.PW_WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    logits, v, off, dout = testgen.gen_pw_inputs(
        w, progress=lambda m: print(m, file=sys.stderr, flush=True))
    bf = w.dtype == "bf16"
    ld_, vd, od, gd = (to_device(logits, False), to_device(v, bf), to_device(off, False),
                       to_device(dout, bf))
    t_gen = time.perf_counter() - t_gen
    kern = (w.kt, w.kh, w.kw)
    out, lse = dsa.pw_forward(ld_, vd, od, kernel=kern)
    f32 = dict(dtype=torch.float32, device=vd.device)
    grads = (torch.empty(logits.shape, **f32), torch.empty(v.shape, **f32),
             torch.empty(off.shape, **f32))
    need = dsa.dsa3d_pw_backward_workspace_size(dsa.make_desc(
        w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw, w.dtype))
    workspace = torch.empty(need, dtype=torch.uint8, device=vd.device)

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    K = args.steps
    ev = [new_events(2) for _ in range(K)]
    ph = [new_events(dsa.DSA3D_BACKWARD_PHASES + 1) for _ in range(K)]

    def step(s=None):
        if s is not None:
            ev[s][0].record()
        dsa.pw_forward(ld_, vd, od, kernel=kern, out=out, lse=lse)
        if s is not None:
            ev[s][1].record()
        dsa.pw_backward(ld_, vd, od, lse, gd, kernel=kern, grads=grads, workspace=workspace,
                        phase_events=None if s is None else ph[s])

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(K):
        step(s)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / K
    kernel_ms = {"fwd_kernel": sum(e[0].elapsed_time(e[1]) for e in ev) / K}
    for i, n in enumerate(PW_BWD_PHASES):
        kernel_ms[n] = sum(p[i].elapsed_time(p[i + 1]) for p in ph) / K
    alg = pw_algorithmic(w)
    kname = max((n for n in kernel_ms if n in alg), key=lambda n: kernel_ms[n])
    roof = kernel_roofline(w, alg, kname, kernel_ms[kname])
    roof["traffic"] = None
    roof["kernel"] = kname
    roof["avg_launch_ms"] = round(kernel_ms[kname], 4)
    step_bytes = alg["forward"]["bytes"] + alg["backward"]["bytes"]
    res = {
        "metric": PW_METRIC, "value": round(w.B * w.N / (ms_step * 1e-3), 1), "unit": "queries/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded Philox inputs shaped like the paper's video-latent grids)",
        "config": {"workload": w.name, "grid_TxHxW": [w.T, w.H, w.W], "batch": w.B,
                   "heads": w.heads, "head_dim": w.head_dim, "kernel": [w.kt, w.kh, w.kw],
                   "points": w.P, "backward": True, "parallelism": "single GPU"},
        "kernel_ms": {n: round(t, 4) for n, t in kernel_ms.items()},
        "kernel_roofline": {n: kernel_roofline(w, alg, n, t) for n, t in kernel_ms.items()
                            if n in alg},
        "hbm_gbs_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "roofline": roof, "input_gen_s": round(t_gen, 1),
    }
    if args.cpu_budget > 0:
        import numpy as np

        import oracle
        shape = (w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw)
        frames = 0
        t0 = time.perf_counter()
        while frames < w.T and time.perf_counter() - t0 < args.cpu_budget:
            rows = (np.arange(w.H * w.W, dtype=np.int64) + frames * w.H * w.W) * w.heads
            oracle.pw_forward(shape, w.dtype, logits, v, off, rows=rows)
            oracle.pw_backward_slab(shape, w.dtype, logits, v, off, dout, 0, 0, frames, frames + 1)
            frames += 1
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {
            "value": frames * w.H * w.W / w.heads / dt, "unit": "queries/s",
            "cores": oracle.threads(), "kind": "oracle", **host_info(),
            "sample": f"head 0 frames [0,{frames}) of {w.name}: forward + backward incl. dV "
                      f"scatter, fp64, {dt:.1f} s; scaled to query tokens (all {w.heads} heads)"}
    print(json.dumps(res), flush=True)


def win_boxes(w):
    """Sizes of the boxes the shifted windows cut the grid into: along each axis the cuts are
    shift + n * window (plus the grid ends); a query attends to every token of its box."""
    import numpy as np

    def axis(size, win, shift):
        off = shift - win if shift > 0 else 0
        n = -(-(size - off) // win)
        lo = np.maximum(off + win * np.arange(n), 0)
        hi = np.minimum(off + win * (np.arange(n) + 1), size)
        return hi - lo

    lt = axis(w.T, w.window[0], w.shift[0])
    lh = axis(w.H, w.window[1], w.shift[1])
    lw = axis(w.W, w.window[2], w.shift[2])
    return (lt[:, None, None] * lh[None, :, None] * lw[None, None, :]).ravel()


def win_algorithmic(w):
    """Algorithmic FLOPs (and HBM bytes) per launch of the window-attention kernels.  A box of n
    tokens and one head costs 2 n^2 D FLOPs per n x n x D product (a multiply-add is 2 FLOPs):
      win_fwd_kernel   S = Q K^T and O = P V: 4 n^2 D; reads q, k, v, writes out, out_res (bf16)
                       and lse
      win_dq_kernel    S, dP = dout V^T and dq = dS K: 6 n^2 D; reads q, k, v, out, out_res,
                       dout, lse, writes dq (fp32) and Delta
      win_dkdv_kernel  S, dP, dV = P^T dout and dK = dS^T Q: 8 n^2 D; reads q, k, v, dout, lse,
                       Delta, writes dk, dv (fp32)
      backward         the two passes (S and dP are formed in both)
    The kernels take P and dS into the products as bf16 hi + lo pairs, which executes 2 n^2 D
    more per such product (6, 8 and 12 n^2 D instead of 4, 6 and 8); those are not counted."""
    n2 = float((win_boxes(w).astype("float64") ** 2).sum())
    per = w.B * w.heads * n2 * w.head_dim
    rows = w.queries
    D = w.head_dim
    work = {
        "win_fwd_kernel": (rows * (5 * 2 * D + 4), 4 * per),
        "win_dq_kernel": (rows * (6 * 2 * D + 4 * D + 8), 6 * per),
        "win_dkdv_kernel": (rows * (4 * 2 * D + 8 * D + 8), 8 * per),
    }
    work["backward"] = (work["win_dq_kernel"][0] + work["win_dkdv_kernel"][0], 14 * per)
    return {k: {"bytes": b, "flops": f} for k, (b, f) in work.items()}


def mfma_roofline(work, ms):
    ach = work["flops"] / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "achieved": round(ach, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(ach / MFMA_BF16_PEAK_TFLOPS, 4)}


def bench_win(args, torch, dsa, testgen, to_device):
    """One step = forward (with the output residual) and backward of the shifted-window
    attention."""
    w = testgen.WIN_WORKLOADS[args.workload]
    t_gen = time.perf_counter()
    host = testgen.gen_win_inputs(w, progress=lambda m: print(m, file=sys.stderr, flush=True))
    print("copying inputs to the GPU", file=sys.stderr, flush=True)
    qd, kd, vd, gd = (to_device(a, True) for a in host)
    t_gen = time.perf_counter() - t_gen
    print(f"inputs resident after {t_gen:.1f} s; timing", file=sys.stderr, flush=True)
    kw = dict(window=w.window, shift=w.shift)
    out, lse, res = dsa.win_forward(qd, kd, vd, **kw)
    f32 = dict(dtype=torch.float32, device=qd.device)
    grads = tuple(torch.empty(qd.shape, **f32) for _ in range(3))
    need = dsa.dsa3d_win_backward_workspace_size(dsa.make_win_desc(
        w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.window, w.shift))
    workspace = torch.empty(need, dtype=torch.uint8, device=qd.device)

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record()
        return evs

    K = args.steps
    ev = [new_events(2) for _ in range(K)]
    ph = [new_events(dsa.DSA3D_WIN_BACKWARD_PHASES + 1) for _ in range(K)]

    def step(s=None):
        if s is not None:
            ev[s][0].record()
        dsa.win_forward(qd, kd, vd, out=out, lse=lse, out_res=res, **kw)
        if s is not None:
            ev[s][1].record()
        dsa.win_backward(qd, kd, vd, out, res, lse, gd, grads=grads, workspace=workspace,
                         phase_events=None if s is None else ph[s], **kw)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for s in range(K):
        step(s)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / K
    kernel_ms = {"win_fwd_kernel": sum(e[0].elapsed_time(e[1]) for e in ev) / K}
    for i, n in enumerate(["win_dq_kernel", "win_dkdv_kernel"]):
        kernel_ms[n] = sum(p[i].elapsed_time(p[i + 1]) for p in ph) / K
    alg = win_algorithmic(w)
    kname = max(kernel_ms, key=lambda n: kernel_ms[n])
    roof = mfma_roofline(alg[kname], kernel_ms[kname])
    roof["traffic"] = measured_traffic(w.name, kname)
    roof["kernel"] = kname
    roof["avg_launch_ms"] = round(kernel_ms[kname], 4)
    step_flops = alg["win_fwd_kernel"]["flops"] + alg["backward"]["flops"]
    res_json = {
        "metric": WIN_METRIC, "value": round(w.B * w.N / (ms_step * 1e-3), 1), "unit": "queries/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Philox inputs shaped like the paper's video-latent grids)",
        "config": {"workload": w.name, "grid_TxHxW": [w.T, w.H, w.W], "batch": w.B,
                   "heads": w.heads, "head_dim": w.head_dim, "window": list(w.window),
                   "shift": list(w.shift), "backward": True, "parallelism": "single GPU"},
        "kernel_ms": {n: round(t, 4) for n, t in kernel_ms.items()},
        "kernel_roofline": {n: mfma_roofline(alg[n], t) for n, t in kernel_ms.items()},
        "step_tflops_algorithmic": round(step_flops / (ms_step * 1e-3) / 1e12, 2),
        "step_mfma_frac_algorithmic": round(step_flops / (ms_step * 1e-3) / 1e12
                                            / MFMA_BF16_PEAK_TFLOPS, 4),
        "roofline": roof, "input_gen_s": round(t_gen, 1),
    }
    if args.cpu_budget > 0:
        import oracle
        q, k, v, dout = host
        frames = []
        t0 = time.perf_counter()
        f = min(1, w.T - 1)
        while f < w.T and time.perf_counter() - t0 < args.cpu_budget:
            oracle.win_forward(w.shape12(), "bf16", q, k, v, frames=(f, f + 1))
            oracle.win_backward(w.shape12(), "bf16", q, k, v, dout, frames=(f, f + 1))
            frames.append(f)
            f += 1
        dt = time.perf_counter() - t0
        res_json["cpu_baseline"] = {
            "value": round(len(frames) * w.H * w.W * w.B / dt, 2), "unit": "queries/s",
            "cores": oracle.threads(), "kind": "oracle", **host_info(),
            "sample": f"frames {frames[0]}..{frames[-1]} of {w.name} (all heads): forward + "
                      f"backward of their queries, fp64, {dt:.1f} s"}
    print(json.dumps(res_json), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--op", choices=["dsa", "dwconv", "pw", "win"], default="dsa",
                    help="dsa: the 3D-DSA operator (default); dwconv: the depthwise 3D "
                         "convolution term of Eq. (1) (workloads dwconv_*); pw: the "
                         "predicted-weights variant (workloads pw_*); win: the Swin-DiT "
                         "shifted-window attention (workloads swin_*)")
    ap.add_argument("--workload", default=None,
                    help=f"default {DEFAULT_WORKLOAD} (dsa) or {DEFAULT_CONV_WORKLOAD} (dwconv)")
    ap.add_argument("--forward-only", action="store_true",
                    help="time the forward alone (workloads without a backward pass)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of CPU-oracle work for cpu_baseline (0 = skip)")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("READS", "WRITES", "COPYR", "COPYW"),
                    help="summarise four rocprofv3 --pmc output folders (READ_COUNTERS and "
                         "WRITE_COUNTERS of a bench command and of --copy-probe) into "
                         "profiles/traffic_<workload>.json (no GPU needed)")
    ap.add_argument("--working-set-probe", action="store_true",
                    help="only print the gather rate against working-set size and exit")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 3 device-to-device copies of MIB MiB and exit (checks the "
                         "traffic counters against a known byte count)")
    args = ap.parse_args()

    if args.workload is None:
        args.workload = {"dwconv": DEFAULT_CONV_WORKLOAD, "pw": DEFAULT_PW_WORKLOAD,
                         "win": DEFAULT_WIN_WORKLOAD}.get(args.op, DEFAULT_WORKLOAD)
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
    if args.working_set_probe:
        working_set_curve()
        return
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
    if args.op == "dwconv":
        bench_dwconv(args, torch, dsa, testgen, to_device)
        return
    if args.op == "pw":
        bench_pw(args, torch, dsa, testgen, to_device)
        return
    if args.op == "win":
        bench_win(args, torch, dsa, testgen, to_device)
        return
    w = testgen.WORKLOADS[args.workload]
    do_bwd = w.backward and not args.forward_only
    t_gen = time.perf_counter()
    host = testgen.gen_inputs(w, progress=lambda m: print(m, file=sys.stderr, flush=True))
    if host[4] is None and do_bwd:
        host = host[:4] + (testgen.gen_tensor(w, testgen.TID_DOUT, w.qkv_shape(), w.dout, True),)
    q, k, v, off, dout = host
    bf = w.dtype == "bf16"
    print("copying inputs to the GPU", file=sys.stderr, flush=True)
    qd, kd, vd = (to_device(a, bf) for a in (q, k, v))
    od = to_device(off, False)
    gd = to_device(dout, bf) if do_bwd else None
    t_gen = time.perf_counter() - t_gen
    print(f"inputs resident after {t_gen:.1f} s; timing", file=sys.stderr, flush=True)
    kern = (w.kt, w.kh, w.kw)
    out, lse = dsa.forward(qd, kd, vd, od, kernel=kern)
    grads = None
    workspace = None
    if do_bwd:
        f32 = dict(dtype=torch.float32, device=qd.device)
        grads = (torch.empty(q.shape, **f32), torch.empty(q.shape, **f32),
                 torch.empty(q.shape, **f32), torch.empty(off.shape, **f32))
        need = dsa.dsa3d_backward_workspace_size(dsa.make_desc(
            w.B, w.T, w.H, w.W, w.heads, w.head_dim, w.kt, w.kh, w.kw, w.dtype))
        workspace = torch.empty(need, dtype=torch.uint8, device=qd.device)

    def new_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:  # create the HIP events before they are handed to the library
            e.record()
        return evs

    nph = dsa.DSA3D_BACKWARD_PHASES
    K = args.steps
    ev = [new_events(3) for _ in range(K)]
    ph = [new_events(nph + 1) for _ in range(K)] if do_bwd else None

    def step(s=None):
        if s is not None:
            ev[s][0].record()
        dsa.forward(qd, kd, vd, od, kernel=kern, out=out, lse=lse)
        if s is not None:
            ev[s][1].record()
        if do_bwd:
            dsa.backward(qd, kd, vd, od, lse, gd, kernel=kern, grads=grads, workspace=workspace,
                         phase_events=None if s is None else ph[s])
        if s is not None:
            ev[s][2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s in range(K):
        step(s)
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    fwd_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / K
    bwd_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / K if do_bwd else 0.0
    ms_step = total_ms / K
    # average duration of each kernel (HIP events on the stream the kernels run on)
    kernel_ms = {"fwd_kernel": fwd_ms}
    if do_bwd:
        for i, n in enumerate(BWD_PHASES):
            kernel_ms[n] = sum(p[i].elapsed_time(p[i + 1]) for p in ph) / K

    alg = algorithmic(w)
    step_bytes = alg["forward"]["bytes"] + (alg["backward"]["bytes"] if do_bwd else 0)
    tokens = w.B * w.N
    # dominant kernel: the longest single kernel of the step
    kname = max((n for n in kernel_ms if n in alg), key=lambda n: kernel_ms[n])
    roof = kernel_roofline(w, alg, kname, kernel_ms[kname])
    tr = measured_traffic(w.name, kname)
    roof["traffic"] = None if tr is None else round(tr)
    roof["kernel"] = kname
    roof["avg_launch_ms"] = round(kernel_ms[kname], 4)

    # the bound the kernels actually meet: bytes through the per-unit vector-memory path
    ceil = gather_ceiling(w.head_dim * (2 if w.dtype == "bf16" else 4))
    vm = vmem_bytes(w)
    gather_path = {"ceiling": ceil}
    for n, b in vm.items():
        if n in kernel_ms:
            tbps = b / (kernel_ms[n] * 1e-3) / 1e12
            gather_path[n] = {"bytes_per_launch": b, "achieved_TBps": round(tbps, 2),
                              "frac_of_l1_ceiling": round(tbps / ceil["l1_TBps"], 3),
                              "frac_of_l2_ceiling": round(tbps / ceil["l2_TBps"], 3)}

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
        "kernel_ms": {n: round(t, 4) for n, t in kernel_ms.items()},
        "kernel_roofline": {n: kernel_roofline(w, alg, n, t) for n, t in kernel_ms.items()
                            if n in alg},
        "hbm_gbs_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "hbm_frac_algorithmic": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "token_head_rows_per_s": round(w.queries / (ms_step * 1e-3), 1),
        "roofline": roof,
        "hbm_rocprof": hbm_rocprof(w.name, do_bwd, ms_step, step_bytes),
        "hbm_ceiling": copy_ceiling(torch),
        "gather_path": gather_path,
        "input_gen_s": round(t_gen, 1),
    }
    if args.cpu_budget > 0:
        res["cpu_baseline"] = cpu_baseline(w, host, args.cpu_budget, backward=do_bwd)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

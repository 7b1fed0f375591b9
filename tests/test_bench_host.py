"""Host-side logic of bench.py (CPU only): roofline classification, kernel-name mapping, the
algorithmic byte and FLOP counts per launch, the rocprof-counted step traffic, the one-GPU rule
and the gather probe's argument checks."""
import ctypes
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import testgen  # noqa: E402


def test_roofline_takes_the_slower_of_memory_and_arithmetic():
    # 8e9 bytes take 1 ms at 8 TB/s; 1e9 flops take 6.4 us at 157.3 TFLOP/s: HBM-bound
    r = bench.roofline({"bytes": 8e9, "flops": 1e9}, 2.0)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"
    assert r["achieved"] == pytest.approx(4000.0) and r["frac"] == pytest.approx(0.5)
    # 1.573e12 flops take 10 ms at the fp32 vector peak; 8e9 bytes 1 ms: ALU-bound
    r = bench.roofline({"bytes": 8e9, "flops": 1.573e12}, 20.0)
    assert r["bound"] == "alu" and r["peak"] == bench.VALU_PEAK_TFLOPS
    assert r["frac"] == pytest.approx(0.5, rel=1e-3)


def test_the_bf16_gather_is_priced_against_the_matrix_peak():
    w16 = testgen.WORKLOADS["fwdbwd_64x34x60"]
    alg = bench.algorithmic(w16)
    g = bench.kernel_roofline(w16, alg, "bwd_gather_kernel", 3.0)
    # 32 P D flops per row against 2.5 PFLOP/s take less time than the HBM bytes at 8 TB/s
    assert g["bound"] == "hbm"
    assert bench.kernel_roofline(w16, alg, "bwd_kpass_kernel", 4.0)["bound"] == "alu"
    w32 = testgen.WORKLOADS["tiny_f32"]
    a32 = bench.algorithmic(w32)
    assert bench.kernel_roofline(w32, a32, "bwd_gather_kernel", 1.0) == bench.roofline(
        a32["bwd_gather_kernel"], 1.0)


def test_kernel_names_map_to_the_phases_the_bench_times():
    assert bench.kernel_base("void dsa3d::(anonymous namespace)::fwd_kernel<64, true, false>"
                             "(dsa3d::Geometry, ...)") == "fwd_kernel"
    assert bench.kernel_base("dsa3d::bwd_gather_mfma_kernel<64, false>(...)") == "bwd_gather_kernel"
    assert bench.kernel_base("dsa3d::bwd_gather_kernel<32, false, false>(...)") == "bwd_gather_kernel"
    assert bench.kernel_base("__amd_rocclr_copyBuffer") == "__amd_rocclr_copyBuffer"


def test_algorithmic_counts_follow_the_documented_per_row_formulas():
    w = testgen.WORKLOADS["tiny_f32"]  # 512 rows, P = 27, D = 32, fp32
    rows, P, D, s = w.queries, w.P, w.head_dim, 4
    alg = bench.algorithmic(w)
    assert alg["fwd_kernel"]["bytes"] == rows * (4 * D * s + 12 * P + 4)
    assert alg["fwd_kernel"]["flops"] == rows * 32 * P * D
    assert alg["bwd_gather_kernel"]["bytes"] == rows * (2 * D * s + 8 * D)
    assert alg["backward"]["flops"] == rows * 80 * P * D
    vm = bench.vmem_bytes(w)
    assert vm["fwd_kernel"] == rows * (16 * P * D * s + 2 * D * s + 12 * P + 4)
    # the K pass keeps the K halves of the records in registers for rows of at most 5 chunks
    # of D s / 16 points (here 4 chunks of 8), and writes and reads them back beyond that
    kpass = 8 * P * D * s + D * s + 24 * P + 4 + 4 * P + 16 * P + 4 * D + 12 * P + 8 * P + 24 * P
    assert vm["bwd_kpass_kernel"] == rows * kpass
    w7 = testgen.WORKLOADS["paper_3x7x7_64x68x120"]  # P = 147, D = 128, bf16: 10 chunks of 16
    P7, D7 = w7.P, w7.head_dim
    kpass7 = (8 * P7 * D7 * 2 + D7 * 2 + 24 * P7 + 4 + 4 * P7 + 16 * P7 + 32 * P7 + 4 * D7
              + 12 * P7 + 8 * P7 + 24 * P7)
    assert bench.vmem_bytes(w7)["bwd_kpass_kernel"] == w7.queries * kpass7


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


def test_gather_probe_rejects_bad_arguments_before_touching_the_device():
    path = bench.PROBE_LIB
    if not os.path.exists(path):
        pytest.skip("probe library not built")
    lib = ctypes.CDLL(path)
    fn = lib.dsa3d_probe_gather
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]
    ms, nb = ctypes.c_float(), ctypes.c_double()
    assert fn(6, 128, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1   # no such source
    assert fn(4, 128, 8, 12, ctypes.byref(ms), ctypes.byref(nb)) == -1  # not 8 loads a step
    assert fn(-1, 128, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1
    assert fn(2, 48, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1    # row size
    assert fn(0, 128, 0, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1   # no blocks
    assert fn(1, 64, 8, 8, None, ctypes.byref(nb)) == -1                # null output
    ws = lib.dsa3d_probe_working_set
    ws.argtypes = [ctypes.c_int, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_int, ctypes.c_int,
                   ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_double)]
    assert ws(192, 256, 1 << 20, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1   # row size
    assert ws(256, 128, 1 << 20, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1   # stride < row
    assert ws(256, 6144, 1 << 30, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1  # span > 4 GB
    assert ws(256, 250, 1 << 20, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1   # not 16-B
    assert ws(256, 256, 100, 8, 8, ctypes.byref(ms), ctypes.byref(nb)) == -1       # < one row


def test_rocprof_step_traffic_sums_the_step_kernels_and_refuses_stale_counters(tmp_path, monkeypatch):
    import json
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    names = ("fwd_kernel",) + bench.BWD_KERNELS
    kernels = {n: {"hbm_bytes": 10 ** i} for i, n in enumerate(names)}
    doc = {"workload": "w", "kernel_source_hash": bench.kernel_source_hash("dsa"), "kernels": kernels}
    (tmp_path / "traffic_w.json").write_text(json.dumps(doc))
    assert bench.measured_step_traffic("w", False) == 1
    assert bench.measured_step_traffic("w", True) == 11111111
    # 8e9 bytes in 1 ms is the 8 TB/s peak
    kernels["fwd_kernel"]["hbm_bytes"] = 8 * 10 ** 9
    (tmp_path / "traffic_w.json").write_text(json.dumps(doc))
    r = bench.hbm_rocprof("w", False, 1.0, 2 * 10 ** 9)
    assert r["GBps"] == pytest.approx(8000.0) and r["frac_of_peak"] == pytest.approx(1.0)
    assert r["ratio_to_algorithmic"] == pytest.approx(4.0) and r["counted_at"] == "L2 egress"
    # a kernel of the step without counters, counters of other sources, no file: no figure
    del kernels["bwd_kpass_kernel"]
    (tmp_path / "traffic_w.json").write_text(json.dumps(doc))
    assert bench.measured_step_traffic("w", True) is None
    doc["kernel_source_hash"] = "0" * 16
    (tmp_path / "traffic_w.json").write_text(json.dumps(doc))
    assert bench.hbm_rocprof("w", False, 1.0, 1) is None
    assert bench.hbm_rocprof("absent", True, 1.0, 1) is None


def _counter_csv(path, rows):
    """rows: (dispatch id, kernel name, counter, value) as rocprofv3 writes them."""
    import csv
    path.mkdir()
    with open(path / "p_counter_collection.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_pmc_summary_counts_read_requests_by_size(tmp_path, monkeypatch):
    """Read bytes are 32, 64 and 128 bytes per request of each size (FETCH_SIZE, which counts
    a 128-byte request as 64 bytes on this GPU, is not used); writes are WRITE_SIZE KiB; the
    copy's figures are stored as a check of the accounting."""
    import json
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path / "profiles"))
    k = "void dsa3d::fwd_kernel<128, true, false>(...)"
    reads = []
    for d in (1, 2):  # two launches, averaged
        reads += [(d, k, "TCC_EA0_RDREQ_32B_sum", 10), (d, k, "TCC_EA0_RDREQ_64B_sum", 20),
                  (d, k, "TCC_EA0_RDREQ_128B_sum", 1000 * d), (d, k, "TCC_EA0_RDREQ_sum", 1030 + 1000 * (d - 1))]
    writes = [(d, k, c, v) for d in (1, 2) for c, v in
              (("WRITE_SIZE", 4.0), ("TCC_ATOMIC_sum", 7), ("TCC_EA0_ATOMIC_sum", 3))]
    cp = "__amd_rocclr_copyBuffer"
    copy_r = [(1, cp, "TCC_EA0_RDREQ_32B_sum", 0), (1, cp, "TCC_EA0_RDREQ_64B_sum", 0),
              (1, cp, "TCC_EA0_RDREQ_128B_sum", 8192), (1, cp, "TCC_EA0_RDREQ_sum", 8192)]
    copy_w = [(1, cp, "WRITE_SIZE", 1024.0), (1, cp, "TCC_ATOMIC_sum", 0),
              (1, cp, "TCC_EA0_ATOMIC_sum", 0)]
    for name, rows in (("r", reads), ("w", writes), ("cr", copy_r), ("cw", copy_w)):
        _counter_csv(tmp_path / name, rows)
    bench.pmc_summary("wl", str(tmp_path / "r"), str(tmp_path / "w"), str(tmp_path / "cr"),
                      str(tmp_path / "cw"), 1)
    doc = json.loads((tmp_path / "profiles" / "traffic_wl.json").read_text())
    kr = doc["kernels"]["fwd_kernel"]
    assert kr["fetch_bytes"] == 32 * 10 + 64 * 20 + 128 * 1500
    assert kr["write_bytes"] == 4096 and kr["hbm_bytes"] == kr["fetch_bytes"] + 4096
    assert kr["atomics_l2"] == 7 and kr["atomics_past_l2"] == 3
    assert kr["read_requests_of_known_size"] == 1.0
    assert doc["copy_check"] == {"mib": 1, "read_bytes_per_byte": 1.0, "write_bytes_per_byte": 1.0}


def test_kernel_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    import shutil
    for name in bench.FAMILY_SOURCES["win"]:
        shutil.copy(os.path.join(bench.CSRC, name), tmp_path / name)
    monkeypatch.setattr(bench, "CSRC", str(tmp_path))
    h0 = bench.kernel_source_hash("win")
    src = tmp_path / bench.FAMILY_SOURCES["win"][0]
    text = src.read_text()
    src.write_text("// a new comment\n/* and a block\n   comment */\n" + text.replace("\n", "  \n", 3))
    assert bench.kernel_source_hash("win") == h0
    src.write_text(text + "\nstatic int added_code = 1;\n")
    assert bench.kernel_source_hash("win") != h0

"""bench.py's host logic without a GPU: the one-GPU contract, and the counter
arithmetic that turns rocprofv3 FETCH_SIZE / WRITE_SIZE rows into traffic."""
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _write_rows(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for d, (kernel, grid, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": d, "Kernel_Name": kernel, "Grid_Size": grid, "Counter_Name": counter,
                        "Counter_Value": value})


def test_unfused_path_rejects_fused_only_options():
    for opt in ("--graph", "--lr-schedule", "--lars"):
        r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--path", "unfused", opt],
                           capture_output=True, text=True, timeout=120)
        assert r.returncode != 0 and "fused path" in r.stderr, (opt, r.stderr)


def test_derive_traffic_scales_by_the_calibration_copy(tmp_path, monkeypatch):
    """Synthetic counter rows: the 1 GiB copy reads FETCH_SIZE = half its bytes
    and WRITE_SIZE = all of them, so the step's rows are scaled by 2 and 1;
    two dispatches of the step kernel average; the ceiling copy (a larger grid)
    is ignored."""
    wl = workloads.WORKLOADS["resnet50_flat"]
    alg = wl.algorithmic_bytes(16)
    read_b, write_b = wl.n * (16 * 4 + 8), wl.n * (8 + 16 * 4)
    gib_kib = (1 << 30) / 1024
    step = "void lsgd::step_flat_ct<float, 4, 4, 2>(lsgd::StepArgs)"
    copy = "lsgd::stream_copy_kernel(unsigned int __vector(4)*)"
    calib_grid = (1 << 28) // 4          # one lane per 16 bytes of the 1 GiB copy
    fetch = [(copy, calib_grid, gib_kib / 2), (copy, calib_grid * 2, 999.0),
             (step, 1, read_b / 1024 / 2), (step, 1, read_b / 1024 / 2)]
    write = [(copy, calib_grid, gib_kib), (step, 1, write_b / 1024), (step, 1, write_b / 1024)]
    fcsv, wcsv = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_rows(fcsv, "FETCH_SIZE", fetch)
    _write_rows(wcsv, "WRITE_SIZE", write)
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    args = bench.parse_args(["--derive-traffic", "--workload", "resnet50_flat", "--fetch-csv", str(fcsv),
                             "--write-csv", str(wcsv)])
    bench.derive_traffic(args)
    out = json.load(open(tmp_path / "traffic_resnet50_flat_R16.json"))
    assert abs(out["fetch_scale"] - 2.0) < 1e-12 and abs(out["write_scale"] - 1.0) < 1e-12
    assert abs(out["traffic_over_algorithmic"] - 1.0) < 1e-9
    assert out["algorithmic_bytes"] == alg and out["kernels"]["step_flat_ct"]["dispatches"] == [2, 2]


def test_derive_traffic_per_kernel_with_a_copy_out_pass(tmp_path, monkeypatch):
    """A step split into the step kernel (writing its share of the replicas,
    4 of 16 binary32 ones here) and the copy-out pass (the other 12): each
    kernel's traffic against its own algorithmic bytes, the step's total, and
    the per-kernel lookup the benchmark's roofline uses."""
    wl = workloads.WORKLOADS["resnet50_flat"]
    R = 16
    k_step = bench.step_replicas(wl, R)
    assert k_step == 4
    gib_kib = (1 << 30) / 1024
    step = "void lsgd::step_flat_ct<float, 4, 4, 2>(lsgd::StepArgs)"
    cpy = "void lsgd::copy_out_rmajor_kernel<4, 2, 1>(lsgd::StepArgs)"
    copy = "lsgd::stream_copy_kernel(unsigned int __vector(4)*)"
    calib_grid = (1 << 28) // 4
    s_read, s_write = wl.n * (16 * 4 + 8), wl.n * (8 + 4 * k_step)
    c_read, c_write = wl.n * 4 * 1.5, wl.n * 4 * (R - k_step)      # the pass reads p 1.5 times here
    fetch = [(copy, calib_grid, gib_kib / 2), (step, 1, s_read / 2048), (cpy, 1, c_read / 2048),
             (step, 1, s_read / 2048), (cpy, 1, c_read / 2048)]
    write = [(copy, calib_grid, gib_kib), (step, 1, s_write / 1024), (cpy, 1, c_write / 1024)]
    fcsv, wcsv = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_rows(fcsv, "FETCH_SIZE", fetch)
    _write_rows(wcsv, "WRITE_SIZE", write)
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    args = bench.parse_args(["--derive-traffic", "--workload", "resnet50_flat", "--fetch-csv", str(fcsv),
                             "--write-csv", str(wcsv)])
    bench.derive_traffic(args)
    out = json.load(open(tmp_path / "traffic_resnet50_flat_R16.json"))
    k = out["kernels"]
    assert set(k) == {"step_flat_ct", "copy_out"}
    assert k["step_flat_ct"]["algorithmic_bytes"] == wl.algorithmic_bytes(k_step)
    assert abs(k["step_flat_ct"]["traffic_over_algorithmic"] - 1.0) < 1e-9
    assert k["copy_out"]["algorithmic_bytes"] == wl.n * (4 + 4 * (R - k_step))
    assert abs(k["copy_out"]["traffic_bytes"] - (c_read + c_write)) < 1.0
    assert abs(out["traffic_bytes"] - (s_read + s_write + c_read + c_write)) < 1.0
    assert bench.stored_traffic(wl, R, False, "copy_out_rmajor_kernel") == k["copy_out"]["traffic_bytes"]
    assert bench.stored_traffic(wl, R, False, "step_flat_ct") == k["step_flat_ct"]["traffic_bytes"]
    assert bench.stored_traffic(wl, R) == out["traffic_bytes"]


def test_all_cores_cpu_baseline_runs_the_oracle_on_blocks(monkeypatch):
    """The all-cores baseline on host tensors of the tiny workload: one block per
    host thread, the result fields, and (separately) that stepping the oracle
    block by block gives the bits of one call over the whole range."""
    import types
    import numpy as np
    import torch
    import oracle
    wl = workloads.WORKLOADS["tiny"]
    monkeypatch.setenv("OMP_NUM_THREADS", "3")
    gen = torch.Generator().manual_seed(5)
    st = types.SimpleNamespace(
        wl=wl, R=2, plan=None, reduction="mean_of_means", broadcast_grad=False, gow=wl.group_of_worker(),
        params=[torch.randn(wl.n, generator=gen)], mom=[torch.zeros(wl.n)],
        grads=[[torch.randn(wl.n, generator=gen) * 1e-2] for _ in range(wl.n_workers)])
    out = bench.cpu_baseline_all_cores(st, 0.05)
    assert out["cores"] == min(3, bench.host_threads()) and out["value"] > 0 and out["kind"] == "oracle"
    # element blocks are independent: blockwise steps equal one whole step, bit for bit
    rng = np.random.default_rng(3)
    n, T = 10_007, 4
    p0 = rng.standard_normal(n).astype(np.float32)
    gs = [rng.standard_normal(n).astype(np.float32) * 1e-2 for _ in range(4)]
    pa, ma, ra = p0.copy(), np.zeros(n, np.float32), [np.zeros(n, np.float32)]
    oracle.lsgd_step(pa, ma, gs, [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4, ra)
    pb, mb, rb = p0.copy(), np.zeros(n, np.float32), [np.zeros(n, np.float32)]
    B = -(-n // T)
    for k in range(T):
        sl = slice(k * B, min(n, (k + 1) * B))
        oracle.lsgd_step(pb[sl], mb[sl], [g[sl] for g in gs], [0, 0, 1, 1], 2, 0.1, 0.9, 1e-4, [rb[0][sl]])
    assert pa.tobytes() == pb.tobytes() and ma.tobytes() == mb.tobytes() and ra[0].tobytes() == rb[0].tobytes()


def test_library_ranges_cover_the_vector():
    """The element ranges of a long flat step with a copy-out pass (or without
    replicas): one range up to 2^26 elements; beyond, ceil(n / 2^24) contiguous
    ranges of at least 2^23 elements that start on multiples of 2^20 elements
    (2 MB in a buffer of 2-byte elements) and cover [0, n)."""
    assert bench.library_ranges(1 << 26) == [(0, 1 << 26)]
    for n in ((1 << 26) + 1, 350_000_000, 352_321_536, (1 << 26) + (1 << 25) + 12_345, (1 << 31) + 7):
        r = bench.library_ranges(n)
        assert len(r) == -(-n // (1 << 24))
        assert r[0][0] == 0 and r[-1][1] == n
        assert all(a % (1 << 20) == 0 and b - a >= 1 << 23 for a, b in r)
        assert all(r[i][1] == r[i + 1][0] for i in range(len(r) - 1))


def test_range_rule_matches_the_library_source():
    """bench.py's copy of the library's range constants equals the values in
    the C++ source (kRangeSplitMin, kRangeElems, kRangeAlign)."""
    import re
    src = open(os.path.join(ROOT, "paper_1906_05936_amd", "csrc", "lsgd_flat.hip")).read()

    def const(name):
        m = re.search(r"constexpr int64_t %s = int64_t\{1\} << (\d+);" % name, src)
        assert m, name
        return 1 << int(m.group(1))
    assert const("kRangeSplitMin") == bench.RANGE_SPLIT_MIN
    assert const("kRangeElems") == bench.RANGE_ELEMS
    assert const("kRangeAlign") == bench.RANGE_ALIGN


def test_derive_traffic_counts_every_range_launch(tmp_path, monkeypatch):
    """A step run in element ranges (the 3.5e8-element workload: 21 launches of
    each kernel per step): the per-dispatch counters are scaled to the step."""
    wl = workloads.WORKLOADS["large"]
    R = wl.n_workers
    K = len(bench.library_ranges(wl.n))
    gib_kib = (1 << 30) / 1024
    step = "void lsgd::step_flat_ct<unsigned short, 8, 8, 1, 0>(lsgd::StepArgs)"
    cpy = "void lsgd::copy_out_rmajor_kernel<8, 1, 2>(lsgd::StepArgs)"
    copy = "lsgd::stream_copy_kernel(unsigned int __vector(4)*)"
    calib_grid = (1 << 28) // 4
    s_read, s_write = wl.n * (64 * 2 + 8) / K, wl.n * 8 / K
    c_read, c_write = wl.n * 4 / K, wl.n * 2 * R / K
    fetch = [(copy, calib_grid, gib_kib / 2)] + [(step, 1, s_read / 2048), (cpy, 1, c_read / 2048)] * K
    write = [(copy, calib_grid, gib_kib)] + [(step, 1, s_write / 1024), (cpy, 1, c_write / 1024)] * K
    fcsv, wcsv = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_rows(fcsv, "FETCH_SIZE", fetch)
    _write_rows(wcsv, "WRITE_SIZE", write)
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    args = bench.parse_args(["--derive-traffic", "--workload", "large", "--fetch-csv", str(fcsv),
                             "--write-csv", str(wcsv)])
    bench.derive_traffic(args)
    out = json.load(open(tmp_path / ("traffic_large_R%d.json" % R)))
    for k in ("step_flat_ct", "copy_out"):
        assert out["kernels"][k]["launches_per_step"] == K
        assert abs(out["kernels"][k]["traffic_over_algorithmic"] - 1.0) < 1e-9, k

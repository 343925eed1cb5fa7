"""The benchmark's JSON line on the GPU: the output contract (one JSON line with
the metric, value, roofline and per-kernel fields) for the default path and for
the measurement variants, on the tiny workload with a few steps."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*extra):
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "5", "--warmup", "1",
           "--no-cpu-baseline"] + list(extra)
    print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout
    return json.loads(lines[0])


def check_common(b):
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in b, key
    assert b["n_gpus"] == 1 and b["steps"] == 5 and b["warmup"] == 1 and b["value"] > 0
    rl = b["roofline"]
    assert rl["bound"] == "hbm" and rl["peak"] == 8000.0 and rl["unit"] == "GB/s"
    assert abs(rl["frac"] - rl["achieved"] / rl["peak"]) < 1e-3
    reps = b["repeats_ms_per_step"]     # five timed loops of K steps; the line reports their median
    assert len(reps) == 5 and abs(b["ms_per_step"] - sorted(reps)[2]) < 1e-6
    st = b["settle"]                    # untimed steps before the first timed loop
    assert st["seconds"] >= 0 and st["steps"] >= (10 if st["seconds"] > 0 else 0)


def test_bench_default_line():
    b = run_bench("--no-r0")
    check_common(b)
    assert b["config"]["workload"] == "tiny" and b["config"]["copy_out"] == "in the step kernel"
    cold = b["cold_cache"]       # a cache flush before every timed step
    assert cold["ms_per_step"] > 0 and len(cold["repeats_ms_per_step"]) == 5


def test_bench_broadcast_and_literal_variants():
    b = run_bench("--no-r0", "--no-cold", "--broadcast-grad", "--reduction", "literal")
    check_common(b)
    assert b["config"]["reduction"] == "literal" and b["config"]["broadcast_grad"]
    assert b["roofline"]["kernel"].startswith("step_flat_ct")


def test_bench_split_step_reports_the_dominant_kernel():
    b = run_bench("--no-r0", "--copy-out", "separate")
    check_common(b)
    names = [k["kernel"] for k in b["kernels"]]
    assert names == ["step_flat_ct", "copy_out_rmajor_kernel"]
    dom = max(b["kernels"], key=lambda k: k["ms"])
    assert b["roofline"]["kernel"] == dom["kernel"] and b["roofline"]["algorithmic_bytes"] == dom["algorithmic_bytes"]


def test_bench_schedule_and_graph_variants():
    b = run_bench("--lr-schedule", "--graph", "--copy-out", "separate")
    check_common(b)
    assert b["config"]["launch"] == "HIP graph replay" and "schedule" in b["config"]["lr"]
    assert b["roofline"]["kernel"] == "schedule_step_kernel + step_flat_ct + copy_out (whole step)"
    assert b["r0"]["GBps"] > 0

"""bench.py's output contract: one JSON line with the metric, the roofline
of the dominant kernel and the oracle's CPU baseline (GPU); and its refusal
of more than one GPU (CPU)."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stderr and r.stdout.strip() == ""


@pytest.mark.gpu
def test_bench_json_line():
    print("[case] bench.py on the 16.7M workload", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "flat16m_k4",
                        "--steps", "4", "--warmup", "4", "--cpu-seconds", "1", "--no-schemes", "--persist", "none"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 4 and d["warmup"] == 4 and d["value"] > 0
    assert d["config"]["workload"] == "flat16m_k4" and d["data"] == "synthetic"
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3 and "traffic" in rf
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    assert d["restore_equals_device_state"] is True
    # host time is counted over the timed steps only, so it cannot exceed
    # their wall time; the default ring plan never blocks the caller
    assert d["host_ms_in_library_per_step"]["window"] <= d["ms_per_step"]
    assert d["config"]["ring_plan"] == "device"
    assert d["stall_ms_per_step"] is not None and len(d["stall_windows_ms_per_step"]) == 3
    # each window is paired with a span of K + 1 = 5 plain steps
    assert len(d["stall_plain_spans_ms"]) == 3
    for ref in d["stall_plain_spans_ms"]:
        assert ref == pytest.approx(5 * d["plain_ms_per_step"], rel=0.2)
    assert d["stall_ms_per_checkpoint"] == pytest.approx(d["stall_ms_per_step"] * 4, abs=0.02)
    assert d["fused_dispatch_steps"].count(1) >= 1 + 1 + 3  # warmup, timed and stall windows

"""The bench's byte accounting against the per-step algorithmic bytes of the
update+pack (28 B per element, plus 12 B per element of the step's part and
2 B per gradient sent) on the two smallest workloads' real bounds (CPU)."""
import numpy as np

import bench
import synth
from paper_2511_07035_amd import GOCKPT_ALIGN_ELEMS, gockpt_plan_bounds

MiB = 1 << 20


def _bounds(name):
    wl = synth.WORKLOADS[name]
    layout = synth.LAYOUTS[wl["layout"]]()
    n = synth.numel(layout)
    align = 256 if wl["partition"] == "bytes" else GOCKPT_ALIGN_ELEMS
    return n, wl["K"], gockpt_plan_bounds(wl["K"], n, align=align)


def test_flat16m_per_step_bytes():
    n, K, b = _bounds("flat16m_k4")
    assert n == 16_777_216 and list(np.diff(b)) == [4_194_304] * 4
    per = [bench.fused_bytes(n, b, s) for s in range(1, K + 1)]
    # 28n = 448 MiB, the part 48 MiB, the gradients of s-1 parts 8 MiB each
    assert [x / MiB for x in per] == [496, 504, 512, 520]
    assert [bench.d2h_bytes(b, s) - bench.RECORD_BYTES for s in range(1, K + 1)] == [
        (48 + 8 * (s - 1)) * MiB for s in range(1, K + 1)]


def test_gpt1p3b_per_step_bytes():
    n, K, b = _bounds("gpt1p3b_k8")
    per = [bench.fused_bytes(n, b, s) for s in range(1, K + 1)]
    assert round(per[0] / 1e9, 1) == 38.7 and round(per[-1] / 1e9, 1) == 41.0
    assert all(y > x for x, y in zip(per, per[1:]))  # each step sends more gradients
    window = sum(bench.d2h_bytes(b, s) - bench.RECORD_BYTES for s in range(1, K + 1))
    assert window == 12 * n + 2 * int(b[:-1].sum())
    assert round(window / 1e9, 1) == 24.9


def test_measured_bytes_of_a_step():
    """What the kernel moved: the update's 28 B per element plus the ring
    stores; a skipped step only reads and writes what it packs."""
    assert bench.fused_bytes_measured(1000, 4096, False) == 28 * 1000 + 4096
    assert bench.fused_bytes_measured(1000, 4096, True) == 2 * 4096


def _fake_counter_run(tmp_path, n, K, alg):
    """Counter CSVs and a bench line as two rocprofv3 passes over the bench
    would leave them: 2 plain steps, then window steps 1..K, a copy probe in
    between; FETCH reads half the bytes (this device's FETCH_SIZE counts
    64-byte requests as 32), WRITE all of them."""
    import json
    order = [0, 0] + list(range(1, K + 1))
    rows_f = ["Kernel_Name,Counter_Name,Counter_Value"]
    rows_w = ["Kernel_Name,Counter_Name,Counter_Value"]
    copy = "(anonymous namespace)::copy_kernel(unsigned int __vector(4) const*, unsigned int __vector(4)*, unsigned long)"
    for _ in range(3):
        rows_f.append(f'"{copy}",FETCH_SIZE,{(4 << 30) / 1024 / 2}')
        rows_w.append(f'"{copy}",WRITE_SIZE,{(4 << 30) / 1024}')
    for s in order:
        b = 28 * n if s == 0 else alg[s]
        rd = 14 * n + (0 if s == 0 else (b - 28 * n))  # reads: g + p, m, v; the pack adds as much read as written
        wr = b - rd
        name = "void gockpt::fused_kernel<true, 1, 0, true>(gockpt::FusedArgs)"
        rows_f.append(f'"{name}",FETCH_SIZE,{rd / 1024 / 2}')
        rows_w.append(f'"{name}",WRITE_SIZE,{wr / 1024}')
    (tmp_path / "f.csv").write_text("\n".join(rows_f) + "\n")
    (tmp_path / "w.csv").write_text("\n".join(rows_w) + "\n")
    line = {"config": {"workload": "flat16m_k4", "n_elems": n, "K": K}, "fused_dispatch_steps": order,
            "window_alg_bytes": {str(s): alg[s] for s in range(1, K + 1)}}
    (tmp_path / "b.json").write_text("[bench] log line\n" + json.dumps(line) + "\n")


def test_traffic_summary_and_lookup(tmp_path):
    """The summarizer scales both counters by the copy kernel's reading,
    matches dispatches to window steps in order, and the bench's lookup
    averages the traffic of exactly the timed window steps -- and gives
    nothing once the kernel sources' hash differs."""
    import json
    n, K = 1 << 20, 4
    alg = {s: 28 * n + 12 * (n // 4) + 2 * (n // 4) * (s - 1) for s in range(1, K + 1)}
    _fake_counter_run(tmp_path, n, K, alg)
    bench.summarize_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(tmp_path / "b.json"),
                            out_dir=str(tmp_path))
    t = json.load(open(tmp_path / "fused_kernel_flat16m_k4_traffic.json"))
    assert abs(t["calibration"]["fetch_factor"] - 2.0) < 1e-12 and abs(t["calibration"]["write_factor"] - 1.0) < 1e-12
    for w in t["window_steps"]:
        assert abs(w["traffic_bytes"] - alg[w["s"]]) < 1.0 and w["algorithmic_bytes"] == alg[w["s"]]
    assert abs(t["plain_step_traffic_bytes"] - 28 * n) < 1.0
    md = (tmp_path / "fused_kernel_flat16m_k4_traffic.md").read_text()
    assert "rocprofv3 --pmc FETCH_SIZE" in md and "rocprofv3 --pmc WRITE_SIZE" in md
    got = bench.measured_traffic("flat16m_k4", [1, 2, 3, 1, 2], out_dir=str(tmp_path))
    assert got == round((alg[1] + alg[2] + alg[3] + alg[1] + alg[2]) / 5)
    assert bench.measured_traffic("flat16m_k4", [5], out_dir=str(tmp_path)) is None  # a step it never measured
    t["source_sha256"] = "0" * 64
    json.dump(t, open(tmp_path / "fused_kernel_flat16m_k4_traffic.json", "w"))
    assert bench.measured_traffic("flat16m_k4", [1], out_dir=str(tmp_path)) is None

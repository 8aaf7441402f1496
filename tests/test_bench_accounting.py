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

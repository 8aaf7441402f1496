"""The paper's headline figures recomputed from its own table (documentation
checks, CPU): they pin the reading that the abstract's percentages compare
GoCkpt-O with Async in Table crash_expr (Sec. 5.4), and that the table's
N_best follows its printed formula with one training-step time for every
scheme."""
import json
import math
import os

import pytest

FIX = os.path.join(os.path.dirname(__file__), "golden", "paper_crash_expr.json")


def _table():
    return json.load(open(FIX))


def test_abstract_percentages_are_gockpt_o_against_async():
    t = _table()
    rows, ab = t["rows"], t["abstract"]
    red = 100.0 * (1.0 - rows["GoCkpt-O"]["t_ckpt"] / rows["Async"]["t_ckpt"])
    gain = 100.0 * (rows["GoCkpt-O"]["tokens_per_s"] / rows["Async"]["tokens_per_s"] - 1.0)
    assert round(red, 1) == ab["interruption_reduction_pct"]
    assert round(gain, 1) == ab["throughput_gain_pct"]
    # against Async-O, the other plausible baseline, the figures would differ
    assert round(100.0 * (1.0 - rows["GoCkpt-O"]["t_ckpt"] / rows["Async-O"]["t_ckpt"]), 1) != ab[
        "interruption_reduction_pct"]


def test_n_best_formula_gives_one_step_time():
    """N_best = sqrt(2 T_ckpt / (p T_step^2)) with p = 1 / crash interval:
    solved for T_step, every row gives the same training step (within the
    rounding of N_best to an integer)."""
    t = _table()
    p = 1.0 / t["crash_interval_s"]
    steps = {k: math.sqrt(2.0 * r["t_ckpt"] / p) / r["n_best"] for k, r in t["rows"].items()}
    lo, hi = min(steps.values()), max(steps.values())
    assert 0.44 < lo and hi < 0.46, steps
    # the spread is what rounding the smallest N_best to an integer allows
    assert hi / lo < 1.0 + 1.0 / min(r["n_best"] for r in t["rows"].values())


@pytest.mark.parametrize("scheme", ["Async-O", "GoCkpt", "GoCkpt-O"])
def test_shorter_stalls_checkpoint_more_often_and_train_faster(scheme):
    """Monotone structure of the table: from Async on, a smaller T_ckpt gives
    a smaller N_best and a higher throughput."""
    order = ["Async", "Async-O", "GoCkpt", "GoCkpt-O"]
    rows = _table()["rows"]
    prev = rows[order[order.index(scheme) - 1]]
    cur = rows[scheme]
    assert cur["t_ckpt"] < prev["t_ckpt"] and cur["n_best"] < prev["n_best"]
    assert cur["tokens_per_s"] > prev["tokens_per_s"]

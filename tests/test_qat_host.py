"""Host-side checks of the annealing loop's schedule and drift budget."""
import json
import math
import os

import pytest

torch = pytest.importorskip("torch")
from paper_2605_10655_amd.qat import anneal_temperatures, drift_budget  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "drift_budget.json")


def test_schedule_is_eq_anneal_sampled_at_both_ends():
    T = anneal_temperatures(0.1, 1e-3, 8)
    assert len(T) == 8 and T[0] == pytest.approx(0.1) and T[-1] == pytest.approx(1e-3)
    ratios = [T[i + 1] / T[i] for i in range(7)]
    for r in ratios:  # geometric: constant ratio (T_end / T0)^(1/7)
        assert r == pytest.approx((1e-3 / 0.1) ** (1 / 7), rel=1e-12)
    assert anneal_temperatures(0.3, 0.01, 1) == [0.3]


def test_drift_budget_reproduces_the_papers_worked_numbers():
    g = json.load(open(GOLDEN))
    for run in g["runs"]:
        b = drift_budget(g["sigma_w"], g["S"], run["lr"], run["steps"], run["g_max"])
        assert b["r_voronoi"] == pytest.approx(g["r_voronoi_approx"], rel=0.01)
        assert b["max_drift"] == pytest.approx(run["max_drift_approx"], rel=1e-9)
        if "escape_possible" in run:
            assert b["escape_possible"] == run["escape_possible"]
    assert drift_budget(1.0, 4, 0.1, 1, 1.0)["r_voronoi"] == pytest.approx(1 / math.sqrt(8 * math.pi))

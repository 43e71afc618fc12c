"""Pins of the oracle's statistics against the numbers the paper prints."""
import numpy as np
import pytest

from oracle import metrics as X
from conftest import load_golden


def _r2(x):
    return float(f"{x:.2f}")


def test_efficiency_table_speedups_recomputed():
    rows = load_golden("efficiency_table.csv")
    native = {r[0]: r for r in rows if r[1] == "native"}
    for model, method, gpu, gpu_sp, o2a, o2a_sp in rows:
        n = native[model]
        assert _r2(X.speedup(float(n[2]), float(gpu))) == float(gpu_sp), (model, method)
        assert _r2(X.speedup(float(n[4]), float(o2a))) == float(o2a_sp), (model, method)


def test_ablation_text_speedups_recomputed():
    rows = {r[0]: r for r in load_golden("ablation_table.csv")}
    n = rows["native"]
    for name, gpu, o2a, sg, so in rows.values():
        if sg:
            assert _r2(X.speedup(float(n[1]), float(gpu))) == float(sg), name
            assert _r2(X.speedup(float(n[2]), float(o2a))) == float(so), name


def test_mean_per_replan_definition():
    # two episodes: foreground + anticipatory seconds over total replans
    assert X.mean_time_per_replan_ms([1.0, 2.0], [0.5, 0.5], [10, 30]) == pytest.approx(100.0)
    assert X.mean_o2a_ms([0.4, 0.4], [4, 4]) == pytest.approx(100.0)
    assert X.o2a(1.25, 1.5) == pytest.approx(0.25)


def test_reuse_rates():
    assert X.rr_rates(8, 10, 20, 100) == (0.8, 0.2)
    r, c = X.or_rates(3, 4, 6)
    assert r == 0.75 and c == 0.5


def test_similarity_and_errors():
    a = np.array([3.0, 4.0])
    assert X.cosine(a, 2 * a) == pytest.approx(1.0)
    assert X.rel_l2(a * 1.1, a) == pytest.approx(0.1)
    assert X.action_rmse(np.zeros((2, 3)), np.ones((2, 3)) * 2) == pytest.approx(2.0)
    assert X.layer_change(a * 1.5, a) == pytest.approx(0.5)
    assert X.output_error(a, a) == 0.0
    assert X.max_rel_err(np.array([1.0, -2.1]), np.array([1.0, -2.0])) == pytest.approx(0.05)

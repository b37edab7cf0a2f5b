"""Paired Student-t interval pinned by the numbers printed in Table 1 and Sec. 5.1."""
import json
import os

from oracle import stats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_p99_itl.json")


def test_table1_reductions_and_interval():
    with open(GOLDEN) as f:
        g = json.load(f)
    red = stats.paired_reductions(g["baseline_p99_itl_ms"], g["dlfp_p99_itl_ms"])
    nd = g["printed_decimals"]
    assert [round(r, nd) for r in red] == g["printed_reduction_pct"]
    mean, lo, hi = stats.student_t_ci(red)
    assert round(mean, nd) == g["printed_mean_reduction_pct"]
    assert [round(lo, nd), round(hi, nd)] == g["printed_ci95_pct"]


def test_interval_symmetry_and_degenerate_spread():
    mean, lo, hi = stats.student_t_ci([5.0, 5.0, 5.0])
    assert mean == lo == hi == 5.0
    mean, lo, hi = stats.student_t_ci([1.0, 2.0, 3.0])
    assert abs((mean - lo) - (hi - mean)) < 1e-12
    # df = 2: t_0.975 = 4.302653, sd = 1, half-width = 4.302653 / sqrt(3)
    assert abs((hi - mean) - 4.302653 / 3 ** 0.5) < 1e-5

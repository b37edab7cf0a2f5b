"""Paired trial statistics (Sec. 4.3, Table 1).

Baseline and candidate are run on the same seed; the per-seed relative
reduction is one trial-level value, and a Student-t 95% interval with
``n - 1`` degrees of freedom is reported over the trials (df = 2 for three
seeds, Sec. 4.3).
"""
from __future__ import annotations

import math
from typing import Sequence, Tuple

from scipy import stats as _st


def paired_reductions(baseline: Sequence[float], candidate: Sequence[float]):
    """Per-trial relative reduction in percent, ``100 * (b - c) / b``."""
    return [100.0 * (b - c) / b for b, c in zip(baseline, candidate)]


def student_t_ci(values: Sequence[float], confidence: float = 0.95) -> Tuple[float, float, float]:
    """(mean, low, high) of a two-sided Student-t interval with n-1 degrees of freedom."""
    n = len(values)
    mean = sum(values) / n
    var = sum((x - mean) ** 2 for x in values) / (n - 1)
    half = _st.t.ppf(0.5 + confidence / 2.0, n - 1) * math.sqrt(var / n)
    return mean, mean - half, mean + half

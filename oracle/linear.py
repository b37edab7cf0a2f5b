"""Dense projection of a layer's tokens, float64 (plain PyTorch CPU ops).

The iteration latency of Eq. 1 (Sec. 2.1) includes the layer's linear
projections, whose cost grows with the number of tokens in the batch.  A
linear layer with weight ``w[n][k]`` maps token ``x[i]`` to
``out[i][j] = sum_l x[i][l] w[j][l]``; bf16 inputs are widened exactly and
the sum is float64.  The matrix product is one library call (the definition
itself); it is pinned against pure-Python loops and closed forms.
"""
from __future__ import annotations

import numpy as np
import torch


def linear(x, w) -> np.ndarray:
    """x: float64 ``[m][k]``; w: float64 ``[n][k]``; returns float64 ``[m][n]``."""
    tx = torch.as_tensor(np.asarray(x, dtype=np.float64))
    tw = torch.as_tensor(np.asarray(w, dtype=np.float64))
    if tx.ndim != 2 or tw.ndim != 2 or tx.shape[1] != tw.shape[1]:
        raise ValueError("x is [m][k] and w is [n][k]")
    return (tx @ tw.T).numpy()

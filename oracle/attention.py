"""Masked softmax attention over logical sequences, float64 (plain PyTorch CPU ops).

Definition followed (no blocking, fusion or reordering beyond it):

In one mixed iteration (Eq. 1, Sec. 2.1) each decoding request issues one
query token and the prefill share issues ``p_t`` prompt tokens; a prompt chunk
attends causally to the prompt's already-cached prefix plus the chunk itself
(chunked prefill, Sec. 2.1).  A query row at absolute position ``j`` of its
sequence sees keys ``0 .. j``; for a sequence holding ``n`` keys of which the
last ``q`` were appended this iteration, query row ``i`` sits at ``n - q + i``
(bottom-right causal alignment).  Query head ``h`` reads KV head ``h // g``
with ``g = Hq / Hkv`` (contiguous grouped-query heads).  For each row and head

    s_j = scale * <q, k_j>            for visible j, else -inf
    w_j = exp(s_j - max_j s_j)
    o   = sum_j w_j v_j / sum_j w_j

The attention computation itself is untouched by the controller (Sec. 3.2).
bf16 inputs are widened exactly; all arithmetic is float64.  The matrix
products and the exponentials are PyTorch CPU library calls (multithreaded),
which only changes how fast the definition is evaluated, not what it is.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np
import torch


def bf16_bits_to_float64(bits) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16 numpy array) to float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def bf16_bits_to_float64_tensor(bits) -> torch.Tensor:
    """Exact widening of bf16 bit patterns (uint16 numpy array, or an int16 / uint16
    / bfloat16 CPU tensor holding them) to a float64 CPU tensor."""
    if isinstance(bits, np.ndarray):
        bits = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    if bits.dtype != torch.bfloat16:
        bits = bits.view(torch.int16).view(torch.bfloat16)
    return bits.to(torch.float64)


def _f64(x) -> torch.Tensor:
    if isinstance(x, torch.Tensor):
        return x.to(device="cpu", dtype=torch.float64)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))


def attention_rows(q, k, v, scale: float, positions) -> np.ndarray:
    """Attention output of query rows at given absolute positions of one sequence.

    q: ``[R][Hq][D]`` float64 query rows; k, v: ``[n][Hkv][D]`` float64 keys and
    values of the sequence (positions ``0 .. n-1``); positions: ``[R]`` absolute
    position of each query row, ``0 <= positions[r] < n``.  Row ``r`` sees keys
    ``0 .. positions[r]``.  Accepts numpy arrays or CPU tensors; returns float64
    numpy ``[R][Hq][D]``.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    r, hq, d = q.shape
    n, hkv, dk = k.shape
    if dk != d or tuple(v.shape) != tuple(k.shape):
        raise ValueError("q/k/v head dims disagree")
    if hq % hkv != 0:
        raise ValueError("query heads must be a multiple of KV heads")
    pos = torch.as_tensor(np.asarray(positions, dtype=np.int64))
    if tuple(pos.shape) != (r,) or (r and (int(pos.min()) < 0 or int(pos.max()) >= n)):
        raise ValueError("query positions outside the sequence")
    g = hq // hkv
    visible = torch.arange(n)[None, :] <= pos[:, None]
    # keys and values of each KV head as [n][D] matrices
    k_heads = [k[:, j, :].contiguous() for j in range(hkv)]
    v_heads = [v[:, j, :].contiguous() for j in range(hkv)]
    out = torch.empty((r, hq, d), dtype=torch.float64)
    for h in range(hq):
        kh = h // g
        s = scale * (q[:, h, :] @ k_heads[kh].T)
        s = torch.where(visible, s, -math.inf)
        m = s.max(dim=1, keepdim=True).values
        w = torch.exp(s - m)
        out[:, h, :] = (w @ v_heads[kh]) / w.sum(dim=1, keepdim=True)
    return out.numpy()


def attention_sequence(q, k, v, scale: float,
                       rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Attention output of one sequence's new tokens.

    q: float64 ``[q_len][Hq][D]`` -- the queries appended this iteration.
    k, v: float64 ``[n][Hkv][D]`` -- every key/value of the sequence, including
    the ``q_len`` appended this iteration.
    rows: optional subset of query rows (0-based within ``q``) to evaluate.
    Returns float64 ``[len(rows)][Hq][D]`` (all rows when ``rows`` is None).
    """
    q_len, n = q.shape[0], k.shape[0]
    if q_len > n:
        raise ValueError("more new queries than keys")
    pos0 = n - q_len
    row_idx = np.arange(q_len) if rows is None else np.asarray(rows, dtype=np.int64)
    return attention_rows(_f64(q)[torch.as_tensor(row_idx)], k, v, scale, pos0 + row_idx)

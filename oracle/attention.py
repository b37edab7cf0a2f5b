"""Masked softmax attention over logical sequences, float64.

Definition followed (no blocking, fusion or reordering beyond it):

In one mixed iteration (Eq. 1, Sec. 2.1) each decoding request issues one
query token and the prefill share issues ``p_t`` prompt tokens; a prompt chunk
attends causally to the prompt's already-cached prefix plus the chunk itself
(chunked prefill, Sec. 2.1).  For a sequence holding ``n`` keys of which the
last ``q`` were appended this iteration, query row ``i`` sits at absolute
position ``n - q + i`` and sees keys ``0 .. n - q + i`` (bottom-right causal
alignment).  Query head ``h`` reads KV head ``h // g`` with ``g = Hq / Hkv``
(contiguous grouped-query heads).  For each row and head

    s_j = scale * <q, k_j>            for visible j, else -inf
    w_j = exp(s_j - max_j s_j)
    o   = sum_j w_j v_j / sum_j w_j

The attention computation itself is untouched by the controller (Sec. 3.2).
bf16 inputs are widened exactly; all arithmetic is float64.
"""
from __future__ import annotations

from typing import Iterable, List, Optional, Sequence

import numpy as np


def bf16_bits_to_float64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def attention_sequence(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float,
                       rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Attention output of one sequence.

    q: float64 ``[q_len][Hq][D]`` -- the queries appended this iteration.
    k, v: float64 ``[n][Hkv][D]`` -- every key/value of the sequence, including
    the ``q_len`` appended this iteration.
    rows: optional subset of query rows (0-based within ``q``) to evaluate.
    Returns float64 ``[len(rows)][Hq][D]`` (all rows when ``rows`` is None).
    """
    q_len, hq, d = q.shape
    n, hkv, dk = k.shape
    if dk != d or v.shape != k.shape:
        raise ValueError("q/k/v head dims disagree")
    if hq % hkv != 0:
        raise ValueError("query heads must be a multiple of KV heads")
    if q_len > n:
        raise ValueError("more new queries than keys")
    g = hq // hkv
    pos0 = n - q_len
    row_idx = np.arange(q_len) if rows is None else np.asarray(rows, dtype=np.int64)
    positions = pos0 + row_idx                      # absolute position of each query row
    visible = np.arange(n)[None, :] <= positions[:, None]
    out = np.empty((len(row_idx), hq, d), dtype=np.float64)
    for h in range(hq):
        kh = h // g
        s = scale * (q[row_idx, h, :] @ k[:, kh, :].T)
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        w = np.exp(s - m)
        out[:, h, :] = (w @ v[:, kh, :]) / w.sum(axis=1, keepdims=True)
    return out


def mixed_iteration(seqs: Iterable, scale: float, rows_per_seq: Optional[List] = None
                    ) -> List[np.ndarray]:
    """Outputs of a whole mixed iteration, one array per sequence in batch order.

    ``seqs`` yields objects with ``q_bits [q_len][Hq][D]``, ``k_bits`` and
    ``v_bits [kv_len][Hkv][D]`` (uint16 bf16 bits).  Concatenating the returned
    arrays gives the packed ``[T_q][Hq][D]`` output in cumulative-query order.
    """
    outs = []
    for i, s in enumerate(seqs):
        rows = None if rows_per_seq is None else rows_per_seq[i]
        outs.append(attention_sequence(bf16_bits_to_float64(s.q_bits),
                                       bf16_bits_to_float64(s.k_bits),
                                       bf16_bits_to_float64(s.v_bits), scale, rows))
    return outs

"""Gather twin: read a sequence's keys and values back out of the paged pool.

PagedAttention keeps the KV cache in fixed-size pages addressed through a
per-sequence block table (Sec. 2.1; the KV layout the controller leaves
unchanged, Sec. 3.2).  The pool layout gathered here is the one the library
declares for its caches (16-token pages, head_dim 128, bf16):

* key pages   ``k_cache[block][kv_head][slot][dim]``  (token rows)
* value pages ``v_cache[block][kv_head][dim][pi(slot)]``  (transposed page;
  ``pi`` swaps bits 2 and 3 of the slot, i.e. slots 4-7 trade places with 8-11)

Token ``j`` of sequence ``s`` lives in block ``block_table[s][j // 16]`` at slot
``j % 16``.  Plain loops, one token at a time.
"""
from __future__ import annotations

import numpy as np

PAGE = 16


def value_position(slot: int) -> int:
    """Position of token slot ``slot`` inside a value page row (bits 2 and 3 swap)."""
    b2, b3 = (slot >> 2) & 1, (slot >> 3) & 1
    return (slot & 3) | (b2 << 3) | (b3 << 2)


def gather_sequence(k_cache: np.ndarray, v_cache: np.ndarray, block_row: np.ndarray,
                    n_tokens: int):
    """Return (K, V) uint16 ``[n_tokens][Hkv][D]`` for one sequence."""
    num_blocks, hkv, page, d = k_cache.shape
    if page != PAGE or v_cache.shape != (num_blocks, hkv, d, page):
        raise ValueError("unexpected pool layout")
    k = np.empty((n_tokens, hkv, d), dtype=np.uint16)
    v = np.empty((n_tokens, hkv, d), dtype=np.uint16)
    for j in range(n_tokens):
        block = int(block_row[j // PAGE])
        slot = j % PAGE
        k[j] = k_cache[block, :, slot, :]
        v[j] = v_cache[block, :, :, value_position(slot)]
    return k, v


def gather_slots(cache_k: np.ndarray, cache_v: np.ndarray, slots: np.ndarray):
    """Return (K, V) rows stored at flat slots (``block * 16 + offset``)."""
    n = len(slots)
    _, hkv, _, d = cache_k.shape
    k = np.empty((n, hkv, d), dtype=np.uint16)
    v = np.empty((n, hkv, d), dtype=np.uint16)
    for i, slot in enumerate(slots):
        block, off = int(slot) // PAGE, int(slot) % PAGE
        k[i] = cache_k[block, :, off, :]
        v[i] = cache_v[block, :, :, value_position(off)]
    return k, v

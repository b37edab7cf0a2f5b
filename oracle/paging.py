"""Gather twin: read a sequence's keys and values back out of the paged pool.

PagedAttention keeps the KV cache in fixed-size pages addressed through a
per-sequence block table (Sec. 2.1; the KV layout the controller leaves
unchanged, Sec. 3.2).  The pool layout gathered here is the one the library
declares for its caches (16-token pages, head_dim 128, bf16):

* key pages   ``k_cache[block][kv_head][slot][dim]``  (token rows)
* value pages ``v_cache[block][kv_head][dim][pi(slot)]``  (transposed page;
  ``pi`` swaps bits 2 and 3 of the slot, i.e. slots 4-7 trade places with 8-11)

Token ``j`` of sequence ``s`` lives in block ``block_table[s][j // 16]`` at slot
``j % 16``.  ``gather_sequence`` is the plain loop, one token at a time;
``gather_pages`` reads the same entries with whole-page array indexing (for
sequences of tens of thousands of tokens) and is checked against the loop.
"""
from __future__ import annotations

import numpy as np
import torch

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


def gather_pages(k_cache, v_cache, block_row, n_tokens: int):
    """``gather_sequence`` by whole pages: returns (K, V) ``[n_tokens][Hkv][D]``.

    Accepts numpy uint16 pools (returns numpy uint16) or CPU tensors of 16-bit
    elements (returns tensors of the same dtype).
    """
    as_numpy = isinstance(k_cache, np.ndarray)
    kc = torch.from_numpy(k_cache.view(np.int16)) if as_numpy else k_cache
    vc = torch.from_numpy(v_cache.view(np.int16)) if as_numpy else v_cache
    num_blocks, hkv, page, d = kc.shape
    if page != PAGE or tuple(vc.shape) != (num_blocks, hkv, d, page):
        raise ValueError("unexpected pool layout")
    n_pages = (int(n_tokens) + PAGE - 1) // PAGE
    blocks = torch.as_tensor(np.asarray(block_row[:n_pages], dtype=np.int64))
    if n_pages and (int(blocks.min()) < 0 or int(blocks.max()) >= num_blocks):
        raise ValueError("block id outside the pool")
    # key page [hkv][slot][dim] -> token rows [slot][hkv][dim]
    k = kc.index_select(0, blocks).permute(0, 2, 1, 3).reshape(n_pages * PAGE, hkv, d)
    # value page [hkv][dim][pi(slot)] -> [slot][hkv][dim]
    perm = torch.tensor([value_position(t) for t in range(PAGE)], dtype=torch.int64)
    v = vc.index_select(0, blocks).index_select(3, perm).permute(0, 3, 1, 2)
    v = v.reshape(n_pages * PAGE, hkv, d)
    k, v = k[:n_tokens].contiguous(), v[:n_tokens].contiguous()
    if as_numpy:
        return k.numpy().view(np.uint16), v.numpy().view(np.uint16)
    return k, v

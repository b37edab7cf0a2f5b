"""Varlen-metadata twin and work-list checker.

A mixed iteration packs the decoders' single query tokens and the prefill
chunk's ``p_t`` tokens into one batch (``D_t`` and ``p_t`` of Eq. 1, Sec. 2.1).
Its metadata has exactly one correct value, written out here with plain loops:

* ``cu_q[s]``        exclusive prefix sum of the per-sequence query counts;
* ``q_pos0[s]``      absolute position of sequence ``s``'s first new token,
                     ``kv_len[s] - q_len[s]``;
* ``slot_mapping``   for every new token, in packed order, the flat pool slot
                     ``block_table[s][pos // 16] * 16 + pos % 16`` it is written
                     to (PagedAttention block addressing, Sec. 2.1).

The work list (how the attention launch splits the iteration into units) has
many valid values, so it is not recomputed; ``check_work_list`` verifies the
properties any valid list must have, and ``check_append_records`` those of the
records that tell a one-launch append which new tokens to write (each prompt
token of each KV head exactly once, in runs that stay inside one page).

What the method fixes and what the library's format fixes.  The clause that
follows from the definition of the iteration (Eq. 1, Sec. 2.1) is coverage:
every visible (query token, key) pair of every (sequence, KV head) belongs to
exactly one unit, and the units of one set of rows combine in split order.
The other clauses check the work-list and workspace format that the library
declares in its header (``include/dlfp.h``): 128 query rows per prefill unit,
a 256-byte workspace header, a fixed region of 65536 split counters, partial
slots of ``rows x 130`` floats padded to 256 bytes, page-aligned key ranges,
prefill units first and the derived row/position fields.  They guard the
launch against a malformed list; the paper says nothing about them.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

PAGE = 16
HEAD_DIM = 128
TILE_ROWS = 128          # query rows (tokens x grouped heads) one prefill unit holds
WS_HEADER = 256          # workspace bytes before the split counters
WS_MAX_GROUPS = 65536    # fixed counter region: one int32 per possible group

# Work-item field indices (16 int32 per unit).
W_SEQ, W_KVHEAD, W_QTOK0, W_QNTOK, W_KVBEGIN, W_KVEND = 0, 1, 2, 3, 4, 5
W_GROUP, W_SPLIT, W_NSPLITS, W_WSOFF, W_WSGROUP, W_KIND = 6, 7, 8, 9, 10, 11
W_QROW0, W_QPOS0 = 12, 13   # derived: cu_q[seq] + first token, q_pos0[seq] + first token
WORK_INTS = 16
KIND_PREFILL, KIND_DECODE, KIND_APPEND = 0, 1, 2


def varlen_meta(q_len: Sequence[int], kv_len: Sequence[int], block_table: np.ndarray
                ) -> Tuple[List[int], List[int], List[int]]:
    """Return (cu_q, q_pos0, slot_mapping) as Python int lists."""
    cu_q = [0]
    q_pos0 = []
    slots = []
    for s in range(len(q_len)):
        cu_q.append(cu_q[-1] + int(q_len[s]))
        first = int(kv_len[s]) - int(q_len[s])
        q_pos0.append(first)
        for pos in range(first, int(kv_len[s])):
            block = int(block_table[s][pos // PAGE])
            slots.append(block * PAGE + pos % PAGE)
    return cu_q, q_pos0, slots


class WorkListError(AssertionError):
    pass


def check_work_list(work: np.ndarray, num_prefill: int, q_len: Sequence[int],
                    kv_len: Sequence[int], num_q_heads: int, num_kv_heads: int,
                    num_groups: int, workspace_bytes: int) -> Dict[str, int]:
    """Raise ``WorkListError`` unless ``work`` is a valid unit list for the iteration.

    Validity: every visible (query token, key) pair of every (sequence, KV head)
    is covered by exactly one unit; units respect sequence bounds and page
    alignment; prefill units precede decode units; a unit is a decode unit iff
    its sequence has a single new token; split groups are complete and ordered;
    partial-result slots are disjoint and inside the workspace; the derived
    row and position fields equal their definitions.
    """
    def fail(msg):
        raise WorkListError(msg)

    g = num_q_heads // num_kv_heads
    n_seq = len(q_len)
    work = np.asarray(work, dtype=np.int64).reshape(-1, WORK_INTS)
    counts = {}
    groups: Dict[int, List[np.ndarray]] = {}
    # workspace: header, the fixed counter region, then partial slots
    if num_groups > WS_MAX_GROUPS:
        fail("more groups than counters")
    partial_base = (WS_HEADER + 4 * WS_MAX_GROUPS) // 4
    slots = []
    cu_q = np.concatenate([[0], np.cumsum(np.asarray(q_len, dtype=np.int64))])
    for u, it in enumerate(work):
        s, kh, t0, nt, kb, ke = (int(x) for x in it[:6])
        grp, split, nsp, wsoff, wsgrp, kind = (int(x) for x in it[6:12])
        if not (0 <= s < n_seq and 0 <= kh < num_kv_heads):
            fail(f"unit {u}: bad seq/head")
        ql, kl = int(q_len[s]), int(kv_len[s])
        pos0 = kl - ql
        if not (0 <= t0 and nt >= 1 and t0 + nt <= ql):
            fail(f"unit {u}: query rows out of range")
        if not (0 <= kb < ke <= kl) or kb % PAGE:
            fail(f"unit {u}: key range [{kb},{ke}) invalid for kv_len {kl}")
        if ke > pos0 + t0 + nt:
            fail(f"unit {u}: keys beyond the last row's position")
        if int(it[W_QROW0]) != int(cu_q[s]) + t0 or int(it[W_QPOS0]) != pos0 + t0:
            fail(f"unit {u}: derived row/position fields")
        want_kind = KIND_DECODE if ql == 1 else KIND_PREFILL
        if kind != want_kind:
            fail(f"unit {u}: kind {kind} but q_len {ql}")
        if (kind == KIND_PREFILL) != (u < num_prefill):
            fail(f"unit {u}: prefill units must come first")
        if kind == KIND_PREFILL and nt * g > TILE_ROWS:
            fail(f"unit {u}: {nt}x{g} rows exceed a tile")
        # at least one visible pair: first key visible to the last row
        if kb > pos0 + t0 + nt - 1:
            fail(f"unit {u}: no visible key")
        key = (s, kh)
        if key not in counts:
            counts[key] = np.zeros((ql, kl), dtype=np.int32)
        counts[key][t0:t0 + nt, kb:ke] += 1
        if nsp < 1 or not (0 <= split < nsp):
            fail(f"unit {u}: bad split {split}/{nsp}")
        if nsp == 1:
            if grp != -1:
                fail(f"unit {u}: single split must have group -1")
        else:
            if not (0 <= grp < num_groups):
                fail(f"unit {u}: group {grp} out of range")
            groups.setdefault(grp, []).append(it)
            rows = nt * g
            slot_floats = (rows * (HEAD_DIM + 2) + 63) // 64 * 64   # padded to 256 bytes
            if wsoff != wsgrp + split * slot_floats:
                fail(f"unit {u}: partial slot offset")
            if wsgrp < partial_base:
                fail(f"unit {u}: partial slot overlaps counters")
            slots.append((wsoff, wsoff + slot_floats))
    for (s, kh), c in counts.items():
        ql, kl = int(q_len[s]), int(kv_len[s])
        pos0 = kl - ql
        vis = np.arange(kl)[None, :] <= (pos0 + np.arange(ql))[:, None]
        if np.any(c[vis] != 1):
            fail(f"seq {s} head {kh}: visible pairs not covered exactly once")
    for s in range(n_seq):
        for kh in range(num_kv_heads):
            if (s, kh) not in counts and int(q_len[s]) > 0:
                fail(f"seq {s} head {kh}: no unit")
    for grp, its in groups.items():
        nsp = int(its[0][W_NSPLITS])
        if len(its) != nsp:
            fail(f"group {grp}: {len(its)} units for {nsp} splits")
        ref = its[0]
        for it in its:
            if any(int(it[f]) != int(ref[f]) for f in (W_SEQ, W_KVHEAD, W_QTOK0, W_QNTOK,
                                                     W_NSPLITS, W_WSGROUP)):
                fail(f"group {grp}: units disagree on rows")
        by_split = sorted(its, key=lambda it: int(it[W_SPLIT]))
        if [int(it[W_SPLIT]) for it in by_split] != list(range(nsp)):
            fail(f"group {grp}: split indices")
        for a, b in zip(by_split, by_split[1:]):
            if int(a[W_KVEND]) != int(b[W_KVBEGIN]):
                fail(f"group {grp}: split ranges not contiguous and ordered")
    slots.sort()
    for (a0, a1), (b0, b1) in zip(slots, slots[1:]):
        if b0 < a1:
            fail("partial slots overlap")
    if slots and slots[-1][1] * 4 > workspace_bytes:
        fail("partial slots exceed the workspace")
    if WS_HEADER + 4 * WS_MAX_GROUPS > workspace_bytes:
        fail("header and counters exceed the workspace")
    return {"units": len(work), "groups": len(groups)}


def check_append_records(records: np.ndarray, work: np.ndarray, num_prefill: int,
                         q_len: Sequence[int], kv_len: Sequence[int], num_kv_heads: int,
                         num_waiting: int) -> Dict[str, int]:
    """Raise ``WorkListError`` unless ``records`` are valid append records.

    Validity: every new token of every prompt sequence (q_len > 1) is covered,
    per KV head, by exactly one record, and no decoder token is; a record's
    tokens are consecutive and lie in one page; its derived row and position
    fields equal their definitions.  ``num_waiting`` must be the number of
    prefill units whose last key lies in a page at or after the page of their
    sequence's first new token (the units that read a page holding a new token).
    """
    def fail(msg):
        raise WorkListError(msg)

    n_seq = len(q_len)
    records = np.asarray(records, dtype=np.int64).reshape(-1, WORK_INTS)
    cu_q = np.concatenate([[0], np.cumsum(np.asarray(q_len, dtype=np.int64))])
    cover = {}
    for r, it in enumerate(records):
        s, kh, t0, nt = (int(x) for x in it[:4])
        if int(it[W_KIND]) != KIND_APPEND:
            fail(f"record {r}: kind {int(it[W_KIND])}")
        if not (0 <= s < n_seq and 0 <= kh < num_kv_heads):
            fail(f"record {r}: bad seq/head")
        ql, kl = int(q_len[s]), int(kv_len[s])
        if ql == 1:
            fail(f"record {r}: decoder token (decode units write their own)")
        pos0 = kl - ql
        if not (0 <= t0 and 1 <= nt <= PAGE and t0 + nt <= ql):
            fail(f"record {r}: tokens out of range")
        if (pos0 + t0) // PAGE != (pos0 + t0 + nt - 1) // PAGE:
            fail(f"record {r}: run crosses a page")
        if int(it[W_QROW0]) != int(cu_q[s]) + t0 or int(it[W_QPOS0]) != pos0 + t0:
            fail(f"record {r}: derived row/position fields")
        c = cover.setdefault((s, kh), np.zeros(ql, dtype=np.int32))
        c[t0:t0 + nt] += 1
    for s in range(n_seq):
        if int(q_len[s]) == 1:
            continue
        for kh in range(num_kv_heads):
            c = cover.get((s, kh))
            if c is None or np.any(c != 1):
                fail(f"seq {s} head {kh}: new tokens not covered exactly once")
    work = np.asarray(work, dtype=np.int64).reshape(-1, WORK_INTS)
    waiting = 0
    for it in work[:num_prefill]:
        pos0 = int(it[W_QPOS0]) - int(it[W_QTOK0])
        if (int(it[W_KVEND]) - 1) // PAGE >= pos0 // PAGE:
            waiting += 1
    if waiting != num_waiting:
        fail(f"{num_waiting} waiting units reported, {waiting} read a page with a new token")
    return {"records": len(records), "waiting": waiting}

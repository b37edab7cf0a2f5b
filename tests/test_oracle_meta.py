"""Metadata twin pinned by a hand-worked example and invariants; work-list checker pinned
by hand-built valid lists and planted defects."""
import numpy as np
import pytest

from oracle import meta as om
from paper_2609_38386_amd import workload as wl


def test_hand_example():
    # prompt chunk of 128 at offset 384, and two decoders with contexts 70 and 65
    q_len = [128, 1, 1]
    kv_len = [512, 70, 65]
    bt = np.full((3, 32), -1, dtype=np.int32)
    bt[0, :32] = np.arange(100, 132)
    bt[1, :5] = [7, 3, 9, 1, 40]
    bt[2, :5] = [2, 5, 6, 8, 11]
    cu_q, q_pos0, slots = om.varlen_meta(q_len, kv_len, bt)
    assert cu_q == [0, 128, 129, 130]
    assert q_pos0 == [384, 69, 64]
    assert len(slots) == 130
    assert slots[0] == 124 * 16 + 0          # position 384 -> page 24 -> block 124, slot 0
    assert slots[127] == 131 * 16 + 15       # position 511 -> page 31 -> block 131, slot 15
    assert slots[128] == 40 * 16 + 5         # decoder 1, position 69 -> page 4, slot 5
    assert slots[129] == 11 * 16 + 0         # decoder 2, position 64 -> page 4, slot 0


def test_slots_unique_and_owned():
    cfg = wl.tiny_config()
    pages = cfg.pages_per_seq()
    bt = wl.block_tables(cfg.seed, pages, cfg.pool_size())
    ctx = cfg.decoder_contexts()
    q_len = [1] * cfg.n_decoders + [128]
    kv_len = [int(c) for c in ctx] + [512]
    cu_q, q_pos0, slots = om.varlen_meta(q_len, kv_len, bt)
    assert len(set(slots)) == len(slots)
    for s in range(len(q_len)):
        for t in range(cu_q[s], cu_q[s + 1]):
            pos = q_pos0[s] + (t - cu_q[s])
            assert slots[t] // 16 == bt[s][pos // 16]
            assert slots[t] % 16 == pos % 16


# the hand-built list below: q_len [70, 1], kv_len [100, 40]
_CU_Q, _POS0 = [0, 70], [30, 39]


def _unit(seq, kh, t0, nt, kb, ke, grp=-1, split=0, nsp=1, wsoff=0, wsgrp=0, kind=0):
    u = np.zeros(om.WORK_INTS, dtype=np.int32)
    u[:14] = [seq, kh, t0, nt, kb, ke, grp, split, nsp, wsoff, wsgrp, kind,
              _CU_Q[seq] + t0, _POS0[seq] + t0]
    return u


def _valid_list():
    """seq 0: prompt chunk of 70 tokens at offset 30 (kv 100), g=2 -> 64 tokens per tile;
    seq 1: decoder with kv 40 split into [0,32) and [32,40).  One KV head."""
    g, rows_t = 2, 64
    slot = lambda rows: (rows * (128 + 2) + 63) // 64 * 64
    base = (256 + 4 * 65536) // 4  # header + fixed counter region, in floats
    units = [
        _unit(0, 0, 0, 64, 0, 48, grp=0, split=0, nsp=2, wsoff=base, wsgrp=base),
        _unit(0, 0, 0, 64, 48, 94, grp=0, split=1, nsp=2, wsoff=base + slot(128), wsgrp=base),
        _unit(0, 0, 64, 6, 0, 100),
    ]
    dbase = base + 2 * slot(128)
    units += [
        _unit(1, 0, 0, 1, 0, 32, grp=1, split=0, nsp=2, wsoff=dbase, wsgrp=dbase, kind=1),
        _unit(1, 0, 0, 1, 32, 40, grp=1, split=1, nsp=2, wsoff=dbase + slot(2), wsgrp=dbase,
              kind=1),
    ]
    ws = (dbase + 2 * slot(2)) * 4
    return np.stack(units), 3, [70, 1], [100, 40], 2, 1, 2, ws


def test_checker_accepts_valid_list():
    work, npre, ql, kl, hq, hkv, ng, ws = _valid_list()
    om.check_work_list(work, npre, ql, kl, hq, hkv, ng, ws)


@pytest.mark.parametrize("defect", ["drop", "overlap", "order", "kind", "gap", "slot",
                                    "rows", "beyond", "align", "splitidx", "ws", "qrow",
                                    "qpos"])
def test_checker_rejects_planted_defects(defect):
    work, npre, ql, kl, hq, hkv, ng, ws = _valid_list()
    work = work.copy()
    if defect == "drop":
        work = np.delete(work, 2, axis=0)
        npre = 2
    elif defect == "overlap":
        work[1, om.W_KVBEGIN] = 32
    elif defect == "order":
        work = work[[0, 3, 1, 2, 4]]
    elif defect == "kind":
        work[2, om.W_KIND] = 1
    elif defect == "gap":
        work[3, om.W_KVEND] = 16
    elif defect == "slot":
        work[4, om.W_WSOFF] = work[3, om.W_WSOFF]
    elif defect == "rows":
        work[2, om.W_QNTOK] = 7
    elif defect == "beyond":
        work[2, om.W_KVEND] = 101
    elif defect == "align":
        work[1, om.W_KVBEGIN] = 40
        work[0, om.W_KVEND] = 40
    elif defect == "splitidx":
        work[1, om.W_SPLIT] = 0
    elif defect == "ws":
        ws = 100
    elif defect == "qrow":
        work[2, om.W_QROW0] += 1
    elif defect == "qpos":
        work[3, om.W_QPOS0] -= 1
    with pytest.raises(om.WorkListError):
        om.check_work_list(work, npre, ql, kl, hq, hkv, ng, ws)


def _append_records():
    """Append records of the hand-built batch: seq 0's new tokens (positions
    30..99) cut at page boundaries, one KV head; the decoder has none."""
    runs = [(30, 2), (32, 16), (48, 16), (64, 16), (80, 16), (96, 4)]
    recs = []
    for pos, n in runs:
        t0 = pos - _POS0[0]
        r = _unit(0, 0, t0, n, pos, pos + n, kind=om.KIND_APPEND)
        recs.append(r)
    return np.stack(recs)


def test_append_checker_accepts_valid_records():
    work, npre, ql, kl, hq, hkv, ng, ws = _valid_list()
    # every prefill unit's last key lies in page 1 or later (the first new token's page)
    assert om.check_append_records(_append_records(), work, npre, ql, kl, hkv, 3) == {
        "records": 6, "waiting": 3}


@pytest.mark.parametrize("defect", ["drop", "dup", "cross", "decoder", "kind", "qrow",
                                    "waiting"])
def test_append_checker_rejects_planted_defects(defect):
    work, npre, ql, kl, hq, hkv, ng, ws = _valid_list()
    recs = _append_records()
    waiting = 3
    if defect == "drop":
        recs = recs[1:]
    elif defect == "dup":
        recs = np.concatenate([recs, recs[2:3]])
    elif defect == "cross":          # tokens 30..33 span pages 1 and 2
        recs[0, om.W_QNTOK] = 4
        recs[1, om.W_QTOK0] += 2
        recs[1, om.W_QNTOK] -= 2
        recs[1, om.W_QROW0] += 2
        recs[1, om.W_QPOS0] += 2
    elif defect == "decoder":
        recs = np.concatenate([recs, _unit(1, 0, 0, 1, 39, 40, kind=om.KIND_APPEND)[None]])
    elif defect == "kind":
        recs[3, om.W_KIND] = om.KIND_PREFILL
    elif defect == "qrow":
        recs[4, om.W_QROW0] += 1
    elif defect == "waiting":
        waiting = 2
    with pytest.raises(om.WorkListError):
        om.check_append_records(recs, work, npre, ql, kl, hkv, waiting)

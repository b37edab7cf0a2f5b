"""Host half of the C ABI (no GPU needed): exports, metadata, work list, controller, errors."""
import json
import math
import os
import re

import numpy as np
import pytest

import _random_mixes as rm
from oracle import controller as oc
from oracle import meta as om
from paper_2609_38386_amd import dlfp as D
from paper_2609_38386_amd import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    txt = open(os.path.join(ROOT, "include", "dlfp.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(?:int|const char\*)\s+(dlfp_\w+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    L = D.lib()
    declared = _declared_functions()
    assert len(declared) >= 14
    for name in declared:
        assert hasattr(L, name), name
    assert set(declared) == set(D.EXPORTS)
    assert L.dlfp_version() == 100
    assert L.dlfp_status_string(-3) == b"capacity or workspace too small"


def _check_against_twin(dims, q_len, kv_len, bt, num_blocks, tuning=None):
    meta = D.dlfp_build_varlen_meta(dims, q_len, kv_len, bt, num_blocks, tuning)
    cu_q, q_pos0, slots = om.varlen_meta(q_len, kv_len, bt)
    n = len(q_len)
    assert meta.num_seqs == n and meta.num_tokens == cu_q[-1]
    assert meta.cu_q[:n + 1].tolist() == cu_q
    assert meta.q_pos0[:n].tolist() == q_pos0
    assert meta.slot_mapping[:meta.num_tokens].tolist() == slots
    om.check_work_list(meta.work, meta.num_prefill_units, q_len, kv_len, dims.num_q_heads,
                       dims.num_kv_heads, meta.num_groups, meta.workspace_bytes)
    om.check_append_records(meta.append_records, meta.work, meta.num_prefill_units, q_len,
                            kv_len, dims.num_kv_heads, meta.num_waiting_units)
    # decode units carry the block ids of their first two pages
    bt = np.asarray(bt)
    for u in meta.work[meta.num_prefill_units:]:
        s, kb, ke = int(u[0]), int(u[4]), int(u[5])
        pg = kb // 16
        assert u[14] == bt[s][pg]
        assert u[15] == (bt[s][pg + 1] if (ke - 1) // 16 >= pg + 1 else -1)
    return meta


def test_meta_tiny_iteration():
    cfg = wl.tiny_config()
    bt = wl.block_tables(cfg.seed, cfg.pages_per_seq(), cfg.pool_size())
    ctx = cfg.decoder_contexts()
    # block table rows: decoders first, then the prompt; batch order prompt first
    q_len = [128] + [1] * 4
    kv_len = [512] + [int(c) for c in ctx]
    rows = np.concatenate([bt[4:5], bt[:4]])
    dims = D.make_dims(16, 8)
    _check_against_twin(dims, q_len, kv_len, rows, cfg.pool_size())
    for tn in [D.dlfp_tuning(16, 64, 0), D.dlfp_tuning(32, 128, 0), D.dlfp_tuning(0, 0, 64),
               D.dlfp_tuning(0, 64, 0, 8)]:
        meta = _check_against_twin(dims, q_len, kv_len, rows, cfg.pool_size(), tn)
        if tn.decode_split_tokens == 16:
            assert meta.num_groups > 0
        if tn.prefill_tile_tokens == 8:   # 128 prompt tokens in tiles of 8, per KV head
            pre = meta.work[:meta.num_prefill_units]
            assert (pre[:, 3] <= 8).all() and len(np.unique(pre[:, 2])) == 16


@pytest.mark.parametrize("p,chunk", [(64, 0), (256, 17), (2048, 3)])
def test_meta_qwen3_0_6b_iterations(p, chunk):
    cfg = wl.qwen3_0_6b_config()
    bt = wl.block_tables(cfg.seed, cfg.pages_per_seq(), cfg.pool_size())
    its = cfg.iteration(p, chunk)
    q_len = [q for _, q, _ in its]
    kv_len = [k for _, _, k in its]
    rows = bt[[s for s, _, _ in its]]
    _check_against_twin(D.make_dims(16, 8), q_len, kv_len, rows, cfg.pool_size())


@pytest.mark.parametrize("seed", range(6))
def test_meta_random_mixes(seed):
    rng = np.random.default_rng(seed)
    g = [1, 2, 4, 8][seed % 4]
    hkv = int(rng.integers(1, 4))
    n = int(rng.integers(1, 7))
    q_len, kv_len = [], []
    for _ in range(n):
        if rng.random() < 0.5:
            q_len.append(1)
            kv_len.append(int(rng.integers(1, 300)))
        else:
            q = int(rng.integers(2, 200))
            q_len.append(q)
            kv_len.append(q + int(rng.integers(0, 300)))
    pages = [wl.pages_for(k) for k in kv_len]
    pool = sum(pages) + 5
    bt = wl.block_tables(seed, pages, pool, max_blocks=max(pages) + 2)
    tn = D.dlfp_tuning(int(rng.choice([0, 16, 48, 128])), int(rng.choice([0, 64, 192])), 0,
                       int(rng.integers(0, 128 // g + 1)))
    _check_against_twin(D.make_dims(g * hkv, hkv), q_len, kv_len, bt, pool, tn)


@pytest.mark.parametrize("i", range(rm.CASES))
def test_meta_of_the_random_gpu_mixes(i):
    """The random mixes the GPU parity test launches: the library's metadata equals
    the twin's, so every case's work list covers exactly the visible pairs before
    any of them runs on a device."""
    g, hkv, specs, tn, _, _ = rm.case(i)
    q_len, kv_len = [q for q, _ in specs], [k for _, k in specs]
    pages = [wl.pages_for(k) for k in kv_len]
    bt = wl.block_tables(rm.seed(i), pages, rm.pool(pages))
    _check_against_twin(D.make_dims(g * hkv, hkv), q_len, kv_len, bt, rm.pool(pages),
                        D.dlfp_tuning(*tn))


def test_meta_small_prefill_share_takes_latency_tiles():
    # a 32-token chunk over a 3000-token prefix next to one decoder (g = 2):
    # too few units at full tiles, so 16-token tiles and 256-key splits
    dims = D.make_dims(16, 8)
    q_len, kv_len = [32, 1], [3032, 2000]
    bt = np.arange(2 * 190, dtype=np.int32).reshape(2, 190)
    meta = _check_against_twin(dims, q_len, kv_len, bt, 2 * 190)
    pre = meta.work[:meta.num_prefill_units]
    assert meta.prefill_split_tokens == 256
    assert pre[:, 3].max() == 16 and len(pre) == 2 * 8 * 12
    # a 2048-token chunk fills the device at full tiles: throughput policy
    cfg = wl.qwen3_0_6b_config()
    bt6 = wl.block_tables(cfg.seed, cfg.pages_per_seq(), cfg.pool_size())
    its = cfg.iteration(2048, 3)
    meta = _check_against_twin(dims, [q for _, q, _ in its], [k for _, _, k in its],
                               bt6[[x for x, _, _ in its]], cfg.pool_size())
    assert meta.prefill_split_tokens >= 1024
    assert meta.work[:meta.num_prefill_units, 3].max() == 64


def test_meta_decode_tail_pieces_in_a_few_queue_rounds():
    # Qwen3-8B decoders alone (32 query / 8 KV heads): several queue rounds of
    # decode units, so each (sequence, KV head) range ends in a half and two
    # quarters of its last split part
    cfg = wl.qwen3_8b_config()
    pages = cfg.pages_per_seq()
    bt = wl.block_tables(cfg.seed, pages, int(sum(pages)))[:cfg.n_decoders]
    kv = [int(c) for c in cfg.decoder_contexts()]
    dims = D.make_dims(cfg.shape.num_q_heads, cfg.shape.num_kv_heads)
    meta = _check_against_twin(dims, [1] * len(kv), kv, bt, int(sum(pages)))
    split = meta.decode_split_tokens
    plain = sum(cfg.shape.num_kv_heads * math.ceil(k / split) for k in kv)
    assert meta.num_units > plain
    w = meta.work
    for s in range(3):
        rows = w[(w[:, 0] == s) & (w[:, 1] == 0)]
        rows = rows[np.argsort(rows[:, 4])]
        lens = rows[:, 5] - rows[:, 4]
        last = lens[-3:].sum()
        if last >= 64:
            assert lens[-3] >= lens[-2] >= lens[-1] and lens[-3] >= last // 2, lens
        assert (rows[:-3, 5] - rows[:-3, 4] == (rows[0, 5] - rows[0, 4])).all()


def test_meta_empty_batch():
    meta = D.dlfp_build_varlen_meta(D.make_dims(16, 8), [], [], np.zeros((0, 1), np.int32), 4)
    assert meta.num_seqs == 0 and meta.num_units == 0 and meta.workspace_bytes >= 256


def test_meta_errors():
    dims = D.make_dims(16, 8)
    bt = np.array([[0, 1, 2]], dtype=np.int32)
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_build_varlen_meta(dims, [0], [5], bt, 4)
    assert e.value.status == -1
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_build_varlen_meta(dims, [6], [5], bt, 4)
    assert e.value.status == -1
    with pytest.raises(D.DlfpError) as e:           # page 2 needs block 2, pool has 2 blocks
        D.dlfp_build_varlen_meta(dims, [1], [40], bt, 2)
    assert e.value.status == -2
    with pytest.raises(D.DlfpError) as e:           # 49 keys need 4 pages, table has 3
        D.dlfp_build_varlen_meta(dims, [1], [49], bt, 4)
    assert e.value.status == -2
    for bad in (D.make_dims(16, 8, head_dim=64), D.make_dims(16, 8, page_size=32),
                D.make_dims(12, 8), D.make_dims(128, 8)):
        with pytest.raises(D.DlfpError) as e:
            D.dlfp_build_varlen_meta(bad, [1], [5], bt, 4)
        assert e.value.status == -5
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_build_varlen_meta(dims, [1], [5], bt, 4, D.dlfp_tuning(10, 0, 0))
    assert e.value.status == -1
    with pytest.raises(D.DlfpError) as e:           # g = 2: at most 64 tokens per tile
        D.dlfp_build_varlen_meta(dims, [1], [5], bt, 4, D.dlfp_tuning(0, 0, 0, 65))
    assert e.value.status == -1


def test_controller_worked_example_and_twin_agreement():
    with open(os.path.join(ROOT, "tests", "golden", "controller_observability.json")) as f:
        g = json.load(f)
    c = D.dlfp_controller_init(g["target_ms"], g["c_initial"], g["c_min"], g["c_max"],
                               g["quantum"])
    assert D.dlfp_controller_step(c, 3, True, g["observed_ms"]) == g["cap_after"]
    rng = np.random.default_rng(5)
    for trial in range(40):
        params = dict(target_ms=float(rng.uniform(5, 120)), c_initial=3072,
                      c_min=int(rng.choice([32, 128, 1024])), c_max=int(rng.choice([4096, 6144])),
                      quantum=128)
        cc = D.dlfp_controller_init(params["target_ms"], params["c_initial"], params["c_min"],
                                    params["c_max"], params["quantum"])
        twin = oc.Controller(params["target_ms"], params["c_initial"], params["c_min"],
                             params["c_max"], params["quantum"])
        for _ in range(50):
            ndec = int(rng.integers(0, 4))
            guarded = bool(rng.random() < 0.7)
            obs = float(rng.lognormal(math.log(params["target_ms"]), 0.8))
            assert D.dlfp_controller_step(cc, ndec, guarded, obs) == twin.step(ndec, guarded, obs)
            assert cc.cap == twin.cap


def test_controller_rejects_bad_observation_without_state_change():
    c = D.dlfp_controller_init(80.0, 3072, 1024, 6144)
    for bad in (0.0, -3.0, float("nan"), float("inf")):
        with pytest.raises(D.DlfpError) as e:
            D.dlfp_controller_step(c, 2, True, bad)
        assert e.value.status == -1
        assert c.cap == 3072
    # an unguarded step ignores the observation entirely
    assert D.dlfp_controller_step(c, 2, False, float("nan")) == 3072
    with pytest.raises(D.DlfpError):
        D.dlfp_controller_init(80.0, 512, 1024, 6144)
    with pytest.raises(D.DlfpError):
        D.dlfp_controller_init(float("nan"), 3072, 1024, 6144)


def test_stream_hold_rejects_out_of_range_durations_before_any_launch():
    for us in (0, -5, D.MAX_HOLD_US + 1):
        with pytest.raises(D.DlfpError) as e:
            D.dlfp_stream_hold(us, stream=0)
        assert e.value.status == -1


def test_grid_layout_and_decode_depth_policy():
    """Launches with both shares and more prefill units than compute units lead with
    one prefill unit per compute unit; otherwise every prefill unit comes first.
    Decode-only launches keep two pages in flight; the overrides are honoured."""
    dims = D.make_dims(64, 8)
    cfg = wl.qwen3_32b_config()
    pages = cfg.pages_per_seq()
    nb = int(sum(pages))
    bt_all = wl.block_tables(cfg.seed, pages, nb)
    for p, c, dec, pre in [(8192, 3, True, True), (512, 5, True, True), (8192, 3, False, True),
                           (512, 0, True, False)]:
        its = [x for x in cfg.iteration(p, c) if (x[1] > 1 and pre) or (x[1] == 1 and dec)]
        ql = [x[1] for x in its]
        kl = [x[2] for x in its]
        bt = bt_all[[x[0] for x in its]]
        m = D.dlfp_build_varlen_meta(dims, ql, kl, bt, nb)
        if dec and pre and m.num_prefill_units > 256:
            assert m.prefill_lead_units == 256
        else:
            assert m.prefill_lead_units == m.num_prefill_units
        assert m.decode_pages_in_flight == (2 if m.num_prefill_units == 0 else
                                            m.decode_pages_in_flight)
        assert m.decode_pages_in_flight in (1, 2)
        forced = D.dlfp_build_varlen_meta(dims, ql, kl, bt, nb,
                                          D.dlfp_tuning(0, 0, 0, 0, -1, 1))
        assert forced.prefill_lead_units == forced.num_prefill_units
        assert forced.decode_pages_in_flight == 1
    with pytest.raises(D.DlfpError):
        D.dlfp_build_varlen_meta(dims, ql, kl, bt, nb, D.dlfp_tuning(0, 0, 0, 0, 0, 3))


def test_probe_library_exports_its_declared_symbols():
    import ctypes
    txt = open(os.path.join(ROOT, "include", "dlfp_probe.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    declared = sorted(set(re.findall(r"\bint\s+(dlfp_probe_\w+)\s*\(", txt)))
    assert declared == ["dlfp_probe_hbm_read", "dlfp_probe_mfma"]
    path = os.path.join(ROOT, "paper_2609_38386_amd", "libdlfp_probe.so")
    L = ctypes.CDLL(path)
    for name in declared:
        assert hasattr(L, name), name

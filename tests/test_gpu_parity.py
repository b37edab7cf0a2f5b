"""GPU parity: the HIP path through the C ABI against the oracle on the same seeded inputs.

Bars: page gathers and metadata bit-exact; attention max |err| <= 1e-2 and
mean |err| <= 1e-3 against the float64 oracle over the logical sequences.
"""
import math

import numpy as np
import pytest
import torch

import _random_mixes as rm
from oracle import attention as oa
from oracle import paging as op
from paper_2609_38386_amd import dlfp as D
from paper_2609_38386_amd import runtime as rt
from paper_2609_38386_amd import workload as wl

pytestmark = pytest.mark.gpu

MAX_ABS = 1e-2
MEAN_ABS = 1e-3
SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    D.lib()
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def ws(dev):
    return rt.Workspace(dev, 64 << 20)


def _oracle(seqs, rows=None):
    outs = []
    for i, s in enumerate(seqs):
        r = None if rows is None else rows[i]
        outs.append(oa.attention_sequence(oa.bf16_bits_to_float64(s.stream.q[s.pos0:s.kv_len]),
                                          oa.bf16_bits_to_float64(s.stream.k[:s.kv_len]),
                                          oa.bf16_bits_to_float64(s.stream.v[:s.kv_len]), SCALE,
                                          r))
    return outs


def _compare(got, seqs, label, rows=None):
    """got: float64 [T][Hq][D] packed in batch order; returns (max, mean) abs error."""
    want = _oracle(seqs, rows)
    errs = []
    off = 0
    for i, s in enumerate(seqs):
        g = got[off:off + s.q_len]
        if rows is not None:
            g = g[rows[i]]
        errs.append(np.abs(g - want[i]).ravel())
        off += s.q_len
    e = np.concatenate(errs)
    mx, mean = float(e.max()), float(e.mean())
    print(f"{label}: max_abs={mx:.3e} mean_abs={mean:.3e} n={e.size}", flush=True)
    if mx > MAX_ABS:
        for i, (s, er) in enumerate(zip(seqs, errs)):
            er = er.reshape(-1, s.stream.shape.num_q_heads, 128) if rows is None else er
            print(f"  seq {i} q_len={s.q_len} kv_len={s.kv_len} max={er.max():.3e}", flush=True)
    assert np.all(np.isfinite(got)), label
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (label, mx, mean)
    return mx, mean


def _to64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _seqs(shape, specs, seed=801):
    """specs: list of (q_len, kv_len); each sequence gets its own stream."""
    out = []
    for i, (q, kv) in enumerate(specs):
        st = wl.SeqStream(seed, wl.ROLE_DECODER if q == 1 else wl.ROLE_PROMPT, i, shape, kv)
        out.append(wl.IterationSeq(st, q, kv))
    return out


def _pool_for(seqs, extra=7):
    return sum(wl.pages_for(s.kv_len) for s in seqs) + extra


def test_kv_append_bit_exact_with_poisoned_pool(dev, ws):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    dims = D.make_dims(16, 8)
    it = rt.Iteration(dims, seqs, cfg.pool_size(), cfg.seed, dev, fill_bits=rt.BF16_NAN_BITS)
    it.batch.append(it.pool, it.k_new, it.v_new)
    torch.cuda.synchronize()
    kc, vc = it.pool.host_bits()
    written = 0
    for i, s in enumerate(seqs):
        k, v = op.gather_sequence(kc, vc, it.block_table[i], s.kv_len)
        assert np.array_equal(k, s.stream.k[:s.kv_len]), i
        assert np.array_equal(v, s.stream.v[:s.kv_len]), i
        written += s.kv_len
    # every slot not written still holds the poison
    nan_k = int(np.sum(kc[:, 0, :, 0] == rt.BF16_NAN_BITS))
    assert nan_k == cfg.pool_size() * 16 - written
    assert int(np.sum(vc[:, 3, 5, :] == rt.BF16_NAN_BITS)) == cfg.pool_size() * 16 - written


def test_slot_mapping_on_device_matches_twin(dev):
    from oracle import meta as om
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    bt = wl.block_tables(cfg.seed, [wl.pages_for(s.kv_len) for s in seqs], cfg.pool_size())
    b = rt.Batch(D.make_dims(16, 8), [s.q_len for s in seqs], [s.kv_len for s in seqs], bt,
                 cfg.pool_size(), dev)
    _, _, slots = om.varlen_meta([s.q_len for s in seqs], [s.kv_len for s in seqs], bt)
    assert b.d_slots.cpu().numpy().tolist() == slots


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_tiny_iteration_parity(dev, ws, out_dtype):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    it = rt.Iteration(D.make_dims(16, 8), seqs, cfg.pool_size(), cfg.seed, dev,
                      fill_bits=rt.BF16_NAN_BITS)
    out = it.run(ws, SCALE, out_dtype)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    got = _to64(out)
    _compare(got[:128], seqs[:1], f"tiny prefill {out_dtype}")
    _compare(got[128:], seqs[1:], f"tiny decode {out_dtype}")


@pytest.mark.parametrize("tn", [(16, 64), (32, 128), (48, 192)])
def test_forced_splits_combine(dev, ws, tn):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    it = rt.Iteration(D.make_dims(16, 8), seqs, cfg.pool_size(), cfg.seed, dev,
                      fill_bits=rt.BF16_NAN_BITS, tuning=D.dlfp_tuning(tn[0], tn[1], 0))
    assert it.batch.meta.num_groups > 0
    out = it.run(ws, SCALE, torch.float32)
    torch.cuda.synchronize()
    _compare(_to64(out), seqs, f"split {tn}")
    # the launch leaves the header and every counter at zero
    hdr = ws.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy()
    assert not hdr.any()


@pytest.mark.parametrize("g,hkv", [(1, 4), (2, 8), (4, 8), (8, 8), (8, 2)])
def test_gqa_groups_ragged(dev, ws, g, hkv):
    shape = wl.AttnShape(g * hkv, hkv)
    specs = [(77, 122), (1, 1), (1, 17), (1, 33), (1, 100), (130, 130), (1, 257), (3, 50)]
    seqs = _seqs(shape, specs, seed=900 + g)
    it = rt.Iteration(D.make_dims(g * hkv, hkv), seqs, _pool_for(seqs), 5, dev,
                      fill_bits=rt.BF16_NAN_BITS, tuning=D.dlfp_tuning(32, 64, 0))
    out = it.run(ws, SCALE, torch.float32)
    torch.cuda.synchronize()
    _compare(_to64(out), seqs, f"g={g} hkv={hkv}")


@pytest.mark.parametrize("split,tile", [(64, 0), (192, 0), (256, 16), (320, 0), (1024, 8),
                                        (512, 1), (0, 0)])
def test_prefill_splits_and_small_tiles(dev, ws, split, tile):
    """Key ranges of 1, 3, 4, 5 and up to 16 tiles with ragged ends; tiles of
    fewer tokens than a full one (down to a single token)."""
    shape = wl.AttnShape(16, 8)
    specs = [(37, 1111), (100, 700), (1, 900), (64, 333), (5, 1029), (1, 70)]
    seqs = _seqs(shape, specs, seed=31 + split + tile)
    it = rt.Iteration(D.make_dims(16, 8), seqs, _pool_for(seqs), 6, dev,
                      fill_bits=rt.BF16_NAN_BITS,
                      tuning=D.dlfp_tuning(64, split, 0, tile))
    out = it.run(ws, SCALE, torch.float32)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    _compare(_to64(out), seqs, f"split={split} tile={tile}")
    hdr = ws.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy()
    assert not hdr.any()


def test_decode_only_and_prefill_only(dev, ws):
    shape = wl.AttnShape(16, 8)
    dec = _seqs(shape, [(1, n) for n in (64, 100, 256, 511, 1000)], seed=11)
    it = rt.Iteration(D.make_dims(16, 8), dec, _pool_for(dec), 3, dev, fill_bits=rt.BF16_NAN_BITS)
    _compare(_to64(it.run(ws, SCALE, torch.float32)), dec, "decode only")
    pre = _seqs(shape, [(128, 512), (64, 64), (200, 1000)], seed=12)
    it = rt.Iteration(D.make_dims(16, 8), pre, _pool_for(pre), 4, dev, fill_bits=rt.BF16_NAN_BITS)
    _compare(_to64(it.run(ws, SCALE, torch.float32)), pre, "prefill only")


def test_decode_path_equals_last_prefill_row(dev, ws):
    """The VALU decode path and the MFMA prefill path agree on the same query."""
    shape = wl.AttnShape(16, 8)
    st = wl.SeqStream(21, wl.ROLE_PROMPT, 0, shape, 300)
    a = rt.Iteration(D.make_dims(16, 8), [wl.IterationSeq(st, 50, 300)], 40, 1, dev)
    b = rt.Iteration(D.make_dims(16, 8), [wl.IterationSeq(st, 1, 300)], 40, 1, dev)
    oa_ = _to64(a.run(ws, SCALE, torch.float32))
    ob = _to64(b.run(ws, SCALE, torch.float32))
    assert np.abs(oa_[-1] - ob[0]).max() <= 2 * MAX_ABS / 4


def test_deterministic_and_counters_reset(dev, ws):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    it = rt.Iteration(D.make_dims(16, 8), seqs, cfg.pool_size(), cfg.seed, dev,
                      tuning=D.dlfp_tuning(16, 64, 0))
    o1 = it.run(ws, SCALE, torch.float32).clone()
    o2 = it.run(ws, SCALE, torch.float32, append=False).clone()
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_bad_block_id_raises_error_word_without_reading(dev):
    shape = wl.AttnShape(16, 8)
    seqs = _seqs(shape, [(1, 40)], seed=3)
    it = rt.Iteration(D.make_dims(16, 8), seqs, 8, 2, dev)
    ws2 = rt.Workspace(dev, 1 << 16)
    bad = it.batch.d_block_table.clone()
    bad[0, 2] = 10_000   # the first two pages' ids travel with the work record
    it.batch.d_block_table = bad
    it.run(ws2, SCALE, torch.float32, append=False)
    assert D.dlfp_workspace_error(ws2.buf) == 1
    # a bad id in a decode record's second-page field is caught the same way
    it2 = rt.Iteration(D.make_dims(16, 8), seqs, 8, 2, dev)
    ws3 = rt.Workspace(dev, 1 << 16)
    w = it2.batch.d_work.clone()
    w[3 * D.WORK_INTS + 15] = 10_000
    it2.batch.d_work = w
    it2.run(ws3, SCALE, torch.float32, append=False)
    assert D.dlfp_workspace_error(ws3.buf) == 1


def test_abi_rejects_bad_arguments(dev, ws):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    it = rt.Iteration(D.make_dims(16, 8), seqs, cfg.pool_size(), cfg.seed, dev)
    out = torch.empty((it.batch.num_tokens, 16, 128), dtype=torch.float32, device=dev)
    small = torch.empty(D.WORKSPACE_PARTIALS - 4, dtype=torch.uint8, device=dev)
    b = it.batch
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_attention_mixed(b.dims, b.meta, b.d_work, b.d_block_table, it.q, it.pool.k,
                               it.pool.v, SCALE, out, small)
    assert e.value.status == -3
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_attention_mixed(b.dims, b.meta, b.d_work, b.d_block_table, it.q, it.pool.k,
                               it.pool.v, -1.0, out, ws.buf)
    assert e.value.status == -1
    with pytest.raises(D.DlfpError) as e:
        D.dlfp_attention_mixed(D.make_dims(16, 8, head_dim=64), b.meta, b.d_work,
                               b.d_block_table, it.q, it.pool.k, it.pool.v, SCALE, out, ws.buf)
    assert e.value.status == -5
    # a batch with work needs its new keys and values: an empty (null) k_new is refused
    nothing = torch.empty((0, 8, 128), dtype=torch.bfloat16, device=dev)
    for k_new, v_new in ((nothing, it.v_new), (it.k_new, nothing)):
        with pytest.raises(D.DlfpError) as e:
            D.dlfp_append_attention_mixed(b.dims, b.meta, b.d_work, b.d_block_table, it.q,
                                          k_new, v_new, it.pool.k, it.pool.v, SCALE, out,
                                          ws.buf)
        assert e.value.status == -1


@pytest.mark.parametrize("p,chunk", [(64, 0), (64, 127), (512, 7), (2048, 0), (2048, 3)])
def test_qwen3_0_6b_iteration_all_rows(dev, ws, p, chunk):
    cfg = wl.qwen3_0_6b_config()
    dec = cfg.decoder_streams()
    ctx = cfg.decoder_contexts()
    prompt = cfg.prompt_stream()
    seqs = [wl.IterationSeq(prompt, p, (chunk + 1) * p)]
    seqs += [wl.IterationSeq(dec[i], 1, int(ctx[i]) + chunk) for i in range(cfg.n_decoders)]
    it = rt.Iteration(D.make_dims(16, 8), seqs, _pool_for(seqs), cfg.seed, dev,
                      fill_bits=rt.BF16_NAN_BITS)
    out = it.run(ws, SCALE, torch.bfloat16)
    torch.cuda.synchronize()
    got = _to64(out)
    _compare(got[:p], seqs[:1], f"0.6b p={p} c={chunk} prefill")
    _compare(got[p:], seqs[1:], f"0.6b p={p} c={chunk} decode")


def test_workspace_reuse_across_iteration_shapes(dev):
    """A small launch's partials must not be read as a later, larger launch's counters."""
    shape = wl.AttnShape(16, 8)
    w = rt.Workspace(dev, 8 << 20)
    small = _seqs(shape, [(128, 512)] + [(1, n) for n in (64, 200)], seed=31)
    big = _seqs(shape, [(77, 300)] + [(1, n) for n in range(100, 1300, 60)], seed=32)
    a = rt.Iteration(D.make_dims(16, 8), small, _pool_for(small), 1, dev,
                     tuning=D.dlfp_tuning(16, 64, 0))
    b = rt.Iteration(D.make_dims(16, 8), big, _pool_for(big), 2, dev,
                     tuning=D.dlfp_tuning(16, 64, 0))
    assert b.batch.meta.num_groups > 4 * a.batch.meta.num_groups
    for _ in range(2):
        _compare(_to64(a.run(w, SCALE, torch.float32)), small, "reuse small")
        _compare(_to64(b.run(w, SCALE, torch.float32)), big, "reuse big")
    torch.cuda.synchronize()
    assert not w.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any()


@pytest.mark.parametrize("g", [2, 8])
def test_score_spikes_far_above_the_rest(dev, ws, g):
    """Keys whose scores exceed every other score by ~300 (natural log units):
    any lane that took a smaller reference maximum than its row's would form
    probabilities near 2^400 and overflow.  Positive queries and keys of 32.0
    in every dim place spikes at keys 5, 13 and 389 only (key % 8 in 4..7,
    which the upper half of a wavefront holds in the prefill score layout, so
    a row maximum taken over the lower half alone misses them)."""
    shape = wl.AttnShape(8 * g, 8)
    seqs = _seqs(shape, [(128, 512), (1, 300), (1, 77)], seed=21 + g)
    spike = np.uint16(0x4200)  # bf16 32.0
    for s in seqs:
        q = s.stream.q
        q &= np.uint16(0x7FFF)  # every query positive
        for key in (5, 13, 389):
            if key < s.kv_len:
                s.stream.k[key] = spike
    it = rt.Iteration(D.make_dims(8 * g, 8), seqs, _pool_for(seqs), 801, dev,
                      fill_bits=rt.BF16_NAN_BITS)
    out = it.run(ws, SCALE, torch.float32)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    _compare(_to64(out), seqs, f"score spikes g={g}")


@pytest.mark.parametrize("g,hkv,fused", [(2, 8, False), (1, 4, True), (8, 2, True), (4, 1, False)])
def test_maximum_unit_sizes(dev, ws, g, hkv, fused):
    """Units at the library's limits: prefill units of exactly
    DLFP_MAX_PREFILL_UNIT_KEYS keys in one split (their block ids fill the LDS
    table), decode units of exactly DLFP_MAX_DECODE_UNIT_KEYS keys (a 4096-key
    decoder whole, a 32768-key decoder in eight splits), a 4097-key context in
    two equal splits, and a one-key decoder; for each decode path (g = 1 on the
    VALU, g >= 2 on MFMA) and both launch forms.  Every row against the oracle;
    the output is NaN-filled."""
    hq = g * hkv
    shape = wl.AttnShape(hq, hkv)
    specs = [(16, 32768), (1, 4096), (1, 4097), (1, 32768), (1, 1)]
    seqs = _seqs(shape, specs, seed=4242 + g)
    it = rt.Iteration(D.make_dims(hq, hkv), seqs, _pool_for(seqs), 8, dev,
                      fill_bits=rt.BF16_NAN_BITS, tuning=D.dlfp_tuning(4096, 32768, 0))
    m = it.batch.meta
    pre = m.work[:m.num_prefill_units]
    dec = m.work[m.num_prefill_units:m.num_units]
    assert len(pre) == hkv and all(int(u[5]) - int(u[4]) == 32768 for u in pre)
    assert int((dec[:, 5] - dec[:, 4]).max()) == 4096
    assert int((dec[:, 5] - dec[:, 4]).min()) == 1
    out = torch.full((m.num_tokens, hq, 128), float("nan"), dtype=torch.float32, device=dev)
    it.run(ws, SCALE, out=out, fused=fused)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    _compare(_to64(out), seqs, f"maximum unit sizes g={g} hkv={hkv} fused={fused}")
    assert not ws.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any()


def test_empty_batch_launches_nothing(dev):
    """A batch with no sequences, every device array empty (null pointers), through
    every launch entry point: each returns success without launching, the pool keeps
    every bit, and the workspace header and counters stay zero."""
    dims = D.make_dims(16, 8)
    meta = D.dlfp_build_varlen_meta(dims, [], [], np.zeros((0, 1), np.int32), 8)
    assert meta.num_units == 0 and meta.num_tokens == 0 and meta.num_append == 0
    pool = rt.KVPool(8, 8, dev, fill_bits=0x7FC1)
    before = pool.host_bits()
    ws0 = rt.Workspace(dev, 1 << 16)

    def empty(*shape, dtype=torch.bfloat16):
        t = torch.empty(shape, dtype=dtype, device=dev)
        assert t.data_ptr() == 0
        return t

    d_work = empty(0, D.WORK_INTS, dtype=torch.int32)
    d_bt = empty(0, 1, dtype=torch.int32)
    q, kv = empty(0, 16, 128), empty(0, 8, 128)
    out = empty(0, 16, 128, dtype=torch.float32)
    D.dlfp_kv_append(dims, kv, kv, empty(0, dtype=torch.int32), pool.k, pool.v)
    D.dlfp_attention_mixed(dims, meta, d_work, d_bt, q, pool.k, pool.v, SCALE, out, ws0.buf)
    D.dlfp_append_attention_mixed(dims, meta, d_work, d_bt, q, kv, kv, pool.k, pool.v, SCALE,
                                  out, ws0.buf)
    D.dlfp_append_attention_mixed_static(dims, meta, d_work, d_bt, q, kv, kv, pool.k, pool.v,
                                         SCALE, out)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws0.buf) == 0
    assert not ws0.buf[:D.WORKSPACE_PARTIALS].cpu().numpy().any()
    after = pool.host_bits()
    assert np.array_equal(before[0], after[0]) and np.array_equal(before[1], after[1])


@pytest.mark.parametrize("i", range(rm.CASES))
def test_random_mix(dev, ws, i):
    """Seeded random mixes of GQA shape, decoders, prompt chunks, tuning, launch
    form and output type (the cases whose metadata the CPU suite checks against
    the twin): every row against the oracle, the error word clear and the
    counters back at zero."""
    g, hkv, specs, tn, fused, fp32_out = rm.case(i)
    shape = wl.AttnShape(g * hkv, hkv)
    seqs = _seqs(shape, specs, seed=rm.seed(i))
    pages = [wl.pages_for(s.kv_len) for s in seqs]
    print(f"random mix {i}: g={g} hkv={hkv} {len(seqs)} sequences, tuning {tn}, "
          f"fused={fused}, fp32 output={fp32_out}", flush=True)
    it = rt.Iteration(D.make_dims(g * hkv, hkv), seqs, rm.pool(pages), rm.seed(i), dev,
                      fill_bits=rt.BF16_NAN_BITS, tuning=D.dlfp_tuning(*tn))
    out = it.run(ws, SCALE, torch.float32 if fp32_out else torch.bfloat16, fused=fused)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    assert not ws.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any()
    _compare(_to64(out), seqs, f"random mix {i}")

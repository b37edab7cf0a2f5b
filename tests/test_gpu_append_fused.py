"""GPU: the one-launch append + attention (dlfp_append_attention_mixed) through the C ABI.

Bars: output and every pool slot bit-identical to dlfp_kv_append followed by
dlfp_attention_mixed on the same inputs (same arithmetic, so equal bits);
attention within max |err| <= 1e-2, mean |err| <= 1e-3 of the float64 oracle;
the workspace header and counters back at zero after every launch.
"""
import math

import numpy as np
import pytest
import torch

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


def _seqs(shape, specs, seed):
    out = []
    for i, (q, kv) in enumerate(specs):
        st = wl.SeqStream(seed, wl.ROLE_DECODER if q == 1 else wl.ROLE_PROMPT, i, shape, kv)
        out.append(wl.IterationSeq(st, q, kv))
    return out


def _pool_for(seqs, extra=7):
    return sum(wl.pages_for(s.kv_len) for s in seqs) + extra


def _oracle_check(got, seqs, label):
    errs = []
    off = 0
    for s in seqs:
        want = oa.attention_sequence(oa.bf16_bits_to_float64(s.stream.q[s.pos0:s.kv_len]),
                                     oa.bf16_bits_to_float64(s.stream.k[:s.kv_len]),
                                     oa.bf16_bits_to_float64(s.stream.v[:s.kv_len]), SCALE)
        errs.append(np.abs(got[off:off + s.q_len] - want).ravel())
        off += s.q_len
    e = np.concatenate(errs)
    print(f"{label}: max_abs={e.max():.3e} mean_abs={e.mean():.3e}", flush=True)
    assert np.all(np.isfinite(got)), label
    assert e.max() <= MAX_ABS and e.mean() <= MEAN_ABS, (label, e.max(), e.mean())


def _header_clear(ws):
    return not ws.buf[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any()


def _fused_vs_two_calls(dev, dims, seqs, pool_blocks, seed, tuning=None, out_dtype=torch.float32,
                        label=""):
    """Run both paths on identical poisoned pools; return the fused output (float64)."""
    tn = None if tuning is None else [getattr(tuning, f) for f, _ in tuning._fields_]
    print(f"case {label}: {len(seqs)} seqs, tuning {tn}", flush=True)
    a = rt.Iteration(dims, seqs, pool_blocks, seed, dev, fill_bits=rt.BF16_NAN_BITS,
                     tuning=tuning)
    b = rt.Iteration(dims, seqs, pool_blocks, seed, dev, fill_bits=rt.BF16_NAN_BITS,
                     tuning=tuning)
    wa, wb = rt.Workspace(dev, 16 << 20), rt.Workspace(dev, 16 << 20)
    oa_ = a.run(wa, SCALE, out_dtype)
    ob = b.run(wb, SCALE, out_dtype, fused=True)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(wb.buf) == 0, label
    assert _header_clear(wb), label
    assert torch.equal(oa_.view(torch.int32 if out_dtype == torch.float32 else torch.int16),
                       ob.view(torch.int32 if out_dtype == torch.float32 else torch.int16)), label
    ka, va = a.pool.host_bits()
    kb_, vb = b.pool.host_bits()
    assert np.array_equal(ka, kb_), label
    assert np.array_equal(va, vb), label
    for i, s in enumerate(seqs):
        k, v = op.gather_sequence(kb_, vb, b.block_table[i], s.kv_len)
        assert np.array_equal(k, s.stream.k[:s.kv_len]), (label, i)
        assert np.array_equal(v, s.stream.v[:s.kv_len]), (label, i)
    return ob.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_tiny_iteration_fused_equals_two_calls(dev, out_dtype):
    cfg = wl.tiny_config()
    seqs = wl.tiny_iteration(cfg)
    got = _fused_vs_two_calls(dev, D.make_dims(16, 8), seqs, cfg.pool_size(), cfg.seed,
                              out_dtype=out_dtype, label=f"tiny {out_dtype}")
    _oracle_check(got, seqs, f"tiny fused {out_dtype}")


@pytest.mark.parametrize("g,hkv", [(1, 4), (2, 8), (4, 8), (8, 8), (8, 2)])
def test_gqa_groups_ragged_fused(dev, g, hkv):
    shape = wl.AttnShape(g * hkv, hkv)
    specs = [(77, 122), (1, 1), (1, 17), (1, 33), (1, 100), (130, 130), (1, 257), (3, 50)]
    seqs = _seqs(shape, specs, seed=900 + g)
    got = _fused_vs_two_calls(dev, D.make_dims(g * hkv, hkv), seqs, _pool_for(seqs), 5,
                              tuning=D.dlfp_tuning(32, 64, 0), label=f"g={g} hkv={hkv}")
    _oracle_check(got, seqs, f"fused g={g} hkv={hkv}")


@pytest.mark.parametrize("split,tile", [(64, 0), (192, 0), (256, 16), (1024, 8), (512, 1),
                                        (0, 0)])
def test_prefill_splits_and_unaligned_chunks_fused(dev, split, tile):
    """Chunks starting mid-page (the page holding the first new token also holds
    cached keys), key splits ending before, in and after that page, and tiles
    down to one token."""
    shape = wl.AttnShape(16, 8)
    specs = [(37, 1111), (100, 700), (1, 900), (64, 333), (5, 1029), (1, 70), (16, 16)]
    seqs = _seqs(shape, specs, seed=131 + split + tile)
    got = _fused_vs_two_calls(dev, D.make_dims(16, 8), seqs, _pool_for(seqs), 6,
                              tuning=D.dlfp_tuning(64, split, 0, tile),
                              label=f"split={split} tile={tile}")
    _oracle_check(got, seqs, f"fused split={split} tile={tile}")


def test_decode_only_and_prefill_only_fused(dev):
    shape = wl.AttnShape(16, 8)
    dec = _seqs(shape, [(1, n) for n in (1, 16, 17, 100, 256, 511, 1000)], seed=11)
    got = _fused_vs_two_calls(dev, D.make_dims(16, 8), dec, _pool_for(dec), 3, label="decode")
    _oracle_check(got, dec, "fused decode only")
    pre = _seqs(shape, [(128, 512), (64, 64), (200, 1000), (2048, 2048)], seed=12)
    got = _fused_vs_two_calls(dev, D.make_dims(16, 8), pre, _pool_for(pre), 4, label="prefill")
    _oracle_check(got, pre, "fused prefill only")


@pytest.mark.parametrize("p,chunk", [(64, 0), (64, 127), (512, 7), (2048, 0), (2048, 3)])
def test_qwen3_0_6b_iteration_fused(dev, p, chunk):
    cfg = wl.qwen3_0_6b_config()
    dec = cfg.decoder_streams()
    ctx = cfg.decoder_contexts()
    seqs = [wl.IterationSeq(cfg.prompt_stream(), p, (chunk + 1) * p)]
    seqs += [wl.IterationSeq(dec[i], 1, int(ctx[i]) + chunk) for i in range(cfg.n_decoders)]
    got = _fused_vs_two_calls(dev, D.make_dims(16, 8), seqs, _pool_for(seqs), cfg.seed,
                              out_dtype=torch.bfloat16, label=f"0.6b p={p} c={chunk}")
    _oracle_check(got, seqs, f"fused 0.6b p={p} c={chunk}")


def test_back_to_back_fused_launches_share_a_workspace(dev):
    """Launches of different shapes on one workspace: each must wait for its own
    append records, never for a count left by the previous launch."""
    shape = wl.AttnShape(16, 8)
    w = rt.Workspace(dev, 16 << 20)
    its = []
    for k, specs in enumerate([[(300, 900)] + [(1, n) for n in (64, 700)],
                               [(64, 64), (1, 33)],
                               [(1000, 3000)] + [(1, n) for n in range(100, 1300, 100)]]):
        seqs = _seqs(shape, specs, seed=70 + k)
        its.append((seqs, rt.Iteration(D.make_dims(16, 8), seqs, _pool_for(seqs), k, dev,
                                       fill_bits=rt.BF16_NAN_BITS)))
    outs = []
    for rep in range(3):
        for seqs, it in its:
            outs.append(it.run(w, SCALE, torch.float32, fused=True))
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(w.buf) == 0
    assert _header_clear(w)
    n = len(its)
    for i, (seqs, _) in enumerate(its):
        first = outs[i]
        for rep in range(1, 3):
            assert torch.equal(first, outs[rep * n + i]), (i, rep)
        _oracle_check(first.cpu().numpy().astype(np.float64), seqs, f"back-to-back {i}")


@pytest.mark.parametrize("specs", [[(1000, 3000), (1, 500)], [(1000, 1000)], [(900, 1900)]])
def test_long_prompt_appended_inside_the_launch(dev, specs):
    """At most 128 append records (here Hkv = 2) are written inside the attention
    launch, so long prefill units wait for them: from the first tile when the
    whole prompt is new, late in their loop over a cached prefix."""
    shape = wl.AttnShape(16, 2)
    seqs = _seqs(shape, specs, seed=55)
    dims = D.make_dims(16, 2)
    it = rt.Batch(dims, [s.q_len for s in seqs], [s.kv_len for s in seqs],
                  wl.block_tables(1, [wl.pages_for(s.kv_len) for s in seqs], _pool_for(seqs)),
                  _pool_for(seqs), dev)
    assert 0 < it.meta.num_append <= 128, it.meta.num_append
    got = _fused_vs_two_calls(dev, dims, seqs, _pool_for(seqs), 9, label=f"long {specs}")
    _oracle_check(got, seqs, f"fused long prompt {specs}")

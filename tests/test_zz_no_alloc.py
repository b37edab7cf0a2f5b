"""GPU: the no-allocation entry point dlfp_append_attention_mixed_static through the C ABI.

It must give what dlfp_append_attention_mixed gives with a caller-allocated
workspace on the same inputs -- the same kernels over the same work list, so
the output and every cache slot are equal bit for bit -- and both are within
the oracle's bounds (max |err| <= 1e-2, mean |err| <= 1e-3).  Two calls in a
row, the second on a smaller iteration, so the second call finds the static
workspace as the first one left it.  A work list whose workspace exceeds the
static array is rejected before anything is launched.
"""
import ctypes
import math

import numpy as np
import pytest
import torch

from oracle import attention as oa
from paper_2609_38386_amd import dlfp as D
from paper_2609_38386_amd import runtime as rt
from paper_2609_38386_amd import workload as wl

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)


def _seqs(shape, specs, seed):
    out = []
    for i, (q, kv) in enumerate(specs):
        st = wl.SeqStream(seed, wl.ROLE_DECODER if q == 1 else wl.ROLE_PROMPT, i, shape, kv)
        out.append(wl.IterationSeq(st, q, kv))
    return out


def _run_pair(dev, g, specs, seed, tuning):
    shape = wl.AttnShape(8 * g, 8)
    dims = D.make_dims(8 * g, 8)
    seqs = _seqs(shape, specs, seed)
    pool_blocks = sum(wl.pages_for(s.kv_len) for s in seqs) + 5
    a = rt.Iteration(dims, seqs, pool_blocks, seed, dev, fill_bits=rt.BF16_NAN_BITS, tuning=tuning)
    b = rt.Iteration(dims, seqs, pool_blocks, seed, dev, fill_bits=rt.BF16_NAN_BITS, tuning=tuning)
    assert a.batch.meta.num_groups > 0   # the workspace holds split partials
    ws = rt.Workspace(dev, 8 << 20)
    shape_out = (a.batch.num_tokens, 8 * g, 128)
    out_a = torch.full(shape_out, float("nan"), dtype=torch.float32, device=dev)
    out_b = torch.full(shape_out, float("nan"), dtype=torch.float32, device=dev)
    ba, bb = a.batch, b.batch
    D.dlfp_append_attention_mixed(dims, ba.meta, ba.d_work, ba.d_block_table, a.q, a.k_new,
                                  a.v_new, a.pool.k, a.pool.v, SCALE, out_a,
                                  ws.ensure(ba.meta.workspace_bytes))
    D.dlfp_append_attention_mixed_static(dims, bb.meta, bb.d_work, bb.d_block_table, b.q,
                                         b.k_new, b.v_new, b.pool.k, b.pool.v, SCALE, out_b)
    torch.cuda.synchronize()
    assert D.dlfp_workspace_error(ws.buf) == 0
    assert torch.equal(out_a.view(torch.int32), out_b.view(torch.int32))
    assert torch.equal(a.pool.k.view(torch.int16), b.pool.k.view(torch.int16))
    assert torch.equal(a.pool.v.view(torch.int16), b.pool.v.view(torch.int16))
    got = out_b.cpu().numpy().astype(np.float64)
    off, errs = 0, []
    for s in seqs:
        want = oa.attention_sequence(oa.bf16_bits_to_float64(s.stream.q[s.pos0:s.kv_len]),
                                     oa.bf16_bits_to_float64(s.stream.k[:s.kv_len]),
                                     oa.bf16_bits_to_float64(s.stream.v[:s.kv_len]), SCALE)
        errs.append(np.abs(got[off:off + s.q_len] - want).ravel())
        off += s.q_len
    e = np.concatenate(errs)
    print(f"g={g} {len(specs)} sequences: max_abs={e.max():.3e} mean_abs={e.mean():.3e}",
          flush=True)
    assert e.max() <= 1e-2 and e.mean() <= 1e-3


def test_static_workspace_equals_caller_workspace_on_two_calls():
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    tuning = D.dlfp_tuning(64, 128, 0)
    big = [(300, 1000)] + [(1, n) for n in range(200, 2600, 120)]
    small = [(40, 90)] + [(1, n) for n in (70, 300, 513)]
    _run_pair(dev, 2, big, 41, tuning)
    _run_pair(dev, 8, small, 42, tuning)


def test_static_workspace_rejects_a_work_list_too_large():
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    dims = D.make_dims(16, 8)
    seqs = _seqs(wl.AttnShape(16, 8), [(1, 64)], 3)
    it = rt.Iteration(dims, seqs, 8, 3, dev)
    m = it.batch.meta
    big = D.dlfp_meta()
    ctypes.pointer(big)[0] = m.c
    big.workspace_bytes = D.STATIC_WORKSPACE_BYTES + 256
    out = torch.empty((1, 16, 128), dtype=torch.float32, device=dev)
    st = D.lib().dlfp_append_attention_mixed_static(
        ctypes.byref(dims), ctypes.byref(big), D._dptr(it.batch.d_work),
        D._dptr(it.batch.d_block_table), int(it.batch.d_block_table.shape[1]), 8,
        D._dptr(it.q), D._dptr(it.k_new), D._dptr(it.v_new), D._dptr(it.pool.k),
        D._dptr(it.pool.v), ctypes.c_float(SCALE), D._dptr(out), 1, D._stream(None))
    assert st == -3

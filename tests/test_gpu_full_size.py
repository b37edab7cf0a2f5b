"""Full-size parity on sampled rows.

Qwen3-8B and Qwen3-32B attention shapes at the sizes the benchmark times and in
its launch configuration: automatic split policy, one bf16 pool per layer
filled on the device by a seeded generator, queries and new keys / values
likewise, one launch per iteration that appends the new keys and values and
attends (dlfp_append_attention_mixed; one case per shape runs the
attention-only launch over a pool appended beforehand).  For sampled query
rows the oracle gathers the pages the row reads (its own gather of the
library's declared layout) -- whose new-token slots must hold the iteration's
keys and values bit for bit -- recomputes the row in float64 and the test
compares every element of the row (all query heads) with the fp32 output:
max |err| <= 1e-2 per row, mean |err| <= 1e-3 over the sampled rows of an
iteration.

Sampled rows per iteration: the decoders with the longest and the shortest
context plus two seeded random ones, and the first, two interior and the last
token of the prefill chunk.
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

SCALE = 1.0 / math.sqrt(128)
MAX_ABS, MEAN_ABS = 1e-2, 1e-3


class FullSize:
    def __init__(self, cfg):
        assert torch.cuda.is_available()
        self.dev = torch.device("cuda:0")
        self.cfg = cfg
        sh = cfg.shape
        self.hq = sh.num_q_heads
        self.dims = D.make_dims(sh.num_q_heads, sh.num_kv_heads)
        pages = cfg.pages_per_seq()
        self.num_blocks = int(sum(pages))
        self.bt = wl.block_tables(cfg.seed, pages, self.num_blocks)  # decoders, then the prompt
        self.pool = rt.KVPool(self.num_blocks, sh.num_kv_heads, self.dev)
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(cfg.seed)
        self.pool.k.normal_(generator=self.gen)
        self.pool.v.normal_(generator=self.gen)
        self.stage = rt.StagedBatch(self.dims, cfg.n_decoders + 1,
                                    max(cfg.chunks) + cfg.n_decoders, 65536, self.dev)
        self.ws = rt.Workspace(self.dev, 64 << 20)
        self.rng = np.random.default_rng(cfg.seed)

    def run(self, p, c, decoders=True, prefill=True, fused=True):
        its = [x for x in self.cfg.iteration(p, c)
               if (x[1] > 1 and prefill) or (x[1] == 1 and decoders)]
        print(f"{self.cfg.name} p={p} c={c} decoders={decoders} prefill={prefill} "
              f"fused={fused}", flush=True)
        q_len = np.array([x[1] for x in its], dtype=np.int32)
        kv_len = np.array([x[2] for x in its], dtype=np.int32)
        bt = np.ascontiguousarray(self.bt[[x[0] for x in its]])
        st = self.stage.build(q_len, kv_len, bt, self.num_blocks)
        d_bt = torch.from_numpy(bt).to(self.dev)
        T = int(q_len.sum())
        q = torch.empty((T, self.hq, 128), dtype=torch.bfloat16, device=self.dev)
        q.normal_(generator=self.gen)
        hkv = self.dims.num_kv_heads
        k_new = torch.empty((T, hkv, 128), dtype=torch.bfloat16, device=self.dev)
        v_new = torch.empty_like(k_new)
        k_new.normal_(generator=self.gen)
        v_new.normal_(generator=self.gen)
        out = torch.empty((T, self.hq, 128), dtype=torch.float32, device=self.dev)
        ws = self.ws.ensure(st.meta.workspace_bytes)
        if fused:
            D.dlfp_append_attention_mixed(self.dims, st.meta, st.d_work, d_bt, q, k_new, v_new,
                                          self.pool.k, self.pool.v, SCALE, out, ws)
        else:
            D.dlfp_kv_append(self.dims, k_new, v_new, st.d_slots, self.pool.k, self.pool.v)
            D.dlfp_attention_mixed(self.dims, st.meta, st.d_work, d_bt, q, self.pool.k,
                                   self.pool.v, SCALE, out, ws)
        torch.cuda.synchronize()
        assert D.dlfp_workspace_error(ws) == 0
        assert not ws[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any()
        self.check(its, q, out, bt, k_new, v_new)
        return st.meta.num_units

    def check(self, its, q, out, bt, k_new, v_new):
        cu = np.concatenate([[0], np.cumsum([x[1] for x in its])])
        dec = [i for i, x in enumerate(its) if x[1] == 1]
        picks = []
        if dec:
            ctx = [its[i][2] for i in dec]
            chosen = {dec[int(np.argmax(ctx))], dec[int(np.argmin(ctx))]}
            chosen |= set(int(i) for i in self.rng.choice(dec, size=2, replace=False))
            picks += [(i, [0]) for i in sorted(chosen)]
        for i, x in enumerate(its):
            if x[1] > 1:
                ql = x[1]
                picks.append((i, sorted({0, ql // 3, (2 * ql) // 3, ql - 1})))
        errs = []
        for i, rows in picks:
            _, ql, kl = its[i]
            n_pages = (kl + 15) // 16
            idx = torch.from_numpy(bt[i, :n_pages].astype(np.int64)).to(self.dev)
            kc = rt.device_to_bits(self.pool.k.index_select(0, idx))
            vc = rt.device_to_bits(self.pool.v.index_select(0, idx))
            k, v = op.gather_sequence(kc, vc, np.arange(n_pages), kl)
            assert np.array_equal(k[kl - ql:], rt.device_to_bits(k_new[cu[i]:cu[i] + ql])), its[i]
            assert np.array_equal(v[kl - ql:], rt.device_to_bits(v_new[cu[i]:cu[i] + ql])), its[i]
            qb = rt.device_to_bits(q[cu[i]:cu[i] + ql])
            want = oa.attention_sequence(oa.bf16_bits_to_float64(qb), oa.bf16_bits_to_float64(k),
                                         oa.bf16_bits_to_float64(v), SCALE, rows=rows)
            got = out[cu[i]:cu[i] + ql].cpu().numpy().astype(np.float64)[rows]
            e = np.abs(got - want)
            assert np.isfinite(got).all()
            assert e.max() <= MAX_ABS, (its[i], rows, float(e.max()))
            errs.append(e.ravel())
        assert np.concatenate(errs).mean() <= MEAN_ABS


def test_qwen3_8b_sampled_rows():
    f = FullSize(wl.qwen3_8b_config())
    f.run(256, 0)
    f.run(256, 63)
    f.run(4096, 3)
    f.run(4096, 3, decoders=False)
    f.run(256, 0, prefill=False)
    f.run(1024, 5, fused=False)


def test_qwen3_32b_sampled_rows():
    f = FullSize(wl.qwen3_32b_config())
    f.run(512, 63)
    f.run(8192, 0)
    f.run(8192, 3)
    f.run(8192, 3, decoders=False)
    f.run(512, 0, prefill=False)
    f.run(2048, 7, fused=False)

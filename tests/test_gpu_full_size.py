"""Full-size parity of the HIP path against the oracle: Qwen3-0.6B, 8B and 32B shapes.

Each shape runs at the sizes and in the launch configuration the benchmark
times: automatic split policy, one launch per iteration that appends the new
keys and values and attends (dlfp_append_attention_mixed; one iteration per
shape runs dlfp_kv_append + dlfp_attention_mixed instead), bf16 output, one
bf16 pool filled on the device by a seeded generator.  The extra decode-only,
prefill-only and two-launch iterations of each shape write fp32 output, so
both output types are compared at every shape and for both shares.

Inputs.  The pool is filled once and copied to the host.  An iteration's new
keys and values are the pool's own bits at the slots of its new tokens (slots
from the oracle's metadata twin, which must also equal the library's slot
mapping).  Those slots are set to bf16 NaN on the device before the launch:
the append must write every one of them back bit for bit (checked after the
launch), a unit that read one before it was written would produce NaN, and
the keys and values the oracle reads are the same host copy for every
iteration.  Queries are fresh N(0,1) per iteration.  The output is filled with
NaN before each launch and must be finite everywhere after it (a row that no
unit wrote would still be NaN).

Rows compared with the float64 oracle (every element of a row, all heads):
* Qwen3-0.6B: every row of the first, middle and last chunk iteration of each p_t;
* Qwen3-8B: the whole sweep, every chunk iteration of every p_t: every decoder
  row, and of the prompt chunk the first and the last token of every prefill
  unit plus the tokens on either side of every key-split boundary of a prefill
  group that falls inside the chunk;
* Qwen3-32B: the first, middle and last chunk iteration of each p_t, rows as
  for 8B.
Decoder rows are checked decoder by decoder after all iterations (one gather
of the decoder's pages serves every iteration's row), prompt rows per
iteration.  Bars: max |err| <= 1e-2 per element, mean |err| <= 1e-3 over the
checked rows of each iteration and share.
"""
import math
import time

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import meta as om
from oracle import paging as op
from paper_2609_38386_amd import dlfp as D
from paper_2609_38386_amd import runtime as rt
from paper_2609_38386_amd import workload as wl

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)
MAX_ABS, MEAN_ABS = 1e-2, 1e-3
NAN_BITS = np.int16(np.uint16(rt.BF16_NAN_BITS).view(np.int16))


def _log(*a):
    print(*a, flush=True)


def stratified_prompt_rows(work, num_prefill, seq, pos0):
    """Tokens (0-based within the chunk) of sequence `seq` that every prefill unit
    touches at its edges: its first and last token, and the tokens at positions
    b - 1 and b for each key-split boundary b (b = the first key of a split
    after the first) that lies among the unit's tokens."""
    rows = set()
    for u in work[:num_prefill]:
        if int(u[om.W_SEQ]) != seq:
            continue
        t0, nt = int(u[om.W_QTOK0]), int(u[om.W_QNTOK])
        rows.add(t0)
        rows.add(t0 + nt - 1)
        if int(u[om.W_NSPLITS]) > 1 and int(u[om.W_SPLIT]) > 0:
            b = int(u[om.W_KVBEGIN])
            for pos in (b - 1, b):
                t = pos - pos0
                if t0 <= t < t0 + nt:
                    rows.add(t)
    return sorted(rows)


class FullSize:
    def __init__(self, cfg):
        assert torch.cuda.is_available()
        t0 = time.time()
        self.dev = torch.device("cuda:0")
        self.cfg = cfg
        sh = cfg.shape
        self.hq, self.hkv = sh.num_q_heads, sh.num_kv_heads
        self.dims = D.make_dims(self.hq, self.hkv)
        pages = cfg.pages_per_seq()
        self.num_blocks = int(sum(pages))
        self.n_dec = cfg.n_decoders
        self.bt = wl.block_tables(cfg.seed, pages, self.num_blocks)  # decoders, then the prompt
        self.pool = rt.KVPool(self.num_blocks, self.hkv, self.dev)
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(cfg.seed)
        self.pool.k.normal_(generator=self.gen)
        self.pool.v.normal_(generator=self.gen)
        torch.cuda.synchronize()
        self.k_host = self.pool.k.view(torch.int16).cpu()
        self.v_host = self.pool.v.view(torch.int16).cpu()
        self.stage = rt.StagedBatch(self.dims, self.n_dec + 1, max(cfg.chunks) + self.n_dec,
                                    1 << 18, self.dev)
        self.ws = rt.Workspace(self.dev, 64 << 20)
        self.vpos = torch.tensor([op.value_position(t) for t in range(16)], device=self.dev)
        self.dec_rows = {d: [] for d in range(self.n_dec)}  # d -> [(iteration, pos, q, out)]
        self.prompt_rows = []                                # (iteration, pos, q, out)
        self.labels = []
        _log(f"{cfg.name}: pool of {self.num_blocks} blocks ready in {time.time() - t0:.1f}s")

    def run(self, p, c, decoders=True, prefill=True, fused=True, all_rows=False,
            out_dtype=torch.bfloat16):
        its = [x for x in self.cfg.iteration(p, c)
               if (x[1] > 1 and prefill) or (x[1] == 1 and decoders)]
        label = (f"{self.cfg.name} p={p} c={c} dec={decoders} pre={prefill} fused={fused} "
                 f"out={str(out_dtype).split('.')[-1]}")
        ii = len(self.labels)
        self.labels.append(label)
        q_len = np.array([x[1] for x in its], dtype=np.int32)
        kv_len = np.array([x[2] for x in its], dtype=np.int32)
        bt = np.ascontiguousarray(self.bt[[x[0] for x in its]])
        st = self.stage.build(q_len, kv_len, bt, self.num_blocks)
        m = st.meta
        T = int(q_len.sum())
        _, _, slots = om.varlen_meta(q_len, kv_len, bt)
        assert np.array_equal(m.slot_mapping[:T], np.asarray(slots, dtype=np.int32)), label
        d_bt = torch.from_numpy(bt).to(self.dev)
        sl = torch.as_tensor(np.asarray(slots, dtype=np.int64), device=self.dev)
        blk, off = sl // 16, sl % 16
        vp = self.vpos[off]
        k16, v16 = self.pool.k.view(torch.int16), self.pool.v.view(torch.int16)
        k_new = k16[blk, :, off, :].clone()      # [T][Hkv][128]: the pool's own bits
        v_new = v16[blk, :, :, vp].clone()
        k16[blk, :, off, :] = NAN_BITS           # poisoned until the append rewrites them
        v16[blk, :, :, vp] = NAN_BITS
        q = torch.empty((T, self.hq, 128), dtype=torch.bfloat16, device=self.dev)
        q.normal_(generator=self.gen)
        out = torch.full((T, self.hq, 128), float("nan"), dtype=out_dtype, device=self.dev)
        ws = self.ws.ensure(m.workspace_bytes)
        _log(f"{label}: {m.num_units} units ({m.num_prefill_units} prefill), "
             f"splits {m.prefill_split_tokens}/{m.decode_split_tokens}")
        kb, vb = k_new.view(torch.bfloat16), v_new.view(torch.bfloat16)
        if fused:
            D.dlfp_append_attention_mixed(self.dims, m, st.d_work, d_bt, q, kb, vb, self.pool.k,
                                          self.pool.v, SCALE, out, ws)
        else:
            D.dlfp_kv_append(self.dims, kb, vb, st.d_slots, self.pool.k, self.pool.v)
            D.dlfp_attention_mixed(self.dims, m, st.d_work, d_bt, q, self.pool.k, self.pool.v,
                                   SCALE, out, ws)
        torch.cuda.synchronize()
        assert D.dlfp_workspace_error(ws) == 0, label
        assert not ws[:D.WORKSPACE_PARTIALS].view(torch.int32).cpu().numpy().any(), label
        assert bool(torch.isfinite(out).all()), label
        assert torch.equal(k16[blk, :, off, :], k_new), label
        assert torch.equal(v16[blk, :, :, vp], v_new), label
        cu = np.concatenate([[0], np.cumsum(q_len)])
        dec = [i for i, x in enumerate(its) if x[1] == 1]
        if dec:
            idx = torch.as_tensor(cu[dec], device=self.dev)
            q_dec, out_dec = q.view(torch.int16)[idx].cpu(), out[idx].float().cpu()
            for j, i in enumerate(dec):
                sid, _, kl = its[i]
                self.dec_rows[sid].append((ii, kl - 1, q_dec[j], out_dec[j]))
        for i, (sid, ql, kl) in enumerate(its):
            if ql > 1:
                pos0 = kl - ql
                rows = (list(range(ql)) if all_rows else
                        stratified_prompt_rows(m.work, m.num_prefill_units, i, pos0))
                r = torch.as_tensor(rows, device=self.dev) + int(cu[i])
                self.prompt_rows.append((ii, pos0 + np.asarray(rows),
                                         q.view(torch.int16)[r].cpu(), out[r].float().cpu()))

    def check(self):
        errs = {}   # (iteration, share) -> [abs errors]
        t0 = time.time()
        # prompt rows, iteration by iteration, over one gather of the prompt's pages
        if self.prompt_rows:
            n = max(int(pos.max()) for _, pos, _, _ in self.prompt_rows) + 1
            k, v = op.gather_pages(self.k_host, self.v_host, self.bt[self.n_dec], n)
            kf, vf = oa.bf16_bits_to_float64_tensor(k), oa.bf16_bits_to_float64_tensor(v)
            for ii, pos, q, out in self.prompt_rows:
                e = int(pos.max()) + 1
                want = oa.attention_rows(oa.bf16_bits_to_float64_tensor(q), kf[:e], vf[:e],
                                         SCALE, pos)
                errs.setdefault((ii, "prefill"), []).append(
                    np.abs(out.numpy().astype(np.float64) - want).ravel())
            _log(f"prompt rows checked in {time.time() - t0:.1f}s")
        # decoder rows, decoder by decoder, every iteration's row at once
        for d, recs in self.dec_rows.items():
            if not recs:
                continue
            pos = np.asarray([r[1] for r in recs])
            k, v = op.gather_pages(self.k_host, self.v_host, self.bt[d], int(pos.max()) + 1)
            q = oa.bf16_bits_to_float64_tensor(torch.stack([r[2] for r in recs]))
            want = oa.attention_rows(q, oa.bf16_bits_to_float64_tensor(k),
                                     oa.bf16_bits_to_float64_tensor(v), SCALE, pos)
            got = torch.stack([r[3] for r in recs]).numpy().astype(np.float64)
            for j, r in enumerate(recs):
                errs.setdefault((r[0], "decode"), []).append(np.abs(got[j] - want[j]).ravel())
            if d % 32 == 31:
                _log(f"decoders 0..{d} checked, {time.time() - t0:.1f}s")
        worst = {}
        for (ii, share), parts in sorted(errs.items()):
            e = np.concatenate(parts)
            mx, mean = float(e.max()), float(e.mean())
            kind = self.labels[ii].rsplit("out=", 1)[1]
            worst[kind] = max(worst.get(kind, 0.0), mx)
            assert mx <= MAX_ABS and mean <= MEAN_ABS, (self.labels[ii], share, mx, mean)
        _log(f"{self.cfg.name}: {len(errs)} (iteration, share) pairs within bounds, worst |err| "
             f"{', '.join(f'{k} output {v:.2e}' for k, v in sorted(worst.items()))}, {sum(len(r) for r in self.dec_rows.values())} decoder "
             f"rows, {sum(len(r[1]) for r in self.prompt_rows)} prompt rows")


def _first_mid_last(cfg, p):
    n = cfg.prompt_len // p
    return sorted({0, n // 2, n - 1})


def test_qwen3_0_6b_every_row_first_mid_last():
    f = FullSize(wl.qwen3_0_6b_config())
    for p in f.cfg.chunks:
        for c in _first_mid_last(f.cfg, p):
            f.run(p, c, all_rows=True)
    f.run(f.cfg.chunks[0], 3, prefill=False, all_rows=True, out_dtype=torch.float32)
    f.run(2048, 3, decoders=False, all_rows=True, out_dtype=torch.float32)
    f.run(512, 9, fused=False, all_rows=True, out_dtype=torch.float32)
    f.check()


def test_qwen3_8b_full_sweep():
    f = FullSize(wl.qwen3_8b_config())
    for p in f.cfg.chunks:
        for c in range(f.cfg.prompt_len // p):
            f.run(p, c)
    f.run(4096, 3, decoders=False, out_dtype=torch.float32)
    f.run(256, 5, prefill=False, out_dtype=torch.float32)
    f.run(1024, 5, fused=False, out_dtype=torch.float32)
    f.check()


def test_qwen3_32b_first_mid_last():
    f = FullSize(wl.qwen3_32b_config())
    for p in f.cfg.chunks:
        for c in _first_mid_last(f.cfg, p):
            f.run(p, c)
    f.run(8192, 3, decoders=False, out_dtype=torch.float32)
    f.run(512, 2, prefill=False, out_dtype=torch.float32)
    f.run(2048, 7, fused=False, out_dtype=torch.float32)
    f.check()

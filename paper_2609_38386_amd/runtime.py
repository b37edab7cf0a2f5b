"""Device-side plumbing around the C ABI: KV pools, per-iteration batches, workspace.

PyTorch supplies device memory and the stream; every step of the iteration
(metadata, KV append, attention, controller) is a libdlfp call.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import dlfp as _d

BF16_NAN_BITS = 0x7FC0


def bits_to_device(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns -> device bfloat16 tensor (same bits)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def device_to_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


class KVPool:
    """Paged KV cache of one layer: K [nb][Hkv][16][128], V [nb][Hkv][128][16] (bf16; the
    value page is transposed with slots 4-7 and 8-11 trading places)."""

    def __init__(self, num_blocks: int, num_kv_heads: int, device, fill_bits: Optional[int] = None):
        shape_k = (num_blocks, num_kv_heads, _d.PAGE_SIZE, _d.HEAD_DIM)
        shape_v = (num_blocks, num_kv_heads, _d.HEAD_DIM, _d.PAGE_SIZE)
        self.k = torch.empty(shape_k, dtype=torch.bfloat16, device=device)
        self.v = torch.empty(shape_v, dtype=torch.bfloat16, device=device)
        if fill_bits is not None:
            self.k.view(torch.int16).fill_(np.int16(np.uint16(fill_bits).view(np.int16)))
            self.v.view(torch.int16).fill_(np.int16(np.uint16(fill_bits).view(np.int16)))
        self.num_blocks = num_blocks
        self.num_kv_heads = num_kv_heads

    def host_bits(self):
        return device_to_bits(self.k), device_to_bits(self.v)


class Workspace:
    """Caller-owned split-K workspace, grown on demand; header and counters zeroed
    once per allocation (every launch leaves the counters zero again)."""

    def __init__(self, device, nbytes: int = 1 << 20, stream=None):
        self.device = device
        self.buf = None
        self._alloc(nbytes, stream)

    def _alloc(self, nbytes: int, stream=None):
        nbytes = max(int(nbytes), _d.WORKSPACE_PARTIALS)
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        _d.dlfp_workspace_init(self.buf, stream)

    def ensure(self, nbytes: int, num_groups: int = 0, stream=None) -> torch.Tensor:
        if self.buf.numel() < nbytes:
            self._alloc(int(nbytes * 1.25), stream)
        return self.buf


class Batch:
    """Metadata of one mixed iteration plus device copies of its arrays."""

    def __init__(self, dims: _d.dlfp_dims, q_len: Sequence[int], kv_len: Sequence[int],
                 block_table: np.ndarray, num_blocks: int, device,
                 tuning: Optional[_d.dlfp_tuning] = None, d_block_table: torch.Tensor = None):
        self.dims = dims
        self.q_len = np.asarray(q_len, dtype=np.int32)
        self.kv_len = np.asarray(kv_len, dtype=np.int32)
        self.meta = _d.dlfp_build_varlen_meta(dims, self.q_len, self.kv_len, block_table,
                                              num_blocks, tuning)
        m = self.meta
        self.num_tokens = m.num_tokens
        host = np.concatenate([m.slot_mapping[:m.num_tokens], m.records.reshape(-1)]
                              ).astype(np.int32)
        dev = torch.from_numpy(host).to(device)
        self.d_slots = dev[:m.num_tokens]
        self.d_work = dev[m.num_tokens:]
        if d_block_table is None:
            d_block_table = torch.from_numpy(np.ascontiguousarray(block_table, dtype=np.int32)
                                             ).to(device)
        self.d_block_table = d_block_table

    def append(self, pool: KVPool, k_new: torch.Tensor, v_new: torch.Tensor, stream=None):
        _d.dlfp_kv_append(self.dims, k_new, v_new, self.d_slots, pool.k, pool.v, stream)

    def attention(self, pool: KVPool, q: torch.Tensor, scale: float, out: torch.Tensor,
                  workspace: Workspace, stream=None):
        ws = workspace.ensure(self.meta.workspace_bytes, self.meta.num_groups, stream)
        _d.dlfp_attention_mixed(self.dims, self.meta, self.d_work, self.d_block_table, q,
                                pool.k, pool.v, scale, out, ws, stream)

    def append_attention(self, pool: KVPool, q: torch.Tensor, k_new: torch.Tensor,
                         v_new: torch.Tensor, scale: float, out: torch.Tensor,
                         workspace: Workspace, stream=None):
        ws = workspace.ensure(self.meta.workspace_bytes, self.meta.num_groups, stream)
        _d.dlfp_append_attention_mixed(self.dims, self.meta, self.d_work, self.d_block_table, q,
                                       k_new, v_new, pool.k, pool.v, scale, out, ws, stream)


class Iteration:
    """One mixed iteration over seeded logical sequences laid out in a fresh pool.

    ``seqs`` are ``workload.IterationSeq``: the iteration appends each
    sequence's last ``q_len`` tokens and attends with their queries; the
    earlier ``kv_len - q_len`` tokens (the cached prefix or decoder history)
    are written beforehand with the same append call.
    """

    def __init__(self, dims: _d.dlfp_dims, seqs, pool_blocks: int, seed: int, device,
                 fill_bits: Optional[int] = None, tuning: Optional[_d.dlfp_tuning] = None,
                 block_table: Optional[np.ndarray] = None):
        from . import workload as wl
        self.dims = dims
        self.seqs = list(seqs)
        self.device = device
        pages = [wl.pages_for(s.kv_len) for s in self.seqs]
        self.block_table = (block_table if block_table is not None
                            else wl.block_tables(seed, pages, pool_blocks))
        self.pool = KVPool(pool_blocks, dims.num_kv_heads, device, fill_bits)
        self._append_history()
        self.batch = Batch(dims, [s.q_len for s in self.seqs], [s.kv_len for s in self.seqs],
                           self.block_table, pool_blocks, device, tuning)
        self.q = bits_to_device(np.concatenate([s.stream.q[s.pos0:s.kv_len] for s in self.seqs]),
                                device)
        self.k_new = bits_to_device(
            np.concatenate([s.stream.k[s.pos0:s.kv_len] for s in self.seqs]), device)
        self.v_new = bits_to_device(
            np.concatenate([s.stream.v[s.pos0:s.kv_len] for s in self.seqs]), device)

    def _append_history(self):
        idx = [i for i, s in enumerate(self.seqs) if s.pos0 > 0]
        for i in idx:   # one sequence at a time keeps each history batch small
            s = self.seqs[i]
            hist = Batch(self.dims, [s.pos0], [s.pos0], self.block_table[i:i + 1],
                         self.pool.num_blocks, self.device)
            hist.append(self.pool, bits_to_device(s.stream.k[:s.pos0], self.device),
                        bits_to_device(s.stream.v[:s.pos0], self.device))

    def run(self, workspace: Workspace, scale: float, out_dtype=torch.bfloat16,
            append: bool = True, out: Optional[torch.Tensor] = None,
            fused: bool = False) -> torch.Tensor:
        """Append (unless `append` is false) and attend; `fused` does both in the one
        launch of dlfp_append_attention_mixed."""
        if out is None:
            out = torch.empty((self.batch.num_tokens, self.dims.num_q_heads, _d.HEAD_DIM),
                              dtype=out_dtype, device=self.device)
        if fused:
            if not append:
                raise ValueError("the fused launch always appends")
            self.batch.append_attention(self.pool, self.q, self.k_new, self.v_new, scale, out,
                                        workspace)
            return out
        if append:
            self.batch.append(self.pool, self.k_new, self.v_new)
        self.batch.attention(self.pool, self.q, scale, out, workspace)
        return out


class StagedBatch:
    """Per-iteration metadata with persistent buffers: the C builder fills host
    arrays, which are packed into one pinned buffer and copied to the device in a
    single stream-ordered transfer.  Reuse requires the previous iteration's copy
    to have completed (callers synchronise on iteration completion anyway)."""

    def __init__(self, dims: _d.dlfp_dims, cap_seqs: int, cap_tokens: int, cap_work: int, device,
                 tuning: Optional[_d.dlfp_tuning] = None):
        import ctypes
        self._ct = ctypes
        self.dims = dims
        self.tuning = tuning if tuning is not None else _d.dlfp_tuning(0, 0, 0)
        self.meta = _d.Meta(cap_seqs, cap_tokens, cap_work)
        total = cap_tokens + cap_work * _d.WORK_INTS
        self.host = torch.empty(total, dtype=torch.int32, pin_memory=True)
        self.host_np = self.host.numpy()
        self.dev = torch.empty(total, dtype=torch.int32, device=device)
        self.lib = _d.lib()

    def build(self, q_len: np.ndarray, kv_len: np.ndarray, block_table: np.ndarray,
              num_blocks: int, stream=None):
        ct = self._ct
        m = self.meta
        st = self.lib.dlfp_build_varlen_meta(
            ct.byref(self.dims), ct.byref(self.tuning), len(q_len), _d._ptr32(q_len),
            _d._ptr32(kv_len), _d._ptr32(block_table), block_table.shape[1], int(num_blocks),
            ct.byref(m.c))
        _d._check(st, "dlfp_build_varlen_meta")
        T, U = m.c.num_tokens, m.c.num_units + m.c.num_append
        h = self.host_np
        o = 0
        offs = []
        for arr, cnt in ((m.slot_mapping, T), (m.work_buf.reshape(-1), U * _d.WORK_INTS)):
            h[o:o + cnt] = arr[:cnt]
            offs.append((o, cnt))
            o += cnt
        self.dev[:o].copy_(self.host[:o], non_blocking=True)
        (d, nd), (e, ne) = offs
        self.d_slots = self.dev[d:d + nd]
        self.d_work = self.dev[e:e + ne]
        self.num_tokens = T
        return self

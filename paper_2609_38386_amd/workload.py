"""Seeded synthetic inputs for mixed continuous-batching iterations.

This module only *draws* inputs: bf16 query/key/value bit patterns, decoder
context lengths, physical page permutations and block tables, and the
per-iteration (q_len, kv_len) schedules of the chunk-size sweeps.  It holds
none of the attention, paging-address, metadata or controller arithmetic;
those live in the HIP library and, independently, in the oracle.

Shapes follow the attention layers of Qwen3-0.6B / 8B / 32B (head_dim 128,
8 KV heads, 16 / 32 / 64 query heads, 16-token KV pages).  The paper's own
workloads are synthetic exact-token sequences (Sec. 4.2, Sec. 9); here the
token stream is replaced by N(0,1) activations rounded to bf16, which is the
value distribution every configuration of the method's hot path is specified
with.

Every tensor comes from its own keyed PCG64 stream
``SeedSequence(seed, spawn_key=(role, index, tensor))`` so that a single
sequence can be regenerated on its own (the oracle never needs the whole KV
pool in memory), and streams are prefix-stable: the first ``n`` positions of a
sequence do not depend on how many positions were requested.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Sequence, Tuple

import numpy as np

HEAD_DIM = 128
PAGE_SIZE = 16

# Stream roles (first element of the spawn key).
ROLE_DECODER = 1
ROLE_PROMPT = 2
ROLE_CONTEXT_LENGTHS = 3
ROLE_PAGE_PERMUTATION = 4
ROLE_ARRIVALS = 5
ROLE_PROMPT_LENGTHS = 6

# Tensor ids (last element of the spawn key).
TENSOR_Q = 0
TENSOR_K = 1
TENSOR_V = 2


def rng_for(seed: int, *key: int) -> np.random.Generator:
    """Independent PCG64 generator for ``(seed, key...)``."""
    return np.random.Generator(
        np.random.PCG64(np.random.SeedSequence(int(seed), spawn_key=tuple(int(k) for k in key))))


def normal_bf16_bits(rng: np.random.Generator, shape) -> np.ndarray:
    """N(0,1) float32 samples rounded to nearest-even bf16; returns uint16 bits."""
    x = rng.standard_normal(size=shape, dtype=np.float32)
    u = x.view(np.uint32)
    u = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    return u.astype(np.uint16)


@dataclasses.dataclass(frozen=True)
class AttnShape:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int = HEAD_DIM
    page_size: int = PAGE_SIZE

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


@dataclasses.dataclass
class SeqStream:
    """Logical (unpaged) Q/K/V of one sequence over positions [0, length).

    Q row ``j`` is the query issued by the token at absolute position ``j``;
    K/V row ``j`` is that token's key/value.  Arrays are uint16 bf16 bits,
    Q ``[length][Hq][D]``, K and V ``[length][Hkv][D]``.
    """

    seed: int
    role: int
    index: int
    shape: AttnShape
    length: int

    def __post_init__(self):
        self._cache: Dict[int, np.ndarray] = {}

    def _tensor(self, tensor: int) -> np.ndarray:
        if tensor not in self._cache:
            heads = self.shape.num_q_heads if tensor == TENSOR_Q else self.shape.num_kv_heads
            rng = rng_for(self.seed, self.role, self.index, tensor)
            self._cache[tensor] = normal_bf16_bits(rng, (self.length, heads, self.shape.head_dim))
        return self._cache[tensor]

    @property
    def q(self) -> np.ndarray:
        return self._tensor(TENSOR_Q)

    @property
    def k(self) -> np.ndarray:
        return self._tensor(TENSOR_K)

    @property
    def v(self) -> np.ndarray:
        return self._tensor(TENSOR_V)


def pages_for(n_tokens: int, page_size: int = PAGE_SIZE) -> int:
    return (int(n_tokens) + page_size - 1) // page_size


def block_tables(seed: int, pages_per_seq: Sequence[int], pool_blocks: int,
                 max_blocks: int | None = None) -> np.ndarray:
    """Block tables drawn from one seeded permutation of the pool.

    Sequence ``s`` receives the next ``pages_per_seq[s]`` entries of the
    permutation, in sequence order.  Unused table entries are -1.
    """
    need = int(sum(pages_per_seq))
    if need > pool_blocks:
        raise ValueError(f"pool of {pool_blocks} blocks cannot hold {need} pages")
    width = int(max(pages_per_seq)) if max_blocks is None else int(max_blocks)
    perm = rng_for(seed, ROLE_PAGE_PERMUTATION).permutation(pool_blocks).astype(np.int32)
    bt = np.full((len(pages_per_seq), max(width, 1)), -1, dtype=np.int32)
    off = 0
    for s, n in enumerate(pages_per_seq):
        bt[s, :n] = perm[off:off + n]
        off += n
    return bt


@dataclasses.dataclass
class IterationSeq:
    """One sequence of a mixed iteration: ``q_len`` new tokens, ``kv_len`` total."""

    stream: SeqStream
    q_len: int
    kv_len: int

    @property
    def pos0(self) -> int:
        return self.kv_len - self.q_len


@dataclasses.dataclass
class SweepConfig:
    """A chunk-size sweep: |D| decoders beside one prompt prefilled in chunks."""

    name: str
    shape: AttnShape
    n_decoders: int
    ctx_lo: int
    ctx_hi: int
    prompt_len: int
    chunks: Tuple[int, ...]
    layers: int
    seed: int = 801
    pool_blocks: int | None = None  # None: exactly what the sweep needs

    def decoder_contexts(self) -> np.ndarray:
        """Initial decoder context lengths (kv_len incl. the token decoded now)."""
        rng = rng_for(self.seed, ROLE_CONTEXT_LENGTHS)
        return rng.integers(self.ctx_lo, self.ctx_hi, size=self.n_decoders,
                            endpoint=True).astype(np.int64)

    def max_decode_steps(self) -> int:
        """Most chunk iterations any sweep point runs (decoders grow by one per iteration)."""
        return max(self.prompt_len // p for p in self.chunks)

    def decoder_streams(self) -> List[SeqStream]:
        ctx = self.decoder_contexts()
        grow = self.max_decode_steps()
        return [SeqStream(self.seed, ROLE_DECODER, i, self.shape, int(c) + grow)
                for i, c in enumerate(ctx)]

    def prompt_stream(self) -> SeqStream:
        return SeqStream(self.seed, ROLE_PROMPT, 0, self.shape, self.prompt_len)

    def pages_per_seq(self) -> List[int]:
        """Pages each sequence needs over the whole sweep: decoders first, then the prompt."""
        ctx = self.decoder_contexts()
        grow = self.max_decode_steps()
        return [pages_for(int(c) + grow, self.shape.page_size) for c in ctx] + \
               [pages_for(self.prompt_len, self.shape.page_size)]

    def pool_size(self) -> int:
        return int(self.pool_blocks) if self.pool_blocks else int(sum(self.pages_per_seq()))

    def iteration(self, p: int, chunk_index: int, decoders_first: bool = False
                  ) -> List[Tuple[int, int, int]]:
        """(sequence id, q_len, kv_len) of chunk iteration ``chunk_index`` at chunk size ``p``.

        Sequence ids: 0..n_decoders-1 are decoders, n_decoders is the prompt.
        Iteration ``c`` prefills prompt tokens [c*p, (c+1)*p) and decodes one
        token per decoder, whose context has grown by ``c`` since the start.
        """
        ctx = self.decoder_contexts()
        prompt = [(self.n_decoders, p, (chunk_index + 1) * p)]
        dec = [(i, 1, int(ctx[i]) + chunk_index) for i in range(self.n_decoders)]
        return dec + prompt if decoders_first else prompt + dec


def tiny_config() -> SweepConfig:
    """Tiny mixed iteration: 4 decoders (context 64-256) + a 128-token chunk at offset 384.

    The described 64-block pool cannot hold the worst case (decoders up to 16
    pages each plus 32 prompt pages), so the pool has 128 blocks.
    """
    return SweepConfig("tiny", AttnShape(16, 8), n_decoders=4, ctx_lo=64, ctx_hi=256,
                       prompt_len=512, chunks=(128,), layers=1, pool_blocks=128)


def qwen3_0_6b_config() -> SweepConfig:
    return SweepConfig("qwen3-0.6b", AttnShape(16, 8), n_decoders=32, ctx_lo=512,
                       ctx_hi=2048, prompt_len=8192,
                       chunks=(64, 128, 256, 512, 1024, 2048), layers=28)


def qwen3_8b_config() -> SweepConfig:
    return SweepConfig("qwen3-8b", AttnShape(32, 8), n_decoders=128, ctx_lo=1024,
                       ctx_hi=8192, prompt_len=16384,
                       chunks=(256, 512, 1024, 2048, 4096), layers=36)


def qwen3_32b_config() -> SweepConfig:
    return SweepConfig("qwen3-32b", AttnShape(64, 8), n_decoders=256, ctx_lo=2048,
                       ctx_hi=32768, prompt_len=32768,
                       chunks=(512, 1024, 2048, 4096, 8192), layers=1)


CONFIGS = {
    "tiny": tiny_config,
    "qwen3-0.6b": qwen3_0_6b_config,
    "qwen3-8b": qwen3_8b_config,
    "qwen3-32b": qwen3_32b_config,
}


def tiny_iteration(cfg: SweepConfig | None = None) -> List[IterationSeq]:
    """The single mixed iteration of the tiny configuration (chunk 128 at offset 384)."""
    cfg = cfg or tiny_config()
    dec = cfg.decoder_streams()
    prompt = cfg.prompt_stream()
    ctx = cfg.decoder_contexts()
    out = [IterationSeq(prompt, 128, 512)]
    out += [IterationSeq(dec[i], 1, int(ctx[i])) for i in range(cfg.n_decoders)]
    return out


# --------------------------------------------------------------------------- replay arrivals

def poisson_arrivals(seed: int, n: int, rate_per_s: float) -> np.ndarray:
    """Open-loop arrival times (seconds) with independent exponential gaps."""
    gaps = rng_for(seed, ROLE_ARRIVALS).exponential(1.0 / rate_per_s, size=n)
    return np.cumsum(gaps)


def prompt_lengths(seed: int, n: int, lo: int, hi: int) -> np.ndarray:
    return rng_for(seed, ROLE_PROMPT_LENGTHS).integers(lo, hi, size=n, endpoint=True)

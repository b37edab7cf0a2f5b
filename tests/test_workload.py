"""Seeded input generator: determinism, prefix stability, bf16 rounding and pool placement."""
import numpy as np
import torch

from paper_2609_38386_amd import workload as wl


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    rng = wl.rng_for(1, 99)
    bits = wl.normal_bf16_bits(rng, (50000,))
    x = wl.rng_for(1, 99).standard_normal(size=(50000,), dtype=np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)


def test_streams_deterministic_and_prefix_stable():
    shape = wl.AttnShape(16, 8)
    a = wl.SeqStream(801, wl.ROLE_DECODER, 3, shape, 100)
    b = wl.SeqStream(801, wl.ROLE_DECODER, 3, shape, 40)
    c = wl.SeqStream(801, wl.ROLE_DECODER, 4, shape, 40)
    assert np.array_equal(a.k[:40], b.k) and np.array_equal(a.v[:40], b.v)
    assert np.array_equal(a.q[:40], b.q)
    assert not np.array_equal(b.k, c.k)
    assert not np.array_equal(b.k, b.v)


def test_block_tables_are_disjoint_pool_draws():
    bt = wl.block_tables(801, [3, 5, 1], 16)
    used = [int(x) for x in bt.ravel() if x >= 0]
    assert len(used) == 9 and len(set(used)) == 9
    assert all(0 <= x < 16 for x in used)
    assert (bt[2, 1:] == -1).all()


def test_config_recipes():
    tiny = wl.tiny_config()
    ctx = tiny.decoder_contexts()
    assert len(ctx) == 4 and ctx.min() >= 64 and ctx.max() <= 256
    assert tiny.pool_size() == 128 and sum(tiny.pages_per_seq()) <= 128
    c1 = wl.qwen3_0_6b_config()
    ctx = c1.decoder_contexts()
    assert ctx.min() >= 512 and ctx.max() <= 2048
    its = c1.iteration(2048, 3)
    assert its[0] == (32, 2048, 8192)
    assert all(q == 1 for _, q, _ in its[1:])
    assert its[1][2] == int(ctx[0]) + 3

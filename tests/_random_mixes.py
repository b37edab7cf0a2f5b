"""Seeded random iteration mixes, shared by the CPU check of the metadata
builder and the GPU parity test of the same cases.

A case: the GQA group g and KV-head count, a ragged mix of decoders (one new
token over 1-3000 keys; none in about a sixth of the cases) and prompt chunks (1-600 new tokens over a cached
prefix of 0-2400 tokens; a 1-token chunk takes the decode path), in random
order, and a random dlfp_tuning that the builder accepts (decode and prefill
splits, resident-wavefront target, tile height, grid layout, page depth, each
automatic about half the time), the one-launch or two-launch form and the
output type.  Sequence s's pages come from wl.block_tables(seed(i), pages,
pool(pages)), as rt.Iteration lays them out.
"""
import os

import numpy as np

# Cases the tests run; DLFP_RANDOM_MIXES raises it for a longer sweep.
CASES = int(os.environ.get("DLFP_RANDOM_MIXES", "24"))


def seed(i):
    return 7000 + i


def pool(pages, extra=7):
    return int(sum(pages)) + extra


def case(i):
    rng = np.random.default_rng(5000 + i)
    g = [1, 2, 4, 8][i % 4]
    hkv = int(rng.choice([1, 2, 4, 8]))
    hkv = min(hkv, 64 // g)
    n_dec = int(rng.integers(0, 33)) if rng.random() >= 1 / 6 else 0
    n_pre = int(rng.integers(0 if n_dec else 1, 4))
    specs = [(1, int(rng.integers(1, 3001))) for _ in range(n_dec)]
    for _ in range(n_pre):
        q = int(rng.integers(1, 601))
        specs.append((q, q + int(rng.integers(0, 2401))))
    specs = [specs[j] for j in rng.permutation(len(specs))]

    def maybe(value):
        return int(value) if rng.random() < 0.5 else 0

    tuning = (maybe(16 * rng.integers(1, 257)),          # decode split, keys
              maybe(64 * rng.integers(1, 65)),           # prefill split, keys
              maybe(rng.choice([256, 1024, 4096])),      # resident wavefronts
              maybe(rng.integers(1, 128 // g + 1)),      # prompt tokens per tile
              int(rng.choice([0, 0, -1, int(rng.integers(1, 600))])),  # lead units
              int(rng.integers(0, 3)))                   # decode pages in flight
    fused = bool(rng.integers(0, 2))
    fp32_out = bool(rng.integers(0, 2))
    return g, hkv, specs, tuning, fused, fp32_out

"""Pins for the attention oracle, parameterised over the implementation under test.

Each check raises AssertionError when ``impl`` (a function with the signature
of ``oracle.attention.attention_sequence``, or of ``attention_rows`` for the
rows checks) disagrees with something fixed
independently of it: brute force in pure-Python float arithmetic, closed forms,
a library routine, or an invariant of masked softmax attention over a cached
prefix.  The mutation test runs these same checks against deliberately broken
copies of the oracle and requires each copy to fail at least one of them.
"""
from __future__ import annotations

import math

import numpy as np
import torch


def _rand(rng, *shape, scale=1.0):
    return rng.standard_normal(shape) * scale


def brute_force_attention(q, k, v, scale):
    """Pure-Python loops with math.exp: one row, one head, one key at a time."""
    q_len, hq, d = q.shape
    n, hkv, _ = k.shape
    g = hq // hkv
    out = np.zeros((q_len, hq, d))
    for i in range(q_len):
        pos = n - q_len + i
        for h in range(hq):
            kh = h // g
            scores = []
            for j in range(pos + 1):
                acc = 0.0
                for t in range(d):
                    acc += float(q[i, h, t]) * float(k[j, kh, t])
                scores.append(scale * acc)
            mx = max(scores)
            ws = [math.exp(x - mx) for x in scores]
            tot = sum(ws)
            for t in range(d):
                acc = 0.0
                for j, w in enumerate(ws):
                    acc += w * float(v[j, kh, t])
                out[i, h, t] = acc / tot
    return out


def check_brute_force(impl):
    rng = np.random.default_rng(11)
    for (q_len, n, hq, hkv, d) in [(1, 1, 1, 1, 4), (3, 5, 2, 1, 4), (4, 8, 4, 2, 4),
                                   (2, 7, 2, 2, 128), (8, 8, 2, 1, 16)]:
        q = _rand(rng, q_len, hq, d)
        k = _rand(rng, n, hkv, d)
        v = _rand(rng, n, hkv, d)
        scale = 1.0 / math.sqrt(d)
        got = impl(q, k, v, scale)
        want = brute_force_attention(q, k, v, scale)
        assert np.allclose(got, want, rtol=0, atol=1e-12), (q_len, n, hq, hkv, d)


def check_large_scores(impl):
    """Scores near 700 overflow exp() unless the row maximum is subtracted first."""
    rng = np.random.default_rng(12)
    q = _rand(rng, 2, 2, 4) * 30.0
    k = _rand(rng, 5, 1, 4) * 30.0
    v = _rand(rng, 5, 1, 4)
    got = impl(q, k, v, 1.0)
    want = brute_force_attention(q, k, v, 1.0)
    assert np.all(np.isfinite(got))
    assert np.allclose(got, want, rtol=0, atol=1e-9)


def check_closed_forms(impl):
    rng = np.random.default_rng(13)
    d = 128
    # A prompt's first token (nothing cached) sees only itself: o = v_0 exactly.
    q = _rand(rng, 6, 4, d)
    k = _rand(rng, 6, 2, d)
    v = _rand(rng, 6, 2, d)
    out = impl(q, k, v, 0.088)
    for h in range(4):
        assert np.array_equal(out[0, h], v[0, h // 2])
    # Zero query: uniform weights over the visible keys -> mean of visible values.
    q = np.zeros((3, 2, d))
    k = _rand(rng, 10, 1, d)
    v = _rand(rng, 10, 1, d)
    out = impl(q, k, v, 0.088)
    for i in range(3):
        vis = 10 - 3 + i + 1
        assert np.allclose(out[i, 0], v[:vis, 0].mean(axis=0), atol=1e-12)
        assert np.allclose(out[i, 1], v[:vis, 0].mean(axis=0), atol=1e-12)
    # Identical value rows: any convex combination returns that row.
    q = _rand(rng, 4, 2, d)
    k = _rand(rng, 9, 2, d)
    row = _rand(rng, 2, d)
    v = np.broadcast_to(row, (9, 2, d)).copy()
    out = impl(q, k, v, 0.5)
    for h in range(2):
        assert np.allclose(out[:, h], row[h], atol=1e-12)


def check_library_sdpa(impl):
    """GQA as MHA over KV heads repeated per group, via torch's SDPA with an explicit
    bottom-right causal mask (torch's own causal flag is top-left when lengths differ)."""
    rng = np.random.default_rng(14)
    for (q_len, n, hq, hkv) in [(5, 21, 4, 2), (1, 33, 8, 2), (16, 16, 2, 2), (7, 40, 8, 1)]:
        d = 128
        q = _rand(rng, q_len, hq, d)
        k = _rand(rng, n, hkv, d)
        v = _rand(rng, n, hkv, d)
        scale = 1.0 / math.sqrt(d)
        g = hq // hkv
        tq = torch.from_numpy(q).permute(1, 0, 2)[None]
        tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)[None]
        tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)[None]
        mask = torch.ones(q_len, n, dtype=torch.bool).tril(diagonal=n - q_len)
        ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask,
                                                               scale=scale)
        ref = ref[0].permute(1, 0, 2).numpy()
        got = impl(q, k, v, scale)
        assert np.allclose(got, ref, rtol=0, atol=1e-10), (q_len, n, hq, hkv)


def check_chunking_invariance(impl):
    """Any split of a prompt into chunks over its cached prefix equals unchunked prefill."""
    rng = np.random.default_rng(15)
    n, hq, hkv, d = 70, 4, 2, 128
    q = _rand(rng, n, hq, d)
    k = _rand(rng, n, hkv, d)
    v = _rand(rng, n, hkv, d)
    full = impl(q, k, v, 0.088)
    for cuts in ([0, 16, 33, 34, 70], [0, 1, 2, 69, 70], [0, 64, 70]):
        for a, b in zip(cuts, cuts[1:]):
            part = impl(q[a:b], k[:b], v[:b], 0.088)
            assert np.allclose(part, full[a:b], rtol=0, atol=1e-12), (cuts, a, b)


def check_decode_equals_last_prefill_row(impl):
    rng = np.random.default_rng(16)
    n, hq, hkv, d = 45, 8, 2, 128
    q = _rand(rng, 12, hq, d)
    k = _rand(rng, n, hkv, d)
    v = _rand(rng, n, hkv, d)
    pre = impl(q, k, v, 0.088)
    dec = impl(q[-1:], k, v, 0.088)
    assert np.allclose(dec[0], pre[-1], rtol=0, atol=1e-12)


def brute_force_rows(q, k, v, scale, positions):
    """Pure-Python loops: row r, at absolute position positions[r], sees keys 0..positions[r]."""
    r_n, hq, d = q.shape
    _, hkv, _ = k.shape
    g = hq // hkv
    out = np.zeros((r_n, hq, d))
    for r in range(r_n):
        for h in range(hq):
            kh = h // g
            scores = [scale * sum(float(q[r, h, t]) * float(k[j, kh, t]) for t in range(d))
                      for j in range(int(positions[r]) + 1)]
            mx = max(scores)
            ws = [math.exp(x - mx) for x in scores]
            tot = sum(ws)
            for t in range(d):
                out[r, h, t] = sum(w * float(v[j, kh, t]) for j, w in enumerate(ws)) / tot
    return out


def check_rows_brute_force(rows_impl):
    """Rows at arbitrary positions (out of order, repeated, the first and the last key)."""
    rng = np.random.default_rng(17)
    for (n, hq, hkv, d, pos) in [(9, 4, 2, 4, [8, 0, 3, 3, 5]), (6, 2, 1, 16, [5, 1]),
                                 (12, 8, 2, 8, [11, 7, 0])]:
        q = _rand(rng, len(pos), hq, d)
        k = _rand(rng, n, hkv, d)
        v = _rand(rng, n, hkv, d)
        got = rows_impl(q, k, v, 0.3, pos)
        want = brute_force_rows(q, k, v, 0.3, pos)
        assert np.allclose(got, want, rtol=0, atol=1e-12), (n, hq, hkv, pos)


ALL_CHECKS = [check_brute_force, check_large_scores, check_closed_forms, check_library_sdpa,
              check_chunking_invariance, check_decode_equals_last_prefill_row]

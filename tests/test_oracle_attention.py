"""Oracle attention pinned against brute force, closed forms, a library routine and invariants."""
import numpy as np
import pytest

from oracle import attention as oa
from oracle import paging
from paper_2609_38386_amd import workload as wl

from _attention_pins import (brute_force_attention, check_brute_force, check_chunking_invariance,
                             check_closed_forms, check_decode_equals_last_prefill_row,
                             check_large_scores, check_library_sdpa, check_rows_brute_force)


def test_brute_force():
    check_brute_force(oa.attention_sequence)


def test_large_scores_need_max_subtraction():
    check_large_scores(oa.attention_sequence)


def test_closed_forms():
    check_closed_forms(oa.attention_sequence)


def test_library_sdpa_gqa_as_repeated_mha():
    check_library_sdpa(oa.attention_sequence)


def test_chunking_invariance():
    check_chunking_invariance(oa.attention_sequence)


def test_decode_row_equals_last_prefill_row():
    check_decode_equals_last_prefill_row(oa.attention_sequence)


def test_row_subset_matches_full():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((9, 4, 128))
    k = rng.standard_normal((30, 2, 128))
    v = rng.standard_normal((30, 2, 128))
    full = oa.attention_sequence(q, k, v, 0.1)
    sub = oa.attention_sequence(q, k, v, 0.1, rows=[0, 4, 8])
    assert np.allclose(sub, full[[0, 4, 8]], rtol=0, atol=1e-13)


def test_bf16_widening_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x7F7F, 0x0001], dtype=np.uint16)
    got = oa.bf16_bits_to_float64(bits)
    assert got[0] == 1.0 and got[1] == -1.0 and got[3] == 0.0
    assert got[2] == 3.140625
    assert np.signbit(got[4])
    assert got[5] == float.fromhex("0x1.fep127")
    assert got[6] == float.fromhex("0x1p-133")


def _scatter(logical_k, logical_v, block_row, pool_blocks):
    """Test-side writer of the pool layout (token rows for K, transposed pages for V)."""
    n, hkv, d = logical_k.shape
    kc = np.zeros((pool_blocks, hkv, 16, d), dtype=np.uint16)
    vc = np.zeros((pool_blocks, hkv, d, 16), dtype=np.uint16)
    for j in range(n):
        b = block_row[j // 16]
        kc[b, :, j % 16, :] = logical_k[j]
        vc[b, :, :, paging.value_position(j % 16)] = logical_v[j]
    return kc, vc


def test_gather_hand_example():
    """Element (block b, head h, slot t, dim d) holds 1000b + 100h + t for K (and + 50 for V)."""
    nb, hkv, d = 4, 2, 3
    kc = np.zeros((nb, hkv, 16, d), dtype=np.uint16)
    vc = np.zeros((nb, hkv, d, 16), dtype=np.uint16)
    for b in range(nb):
        for h in range(hkv):
            for t in range(16):
                kc[b, h, t, :] = 1000 * b + 100 * h + t
                vc[b, h, :, paging.value_position(t)] = 1000 * b + 100 * h + t + 50
    k, v = paging.gather_sequence(kc, vc, np.array([3, 1]), 20)
    # token 0 -> block 3 slot 0; token 15 -> block 3 slot 15; token 17 -> block 1 slot 1
    assert k[0, 0, 0] == 3000 and k[15, 1, 2] == 3115 and k[17, 0, 1] == 1001
    assert v[17, 1, 0] == 1151 and v[19, 0, 2] == 1053


def test_value_page_slot_order_is_the_declared_one():
    """A value page row stores token slot t at position pi(t), pi trading slots 4-7
    with 8-11 (bits 2 and 3 of t swapped), as the pool layout declares."""
    assert [paging.value_position(t) for t in range(16)] == \
        [0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15]
    assert all(paging.value_position(paging.value_position(t)) == t for t in range(16))
    # a gather through a literal page, written without value_position
    vc = np.zeros((1, 1, 1, 16), dtype=np.uint16)
    vc[0, 0, 0] = [0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15]
    kc = np.zeros((1, 1, 16, 1), dtype=np.uint16)
    _, v = paging.gather_sequence(kc, vc, np.array([0]), 16)
    assert v[:, 0, 0].tolist() == list(range(16))


def test_page_permutation_invariance():
    """Two different physical placements gather to the same bits, hence the same outputs."""
    shape = wl.AttnShape(4, 2)
    st = wl.SeqStream(5, wl.ROLE_DECODER, 0, shape, 53)
    outs = []
    for seed in (1, 2):
        bt = wl.block_tables(seed, [wl.pages_for(53)], 16)[0]
        kc, vc = _scatter(st.k, st.v, bt, 16)
        k, v = paging.gather_sequence(kc, vc, bt, 53)
        assert np.array_equal(k, st.k) and np.array_equal(v, st.v)
        outs.append(oa.attention_sequence(oa.bf16_bits_to_float64(st.q[-7:]),
                                          oa.bf16_bits_to_float64(k),
                                          oa.bf16_bits_to_float64(v), 0.088))
    assert np.array_equal(outs[0], outs[1])


def test_rows_at_positions_brute_force():
    check_rows_brute_force(oa.attention_rows)


def test_rows_of_several_iterations_share_one_key_tensor():
    """A decoder row at position j over a key tensor that runs past j equals the
    row over exactly its j + 1 keys: keys beyond a row's position are invisible."""
    rng = np.random.default_rng(8)
    k = rng.standard_normal((40, 2, 128))
    v = rng.standard_normal((40, 2, 128))
    q = rng.standard_normal((3, 8, 128))
    got = oa.attention_rows(q, k, v, 0.088, [10, 25, 39])
    for r, j in enumerate([10, 25, 39]):
        want = brute_force_attention(q[r:r + 1], k[:j + 1], v[:j + 1], 0.088)
        assert np.allclose(got[r], want[0], rtol=0, atol=1e-12)


def test_rows_reject_positions_outside_the_sequence():
    z = np.zeros((2, 2, 8))
    with pytest.raises(ValueError):
        oa.attention_rows(z, np.zeros((4, 1, 8)), np.zeros((4, 1, 8)), 1.0, [0, 4])
    with pytest.raises(ValueError):
        oa.attention_rows(z, np.zeros((4, 1, 8)), np.zeros((4, 1, 8)), 1.0, [-1, 2])


def test_bf16_widening_tensor_matches_numpy():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x7F7F, 0x0001, 0x7FC0],
                    dtype=np.uint16)
    t = oa.bf16_bits_to_float64_tensor(bits).numpy()
    n = oa.bf16_bits_to_float64(bits)
    assert t[2] == 3.140625 and t[6] == float.fromhex("0x1p-133") and np.isnan(t[7])
    assert np.array_equal(t[:7], n[:7])
    import torch
    tt = oa.bf16_bits_to_float64_tensor(torch.from_numpy(bits.view(np.int16))).numpy()
    assert np.array_equal(tt[:7], n[:7])


def test_gather_pages_hand_example():
    nb, hkv, d = 4, 2, 3
    kc = np.zeros((nb, hkv, 16, d), dtype=np.uint16)
    vc = np.zeros((nb, hkv, d, 16), dtype=np.uint16)
    for b in range(nb):
        for h in range(hkv):
            for t in range(16):
                kc[b, h, t, :] = 1000 * b + 100 * h + t
                vc[b, h, :, paging.value_position(t)] = 1000 * b + 100 * h + t + 50
    k, v = paging.gather_pages(kc, vc, np.array([3, 1]), 20)
    assert k.shape == (20, 2, 3) and v.shape == (20, 2, 3)
    assert k[0, 0, 0] == 3000 and k[15, 1, 2] == 3115 and k[17, 0, 1] == 1001
    assert v[17, 1, 0] == 1151 and v[19, 0, 2] == 1053
    # slot 5 of a value row sits at position 9, slot 9 at 5 (bits 2 and 3 swap)
    assert v[5, 0, 0] == 3055 and v[9, 0, 0] == 3059


@pytest.mark.parametrize("n", [1, 15, 16, 17, 100, 161])
def test_gather_pages_equals_token_loop(n):
    import torch
    rng = np.random.default_rng(n)
    nb, hkv, d = 24, 3, 8
    kc = rng.integers(0, 1 << 16, size=(nb, hkv, 16, d), dtype=np.uint16)
    vc = rng.integers(0, 1 << 16, size=(nb, hkv, d, 16), dtype=np.uint16)
    row = rng.permutation(nb)[:(n + 15) // 16]
    k0, v0 = paging.gather_sequence(kc, vc, row, n)
    k1, v1 = paging.gather_pages(kc, vc, row, n)
    assert np.array_equal(k0, k1) and np.array_equal(v0, v1)
    kt, vt = paging.gather_pages(torch.from_numpy(kc.view(np.int16)),
                                 torch.from_numpy(vc.view(np.int16)), row, n)
    assert np.array_equal(kt.numpy().view(np.uint16), k0)
    assert np.array_equal(vt.numpy().view(np.uint16), v0)


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oa.attention_sequence(np.zeros((2, 3, 8)), np.zeros((4, 2, 8)), np.zeros((4, 2, 8)), 1.0)
    with pytest.raises(ValueError):
        oa.attention_sequence(np.zeros((5, 2, 8)), np.zeros((4, 2, 8)), np.zeros((4, 2, 8)), 1.0)

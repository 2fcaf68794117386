"""Pins of the float64 paged decode attention oracle.

Each test checks the oracle against something other than itself: torch's own
scaled-dot-product attention on the contiguous cache (a library routine), closed
forms, special cases and symmetry. The paged inputs are packed by the input
generator's byte-format code, which is written separately from the oracle's
layout decoder, so a layout slip on either side fails here.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from synth import random_16bit, round_to_16bit, pack_block, LAYOUT_ATTN, NAN16, element_index


def build_paged(rng, lens, hkv, d, bs, dtype, tail=None):
    """Random contiguous K/V per sequence, packed into blocks at scattered
    physical ids. Returns (pool, table, K list, V list) where K/V are the
    logical uint16 [Hkv][len][D] of each sequence."""
    nblk = [(int(n) + bs - 1) // bs for n in lens]
    total = sum(nblk)
    perm = rng.permutation(max(total, 1))
    pool = np.zeros((max(total, 1), 2 * bs * hkv * d * 2), dtype=np.uint8)
    table = np.full((len(lens), max(max(nblk), 1)), -1, dtype=np.int64)
    Ks, Vs, k = [], [], 0
    for b, n in enumerate(lens):
        K = random_16bit(rng, (hkv, nblk[b] * bs, d), dtype)
        V = random_16bit(rng, (hkv, nblk[b] * bs, d), dtype)
        if tail is not None:
            K[:, n:] = tail
            V[:, n:] = tail
        Ks.append(K[:, :n])
        Vs.append(V[:, :n])
        for j in range(nblk[b]):
            u = perm[k]
            k += 1
            table[b, j] = u
            pool[u] = pack_block(K[:, j * bs:(j + 1) * bs], V[:, j * bs:(j + 1) * bs], LAYOUT_ATTN)
    return pool, table, Ks, Vs


def sdpa_reference(q64, K64, V64):
    """torch SDPA (float64, CPU) on the contiguous cache; GQA by repeating kv heads."""
    hq, d = q64.shape
    hkv = K64.shape[0]
    if K64.shape[1] == 0:
        return np.zeros((hq, d))
    g = hq // hkv
    Kr = torch.from_numpy(K64).repeat_interleave(g, dim=0)
    Vr = torch.from_numpy(V64).repeat_interleave(g, dim=0)
    q = torch.from_numpy(q64)[:, None, :]
    return F.scaled_dot_product_attention(q, Kr, Vr)[:, 0, :].numpy()


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("hq,hkv,bs", [(8, 8, 16), (32, 8, 16), (8, 1, 32), (4, 2, 64)])
def test_paged_matches_torch_sdpa_on_contiguous_cache(dtype, hq, hkv, bs):
    rng = np.random.default_rng(1 + hq + bs)
    d = 128
    lens = [1, bs - 1, bs, bs + 1, 3 * bs + 7, int(rng.integers(1, 200))]
    pool, table, Ks, Vs = build_paged(rng, lens, hkv, d, bs, dtype)
    q16 = random_16bit(rng, (len(lens), hq, d), dtype)
    out = oracle.paged_decode_attention(q16, table, lens, lambda u: pool[u], hkv, d, bs, dtype)
    q64 = oracle.to_float64(q16, dtype)
    for b in range(len(lens)):
        ref = sdpa_reference(q64[b], oracle.to_float64(Ks[b], dtype), oracle.to_float64(Vs[b], dtype))
        np.testing.assert_allclose(out[b], ref, rtol=1e-12, atol=1e-13)


def test_len_one_returns_first_value_row():
    rng = np.random.default_rng(2)
    pool, table, Ks, Vs = build_paged(rng, [1], 2, 128, 16, "bf16")
    q16 = random_16bit(rng, (1, 4, 128), "bf16")
    out = oracle.paged_decode_attention(q16, table, [1], lambda u: pool[u], 2, 128, 16, "bf16")
    V = oracle.to_float64(Vs[0], "bf16")
    for h in range(4):
        np.testing.assert_array_equal(out[0, h], V[h // 2, 0])


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(3)
    n = 77
    pool, table, Ks, Vs = build_paged(rng, [n], 1, 128, 16, "f16")
    q16 = np.zeros((1, 1, 128), dtype=np.uint16)
    out = oracle.paged_decode_attention(q16, table, [n], lambda u: pool[u], 1, 128, 16, "f16")
    V = oracle.to_float64(Vs[0], "f16")
    np.testing.assert_allclose(out[0, 0], V[0].mean(axis=0), rtol=1e-13, atol=1e-15)


def test_equal_keys_give_mean_of_values():
    rng = np.random.default_rng(4)
    n = 40
    pool, table, Ks, Vs = build_paged(rng, [n], 1, 128, 16, "bf16")
    k_row = random_16bit(rng, (128,), "bf16")
    Kfix = np.broadcast_to(k_row, (1, 48, 128)).copy()
    Vfull = np.zeros((1, 48, 128), dtype=np.uint16)
    Vfull[:, :n] = Vs[0]
    for j in range(3):
        pool[table[0, j]] = pack_block(Kfix[:, 16 * j:16 * j + 16], Vfull[:, 16 * j:16 * j + 16],
                                       LAYOUT_ATTN)
    q16 = random_16bit(rng, (1, 1, 128), "bf16")
    out = oracle.paged_decode_attention(q16, table, [n], lambda u: pool[u], 1, 128, 16, "bf16")
    np.testing.assert_allclose(out[0, 0], oracle.to_float64(Vs[0], "bf16")[0].mean(axis=0),
                               rtol=1e-13, atol=1e-15)


def test_dominant_logit_selects_its_value_row():
    rng = np.random.default_rng(5)
    n, t0 = 50, 23
    pool, table, Ks, Vs = build_paged(rng, [n], 1, 128, 16, "f16")
    q = np.zeros(128, dtype=np.float32)
    q[7] = 64.0
    K = np.zeros((1, 64, 128), dtype=np.float32)
    K[0, t0, 7] = 64.0          # logit 64*64/sqrt(128) ~ 362 against 0 for the rest
    Kb = round_to_16bit(K, "f16")
    Vfull = np.zeros((1, 64, 128), dtype=np.uint16)
    Vfull[:, :n] = Vs[0]
    for j in range(4):
        pool[table[0, j]] = pack_block(Kb[:, 16 * j:16 * j + 16], Vfull[:, 16 * j:16 * j + 16],
                                       LAYOUT_ATTN)
    q16 = round_to_16bit(q, "f16").reshape(1, 1, 128)
    out = oracle.paged_decode_attention(q16, table, [n], lambda u: pool[u], 1, 128, 16, "f16")
    np.testing.assert_allclose(out[0, 0], oracle.to_float64(Vs[0], "f16")[0, t0], rtol=1e-12,
                               atol=1e-12)


def test_empty_sequence_gives_zeros():
    rng = np.random.default_rng(6)
    pool, table, _, _ = build_paged(rng, [5], 1, 128, 16, "f16")
    table = np.vstack([table, np.full_like(table, -1)])
    q16 = random_16bit(rng, (2, 1, 128), "f16")
    out = oracle.paged_decode_attention(q16, table, [5, 0], lambda u: pool[u], 1, 128, 16, "f16")
    assert np.all(out[1] == 0.0)
    assert np.all(np.isfinite(out[0]))


def test_grouped_query_head_map():
    """Query head h reads kv head h // (Hq/Hkv): give each kv head a constant V."""
    hkv, hq, n = 2, 6, 20
    K = np.zeros((hkv, 32, 128), dtype=np.float32)
    V = np.zeros((hkv, 32, 128), dtype=np.float32)
    V[0] = 1.0
    V[1] = -2.0
    Kb, Vb = round_to_16bit(K, "bf16"), round_to_16bit(V, "bf16")
    pool = np.stack([pack_block(Kb[:, :16], Vb[:, :16], LAYOUT_ATTN),
                     pack_block(Kb[:, 16:], Vb[:, 16:], LAYOUT_ATTN)])
    table = np.array([[1, 0]])
    q16 = random_16bit(np.random.default_rng(7), (1, hq, 128), "bf16")
    out = oracle.paged_decode_attention(q16, table, [n], lambda u: pool[u], hkv, 128, 16, "bf16")
    np.testing.assert_array_equal(out[0, :3], 1.0)
    np.testing.assert_array_equal(out[0, 3:], -2.0)


def test_softmax_scale_closed_form():
    """Two tokens, k0 = e0, k1 = 0, q = a*e0, v0 = 1, v1 = 0: the output is
    sigmoid(a / sqrt(D)) in every channel."""
    a, d = 8.0, 128
    K = np.zeros((1, 16, d), dtype=np.float32)
    V = np.zeros((1, 16, d), dtype=np.float32)
    K[0, 0, 0] = 1.0
    V[0, 0, :] = 1.0
    pool = pack_block(round_to_16bit(K, "f16"), round_to_16bit(V, "f16"), LAYOUT_ATTN)[None]
    q = np.zeros((1, 1, d), dtype=np.float32)
    q[0, 0, 0] = a
    out = oracle.paged_decode_attention(round_to_16bit(q, "f16"), np.array([[0]]), [2],
                                        lambda u: pool[u], 1, d, 16, "f16")
    expect = 1.0 / (1.0 + np.exp(-a / np.sqrt(d)))
    np.testing.assert_allclose(out[0, 0], expect, rtol=1e-14)


def test_nan_in_unused_tail_slots_is_masked():
    rng = np.random.default_rng(8)
    lens = [17, 31, 5]
    pool, table, Ks, Vs = build_paged(rng, lens, 2, 128, 16, "bf16", tail=NAN16["bf16"])
    q16 = random_16bit(rng, (3, 4, 128), "bf16")
    out = oracle.paged_decode_attention(q16, table, lens, lambda u: pool[u], 2, 128, 16, "bf16")
    assert np.all(np.isfinite(out))
    q64 = oracle.to_float64(q16, "bf16")
    for b in range(3):
        ref = sdpa_reference(q64[b], oracle.to_float64(Ks[b], "bf16"),
                             oracle.to_float64(Vs[b], "bf16"))
        np.testing.assert_allclose(out[b], ref, rtol=1e-12, atol=1e-13)


def test_physical_block_permutation_leaves_output_unchanged():
    rng = np.random.default_rng(9)
    lens = [100, 33]
    pool, table, _, _ = build_paged(rng, lens, 1, 128, 16, "f16")
    q16 = random_16bit(rng, (2, 2, 128), "f16")
    out = oracle.paged_decode_attention(q16, table, lens, lambda u: pool[u], 1, 128, 16, "f16")
    perm = rng.permutation(len(pool))            # new physical id of old block u
    pool2 = np.empty_like(pool)
    pool2[perm] = pool
    table2 = np.where(table >= 0, perm[np.maximum(table, 0)], -1)
    out2 = oracle.paged_decode_attention(q16, table2, lens, lambda u: pool2[u], 1, 128, 16, "f16")
    np.testing.assert_array_equal(out, out2)


def test_sixteen_bit_upcast_is_exact():
    bf = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F], dtype=np.uint16)
    np.testing.assert_array_equal(oracle.to_float64(bf, "bf16"),
                                  [1.0, -2.0, 2.0 ** -133, 3.3895313892515355e38])
    hf = np.array([0x3C00, 0xC000, 0x0001, 0x7BFF], dtype=np.uint16)
    np.testing.assert_array_equal(oracle.to_float64(hf, "f16"), [1.0, -2.0, 2.0 ** -24, 65504.0])


def test_element_positions_agree_between_generator_and_oracle():
    """The oracle's layout decoder and the generator's element_index agree."""
    hkv, d, bs = 3, 128, 16
    for layout in (oracle.LAYOUT_ATTN, oracle.LAYOUT_NHD):
        blk = np.arange(2 * hkv * bs * d, dtype=np.uint16).view(np.uint8)
        K, V = oracle.decode_block(blk, layout, hkv, d, bs)
        for (h, t, c) in [(0, 0, 0), (2, 15, 127), (1, 7, 64), (2, 0, 1)]:
            assert K[h, t, c] == element_index(layout, 0, h, t, c, hkv, bs, d)
            assert V[h, t, c] == element_index(layout, 1, h, t, c, hkv, bs, d)

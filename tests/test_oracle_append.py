"""Oracle pins for the decode-step append and the staged-copy write-back.

The append is pinned against the generator's own byte packer (synth.gen, written
independently of the oracle's layout code): after appending tokens one by one
from an empty cache, unpacking the blocks gives back exactly the appended
arrays, in order, and bytes outside the written rows never change. Write-back
is pinned as the inverse of prefetch in both slice layouts.
"""
import numpy as np
import pytest

import oracle
import synth

HKV, D, BS = 2, 128, 16


def _state(layout, n_local=12, n_slice=8):
    bb = oracle.block_bytes(HKV, D, BS)
    st = oracle.SliceOracle(HKV, D, BS, "bf16", layout, n_local * bb, n_slice * bb)
    rng = np.random.default_rng(3)
    st.local[:] = rng.integers(0, 256, st.local.shape, dtype=np.uint8)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)
    return st, rng


def test_append_token_by_token_rebuilds_the_sequence():
    st, rng = _state(0)
    B, T = 3, 40                                    # 40 tokens: 3 blocks, ragged tail
    nb = -(-T // BS)
    table = np.full((B, nb), -1, dtype=np.int64)
    for b in range(B):
        table[b] = st.alloc_blocks(oracle.LOCAL, [b] * nb)
    ks = rng.integers(0, 1 << 16, (T, B, HKV, D), dtype=np.uint16)
    vs = rng.integers(0, 1 << 16, (T, B, HKV, D), dtype=np.uint16)
    before = st.local.copy()
    for t in range(T):
        st.kv_append(ks[t], vs[t], table, np.full(B, t + 1))
    for b in range(B):
        K = np.concatenate([synth.unpack_block(st.local[table[b, j]], synth.LAYOUT_ATTN, HKV, BS,
                                               D)[0] for j in range(nb)], axis=1)[:, :T]
        V = np.concatenate([synth.unpack_block(st.local[table[b, j]], synth.LAYOUT_ATTN, HKV, BS,
                                               D)[1] for j in range(nb)], axis=1)[:, :T]
        assert np.array_equal(K, ks[:, b].transpose(1, 0, 2))
        assert np.array_equal(V, vs[:, b].transpose(1, 0, 2))
        # the unwritten tail rows of the last block keep their old bytes
        last = table[b, nb - 1]
        k_old, v_old = synth.unpack_block(before[last], synth.LAYOUT_ATTN, HKV, BS, D)
        k_new, v_new = synth.unpack_block(st.local[last], synth.LAYOUT_ATTN, HKV, BS, D)
        r = T - (nb - 1) * BS
        assert np.array_equal(k_old[:, r:], k_new[:, r:]) and np.array_equal(v_old[:, r:], v_new[:, r:])
    untouched = np.setdiff1d(np.arange(st.n_local), table.ravel())
    assert np.array_equal(st.local[untouched], before[untouched])


def test_append_skips_empty_sequences_and_rejects_non_local_targets():
    st, rng = _state(0)
    t_local = st.alloc_blocks(oracle.LOCAL, [0])
    t_slice = st.alloc_blocks(oracle.SLICE, [1])
    k = rng.integers(0, 1 << 16, (2, HKV, D), dtype=np.uint16)
    before = st.local.copy()
    st.kv_append(k, k, np.array([[t_local[0]], [t_slice[0]]]), [0, 0])   # nothing to store
    assert np.array_equal(st.local, before)
    with pytest.raises(oracle.OracleError):
        st.kv_append(k, k, np.array([[t_local[0]], [t_slice[0]]]), [1, 1])  # slice target
    assert np.array_equal(st.local, before)                               # all or nothing
    with pytest.raises(oracle.OracleError):
        st.kv_append(k, k, np.array([[t_local[0]], [t_local[0]]]), [1, BS + 1])  # no block 1


@pytest.mark.parametrize("layout", [0, 1])
def test_writeback_is_the_inverse_of_prefetch(layout):
    st, rng = _state(layout)
    src = st.alloc_blocks(oracle.SLICE, [0, 1, 1])
    stg = st.alloc_blocks(oracle.LOCAL, [oracle.STAGING] * 3)
    orig = st.slice[src - st.n_local].copy()
    st.prefetch(src, stg)
    # modify one token of each staged copy, write back, and compare logically
    k = rng.integers(0, 1 << 16, (3, HKV, D), dtype=np.uint16)
    st.kv_append(k, k, stg.reshape(3, 1), [5, 5, 5])
    st.writeback(stg, src)
    for i, u in enumerate(src):
        K, V = synth.unpack_block(st.slice[u - st.n_local], layout, HKV, BS, D)
        K0, V0 = synth.unpack_block(orig[i], layout, HKV, BS, D)
        K0[:, 4, :] = k[i]
        V0[:, 4, :] = k[i]
        assert np.array_equal(K, K0) and np.array_equal(V, V0)


def test_writeback_validates_tags():
    st, _ = _state(0)
    src = st.alloc_blocks(oracle.SLICE, [0])
    owned_local = st.alloc_blocks(oracle.LOCAL, [0])
    stg = st.alloc_blocks(oracle.LOCAL, [oracle.STAGING])
    with pytest.raises(oracle.OracleError):
        st.writeback(owned_local, src)           # source is not a staging block
    with pytest.raises(oracle.OracleError):
        st.writeback(stg, owned_local)           # destination is not a slice block

"""Pins of the slice-state oracle: allocation, copies, lend and reclaim.

What the paper fixes is checked as invariants (exactly-once ownership of every
segment, section 4; the lender regains its full static allocation, sections 3
and 4.1; a preempted request releases its whole dependency chain, section 4.1).
The block-granular reclaim policy is the oracle's reading of a logical
description; the small cases below were worked out by hand from that reading,
step by step in the comments, not produced by running the oracle.
"""
import numpy as np
import pytest

import oracle
from oracle import FREE, STAGING, LENDER, LOCAL, SLICE
from synth import random_16bit, pack_block, unpack_block, LAYOUT_ATTN, LAYOUT_NHD
from slice_trace import Cache, OracleBackend, random_trace

HKV, D, BS = 2, 128, 16
BB = 2 * BS * HKV * D * 2


def make(n_local, n_slice, layout=LAYOUT_ATTN, dtype="f16"):
    return oracle.SliceOracle(HKV, D, BS, dtype, layout, n_local * BB, n_slice * BB)


def set_owners(st, local, slc):
    st.own_local[:] = local
    st.own_slice[:] = slc


def fill_random(st, rng):
    st.local[:] = rng.integers(0, 256, st.local.shape, dtype=np.uint8)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)


# ---- allocation ----------------------------------------------------------------

def test_alloc_takes_lowest_free_slots_and_is_all_or_nothing():
    st = make(6, 4)
    assert list(st.alloc_blocks(LOCAL, [5, 5, 5])) == [0, 1, 2]
    st.free_blocks([1])
    assert list(st.alloc_blocks(LOCAL, [7, 8])) == [1, 3]
    assert list(st.own_local) == [5, 7, 5, 8, FREE, FREE]
    before = st.own_local.copy()
    with pytest.raises(oracle.OracleError) as e:
        st.alloc_blocks(LOCAL, [1, 1, 1])
    assert e.value.code == oracle.ERR_NOMEM
    assert np.array_equal(st.own_local, before)
    assert list(st.alloc_blocks(SLICE, [9, 9])) == [6, 7]     # unified ids n_local + slot


def test_slice_alloc_stops_at_lent_limit_and_lend_caps_at_pool_size():
    st = make(2, 4)
    st.reclaim(3)                       # nothing owned: lim 4 -> 1, no moves
    assert st.lim == 1 and list(st.own_slice) == [FREE, LENDER, LENDER, LENDER]
    with pytest.raises(oracle.OracleError) as e:
        st.alloc_blocks(SLICE, [0, 0])
    assert e.value.code == oracle.ERR_NOMEM
    assert st.lend(10) == 3 and st.lim == 4
    assert list(st.own_slice) == [FREE] * 4


def test_free_errors_leave_state_unchanged():
    st = make(4, 2)
    st.alloc_blocks(LOCAL, [0, 0])
    before = st.own_local.copy()
    for ids, code in [([0, 2], oracle.ERR_OWNER), ([0, 0], oracle.ERR_INVAL),
                      ([0, 99], oracle.ERR_INVAL)]:
        with pytest.raises(oracle.OracleError) as e:
            st.free_blocks(ids)
        assert e.value.code == code
        assert np.array_equal(st.own_local, before)


def test_staging_only_local_and_bad_owner_rejected():
    st = make(2, 2)
    for where, owners in [(SLICE, [STAGING]), (LOCAL, [-5]), (LOCAL, [LENDER])]:
        with pytest.raises(oracle.OracleError) as e:
            st.alloc_blocks(where, owners)
        assert e.value.code == oracle.ERR_INVAL


# ---- layouts and copies ----------------------------------------------------------

@pytest.mark.parametrize("layout", [LAYOUT_ATTN, LAYOUT_NHD])
def test_oracle_layout_decoder_matches_generator_packer(layout):
    rng = np.random.default_rng(10)
    K = random_16bit(rng, (HKV, BS, D), "bf16")
    V = random_16bit(rng, (HKV, BS, D), "bf16")
    blk = pack_block(K, V, layout)
    K2, V2 = oracle.decode_block(blk, layout, HKV, D, BS)
    assert np.array_equal(K, K2) and np.array_equal(V, V2)
    assert np.array_equal(oracle.encode_block(K, V, layout), blk)


def test_layout_conversion_round_trip_and_logical_content():
    rng = np.random.default_rng(11)
    blk = rng.integers(0, 256, BB, dtype=np.uint8)
    nhd = oracle.convert_block(blk, LAYOUT_ATTN, LAYOUT_NHD, HKV, D, BS)
    assert not np.array_equal(nhd, blk)
    assert np.array_equal(oracle.convert_block(nhd, LAYOUT_NHD, LAYOUT_ATTN, HKV, D, BS), blk)
    k1, v1 = unpack_block(blk, LAYOUT_ATTN, HKV, BS, D)
    k2, v2 = unpack_block(nhd, LAYOUT_NHD, HKV, BS, D)
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


@pytest.mark.parametrize("layout", [LAYOUT_ATTN, LAYOUT_NHD])
def test_prefetch_copies_slice_blocks_into_staging(layout):
    rng = np.random.default_rng(12)
    st = make(6, 4, layout)
    fill_random(st, rng)
    src = st.alloc_blocks(SLICE, [0, 1, 0])            # 6, 7, 8
    dst = st.alloc_blocks(LOCAL, [STAGING] * 3)        # 0, 1, 2
    untouched = st.local[3:].copy()
    st.prefetch([8, 6], [1, 0])
    for s, d in [(8, 1), (6, 0)]:
        ks, vs = unpack_block(st.slice[s - 6], layout, HKV, BS, D)
        kd, vd = unpack_block(st.local[d], LAYOUT_ATTN, HKV, BS, D)
        assert np.array_equal(ks, kd) and np.array_equal(vs, vd)
    assert np.array_equal(st.local[3:], untouched)
    assert list(src) == [6, 7, 8] and list(dst) == [0, 1, 2]


def test_prefetch_validation():
    st = make(4, 4)
    st.alloc_blocks(SLICE, [0, 0])                     # 4, 5
    st.alloc_blocks(LOCAL, [STAGING, STAGING, 3])      # 0, 1, 2(owned by 3)
    bad = [([4, 5], [0, 0]),      # duplicate destination
           ([4], [2]),            # destination not staging
           ([6], [0]),            # free slice slot
           ([0], [1]),            # source not in the slice
           ([4, 5], [0])]         # length mismatch
    for src, dst in bad:
        with pytest.raises(oracle.OracleError) as e:
            st.prefetch(src, dst)
        assert e.value.code == oracle.ERR_INVAL


# ---- reclaim: hand-worked cases ----------------------------------------------------

def test_reclaim_compacts_within_the_slice():
    # n_local 4 (all free), n_slice 6, lim 6. Slice owners A=0, B=1:
    #   slot: 0 1 2 3 4 5
    #         A . B . A B
    # reclaim(2): cut = 4. Movers = owned slots in [4,6) = [4(A), 5(B)].
    # Destinations = free slice slots below 4 = [1, 3], then local [0..3].
    # 4 -> slot 1, 5 -> slot 3. Slots 4, 5 become the lender's; lim = 4.
    st = make(4, 6)
    set_owners(st, [FREE] * 4, [0, FREE, 1, FREE, 0, 1])
    fill_random(st, np.random.default_rng(13))
    moved_a, moved_b = st.slice[4].copy(), st.slice[5].copy()
    tables = np.array([[4 + 0, 4 + 4], [4 + 2, 4 + 5]])
    r = st.reclaim(2, tables)
    assert r["moves"] == [(8, 5), (9, 7)]
    assert r["moved"] == 2 and r["written_back"] == 0 and r["victims"] == [] and r["lim"] == 4
    assert list(st.own_slice) == [0, 0, 1, 1, LENDER, LENDER]
    assert np.array_equal(tables, [[4, 5], [6, 7]])
    assert np.array_equal(st.slice[1], moved_a) and np.array_equal(st.slice[3], moved_b)


@pytest.mark.parametrize("layout", [LAYOUT_ATTN, LAYOUT_NHD])
def test_reclaim_writes_back_to_local_when_the_slice_is_full(layout):
    # n_local 4, n_slice 4. Slice [A B A B], local [. A . .].
    # reclaim(2): cut = 2, movers [2(A), 3(B)], no free slice slot below 2,
    # local free [0, 2, 3]: 2 -> local 0, 3 -> local 2 (written back, re-laid
    # into the local layout).
    st = make(4, 4, layout)
    set_owners(st, [FREE, 0, FREE, FREE], [0, 1, 0, 1])
    fill_random(st, np.random.default_rng(14))
    src2, src3 = st.slice[2].copy(), st.slice[3].copy()
    tables = np.array([[1, 4, 6], [5, 7, -1]])
    r = st.reclaim(2, tables)
    assert r["moves"] == [(6, 0), (7, 2)] and r["written_back"] == 2
    assert list(st.own_local) == [0, 0, 1, FREE]
    assert list(st.own_slice) == [0, 1, LENDER, LENDER]
    assert np.array_equal(tables, [[1, 4, 0], [5, 2, -1]])
    for src, dst in [(src2, 0), (src3, 2)]:
        ks, vs = unpack_block(src, layout, HKV, BS, D)
        kd, vd = unpack_block(st.local[dst], LAYOUT_ATTN, HKV, BS, D)
        assert np.array_equal(ks, kd) and np.array_equal(vs, vd)


def test_reclaim_preempts_the_owner_with_most_blocks_in_the_range():
    # n_local 2 (owned by A=0 and C=2), n_slice 4: slice [B A B B], B=1.
    # reclaim(3): cut = 1, movers [1(A), 2(B), 3(B)], destinations: none
    # (slot 0 is B's, local full). |M| = 3 > 0: victim = B (2 movers vs 1).
    # B frees slots 0, 2, 3. Movers [1(A)], destinations [slot 0]. 1 -> 0.
    # Unified ids are 2 + slot: remap 3 -> 2, and B's blocks 2, 4, 5 -> -1.
    st = make(2, 4)
    set_owners(st, [0, 2], [1, 0, 1, 1])
    tables = np.array([[0, 3], [2, 4], [5, -1], [1, -1]])
    r = st.reclaim(3, tables)
    assert r["victims"] == [1] and r["moves"] == [(3, 2)] and r["lim"] == 1
    assert list(st.own_slice) == [0, LENDER, LENDER, LENDER]
    assert list(st.own_local) == [0, 2]
    assert np.array_equal(tables, [[0, 2], [-1, -1], [-1, -1], [1, -1]])


def test_reclaim_victim_tie_goes_to_larger_owner_id_and_chain_is_released():
    # n_local 2 owned by [3, 5]; slice [3 5 3 5], reclaim(4): cut 0, movers
    # [0(3), 1(5), 2(3), 3(5)], no destinations. Counts 3:2, 5:2 -> victim 5,
    # which also releases local block 1 (its dependency chain). Movers
    # [0(3), 2(3)], destinations [local 1]: still 2 > 1 -> victim 3, which
    # releases local 0. No movers remain; the lender holds all 4 slots.
    st = make(2, 4)
    set_owners(st, [3, 5], [3, 5, 3, 5])
    r = st.reclaim(4)
    assert r["victims"] == [5, 3] and r["moves"] == [] and r["lim"] == 0
    assert list(st.own_local) == [FREE, FREE]
    oracle.check_sd_symmetry(st)


def test_reclaim_clamps_to_lent_amount_and_zero_is_a_no_op():
    st = make(2, 3)
    set_owners(st, [FREE, FREE], [0, FREE, FREE])
    r = st.reclaim(0)
    assert r["reclaimed"] == 0 and st.lim == 3
    r = st.reclaim(100)
    assert r["reclaimed"] == 3 and r["moves"] == [(2, 0)] and st.lim == 0
    with pytest.raises(oracle.OracleError):
        st.reclaim(-1)


# ---- invariants over random traces ------------------------------------------------

@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("layout", [LAYOUT_ATTN, LAYOUT_NHD])
def test_random_trace_keeps_invariants(seed, layout):
    rng = np.random.default_rng(100 + seed)
    st = oracle.SliceOracle(HKV, D, BS, "f16", layout, 24 * BB, 16 * BB)
    data_rng = np.random.default_rng(seed)

    def write(u):
        st.write_block(u, data_rng.integers(0, 256, BB, dtype=np.uint8))

    cache = Cache([OracleBackend(st)], layers=2, batch=5, maxblk=6, rng=rng, write_data=write)

    def check_prefetch(src, dst):
        for s, d in zip(src, dst):
            ks, vs = oracle.decode_block(st.read_block(s), layout, HKV, D, BS)
            kd, vd = oracle.decode_block(st.read_block(d), LAYOUT_ATTN, HKV, D, BS)
            assert np.array_equal(ks, kd) and np.array_equal(vs, vd)       # I5

    view = {}

    def on_step(step, op):
        nonlocal view
        oracle.check_ownership(st, cache.tables)                           # I1
        oracle.check_conservation(st)                                      # I2
        new_view = oracle.logical_view(st, cache.tables)
        for key, kv in new_view.items():                                   # I4
            if key in view and cache.log[-1][0] not in ("grow",):
                assert np.array_equal(view[key][0], kv[0]) and np.array_equal(view[key][1], kv[1])
        view = new_view

    orig = cache.prefetch_layer
    cache.prefetch_layer = lambda l, check=None: orig(l, check_prefetch)
    random_trace(cache, 150, rng, on_step)
    cache.reclaim(st.lim)
    oracle.check_sd_symmetry(st)                                           # I3
    oracle.check_ownership(st, cache.tables)
    assert st.n_local == 24 and st.n_slice == 16

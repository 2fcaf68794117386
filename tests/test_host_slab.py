"""The library's slab bookkeeping against the slab oracle, on the CPU.

The library is created host-only (no device memory) and switched to slabs;
random traces of slab allocations and frees, local allocations, migrations
into and out of slabs, lends and slab reclaims run on it and on the oracle
side by side. After every operation: the same positions, error codes, slab
tags, position owners and per-slot owner tags; the library's block ids,
staged ids and layer-group runs equal the oracle's for every layout.
"""
import os

import numpy as np
import pytest

import oracle
from oracle import GROUP_MAJOR, LAYER_MAJOR, SLAB_MAJOR, STAGING

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2609_27040_amd", "lib", "libema_slice.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")

HKV, D, BS = 1, 128, 16
BB = 2 * BS * HKV * D * 2


def pair(n_local, n_slice, L, S, k, layout):
    from paper_2609_27040_amd import ema
    h = ema.slice_create(HKV, D, BS, "f16", 0, n_local * BB, n_slice * BB, host_only=True)
    ema.slab_init(h, L, S, k, layout)
    st = oracle.SlabSliceOracle(HKV, D, BS, "f16", 0, n_local * BB, n_slice * BB, layers=L,
                                slab_blocks=S, group=k, slab_layout=layout, with_data=False)
    return ema, h, st


def same_state(ema, h, st):
    info = ema.slab_get_info(h)
    assert np.array_equal(info["slab_tag"], st.slab_tag)
    assert np.array_equal(info["pos_owner"], st.pos_owner)
    own_l, own_s, _ = ema.slice_owners(h)
    assert np.array_equal(own_l, st.own_local) and np.array_equal(own_s, st.own_slice)


def both(ema, lib_call, or_call):
    """Runs both; they must succeed together or fail with the same code."""
    err_l = err_o = None
    try:
        rl = lib_call()
    except ema.EmaError as e:
        err_l, rl = e.code, None
    try:
        ro = or_call()
    except oracle.OracleError as e:
        err_o, ro = e.code, None
    assert err_l == err_o, (err_l, err_o)
    return rl, ro


@pytest.mark.parametrize("layout", [LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR])
@pytest.mark.parametrize("L,S,k", [(4, 3, 2), (6, 1, 3), (4, 5, 4)])
def test_slab_bookkeeping_matches_oracle_on_random_traces(layout, L, S, k):
    rng = np.random.default_rng(L * 100 + S * 10 + k + layout)
    n_slabs, extra = 7, 3
    n_local = 60 + n_slabs * k * S          # room for a staging image of every slab
    ema, h, st = pair(n_local, n_slabs * L * S + extra, L, S, k, layout)
    B, maxblk = 6, 16
    tables = np.full((L, B, maxblk), -1, dtype=np.int64)
    try:
        same_state(ema, h, st)
        for step in range(250):
            op = int(rng.integers(7))
            b = int(rng.integers(B))
            if op == 0:                                     # grow in slabs
                n = int(rng.integers(1, 2 * S + 2))
                pl, po = both(ema, lambda: ema.slab_alloc(h, [b] * n),
                              lambda: st.slab_alloc([b] * n))
                if pl is not None:
                    assert np.array_equal(pl, po)
                    for p in pl:
                        j = int(np.sum(tables[0, b] >= 0))
                        if j >= maxblk:
                            ema.slab_free(h, [p])
                            st.slab_free([p])
                            continue
                        ids = [st.block_id(p, l) for l in range(L)]
                        for l in range(L):
                            assert ema.slab_block_ids(h, [p], l)[0] == ids[l]
                            tables[l, b, j] = ids[l]
            elif op == 1:                                   # grow locally (every layer)
                n = int(rng.integers(1, 3))
                ul, uo = both(ema, lambda: ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [b] * (n * L)),
                              lambda: st.alloc_blocks(oracle.LOCAL, [b] * (n * L)))
                if ul is not None:
                    assert np.array_equal(ul, uo)
                    for q in range(n):
                        j = int(np.sum(tables[0, b] >= 0))
                        if j >= maxblk:
                            ema.slice_free_blocks(h, ul[q * L:(q + 1) * L])
                            st.free_blocks(ul[q * L:(q + 1) * L])
                            continue
                        tables[:, b, j] = ul[q * L:(q + 1) * L]
            elif op == 2:                                   # a sequence finishes
                ids = tables[:, b][tables[:, b] >= 0]
                loc = ids[ids < st.n_local]
                pos = [int(p) for p in np.nonzero(st.pos_owner == b)[0]]
                ema.slice_free_blocks(h, loc)
                st.free_blocks(loc)
                ema.slab_free(h, pos)
                st.slab_free(pos)
                tables[:, b] = -1
            elif op == 3:                                   # lender lends
                n = int(rng.integers(0, 3))
                assert ema.slice_lend(h, n) == st.lend(n)
            elif op == 4:                                   # lender reclaims slabs
                n = int(rng.integers(0, 3))
                r = ema.slab_reclaim(h, n)
                ro = st.reclaim(n, tables)
                assert r["reclaimed"] == ro["reclaimed"] and r["slabs"] == ro["slabs"]
                assert r["victims"] == ro["victims"] and r["released"] == len(ro["released"])
                for v in ro["victims"]:
                    assert np.all(tables[:, v] == -1)        # the oracle rewrote them
            elif op == 5:                                   # migrate a logical block in
                locj = [j for j in range(maxblk) if 0 <= tables[0, b, j] < st.n_local]
                if not locj:
                    continue
                j = locj[int(rng.integers(len(locj)))]
                pl, po = both(ema, lambda: ema.slab_alloc(h, [b]), lambda: st.slab_alloc([b]))
                if pl is None:
                    continue
                dst = [st.block_id(pl[0], l) for l in range(L)]
                src = tables[:, b, j].copy()
                ema.slice_migrate(h, src, np.asarray(dst))
                st.migrate(src, dst)
                ema.slice_free_blocks(h, src)
                st.free_blocks(src)
                tables[:, b, j] = dst
            else:                                           # error paths
                both(ema, lambda: ema.slab_free(h, [10 ** 6]), lambda: st.slab_free([10 ** 6]))
                free_pos = [int(p) for p in np.nonzero(st.pos_owner == oracle.FREE)[0][:1]]
                both(ema, lambda: ema.slab_free(h, free_pos), lambda: st.slab_free(free_pos))
                both(ema, lambda: ema.slice_alloc_blocks(h, ema.POOL_SLICE, [b]),
                     lambda: st.alloc_blocks(oracle.SLICE, [b]))
            same_state(ema, h, st)
            oracle.check_slab_tags(st)
            oracle.check_ownership(st, tables)
            # runs and staged ids of every group, for the current borrowed set
            m = len(st.borrowed())
            for g in range(L // k):
                a, d, n = ema.slab_group_runs(h, g, 7)
                assert list(zip(a.tolist(), d.tolist(), n.tolist())) == st.group_runs(g, 7)
            used = [int(p) for p in np.nonzero(st.pos_owner >= 0)[0]]
            if used and m:
                l = int(rng.integers(L))
                got = ema.slab_block_ids(h, used, l, 5)
                assert got.tolist() == [st.staged_id(p, l, 5) for p in used]
        ema.slab_reclaim(h, 10 ** 6)
        st.reclaim(10 ** 6, tables)
        same_state(ema, h, st)
        oracle.check_slab_sd_symmetry(st, tables)
    finally:
        ema.slice_destroy(h)


def test_slab_group_prefetch_validates_its_staging_image():
    ema, h, st = pair(40, 3 * 4 * 2, 4, 2, 2, GROUP_MAJOR)
    try:
        ema.slab_alloc(h, [0, 0, 1])                  # slabs 0 and 1 borrowed: 2*2*2 = 8 blocks
        stg = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [STAGING] * 8)
        assert stg.tolist() == list(range(8))
        ema.slab_prefetch_group(h, 1, 0)
        for first in (1, -1):                          # runs past the staging blocks, negative
            with pytest.raises(ema.EmaError) as e:
                ema.slab_prefetch_group(h, 1, first)
            assert e.value.code == ema.ERR_INVAL
        with pytest.raises(ema.EmaError):
            ema.slab_prefetch_group(h, 2, 0)            # group out of range
        with pytest.raises(ema.EmaError):              # already in slabs
            ema.slab_init(h, 4, 2, 2, GROUP_MAJOR)
        with pytest.raises(ema.EmaError):              # block-mode reclaim refused
            ema.slice_reclaim(h, 1)
    finally:
        ema.slice_destroy(h)


def test_slab_init_needs_an_untouched_slice_and_a_whole_slab():
    from paper_2609_27040_amd import ema
    h = ema.slice_create(HKV, D, BS, "f16", 0, 10 * BB, 10 * BB, host_only=True)
    try:
        ema.slice_alloc_blocks(h, ema.POOL_SLICE, [0])
        with pytest.raises(ema.EmaError):
            ema.slab_init(h, 2, 2, 1)
    finally:
        ema.slice_destroy(h)
    h = ema.slice_create(HKV, D, BS, "f16", 0, 10 * BB, 10 * BB, host_only=True)
    try:
        for cfg in [(4, 3, 1), (4, 2, 3), (0, 1, 1), (2, 1, 1, 5)]:
            with pytest.raises(ema.EmaError):
                ema.slab_init(h, *cfg)                  # 12 > 10 slots, 3 !| 4, L 0, layout
        ema.slab_init(h, 2, 2, 2)
        assert ema.slab_get_info(h)["n_slabs"] == 2
    finally:
        ema.slice_destroy(h)

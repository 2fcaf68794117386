"""Pins of the slab oracle (section 4.2.1-4.2.3).

Hand-worked cases (written out in the comments, not produced by running the
oracle) for the three placements, allocation, freeing, lending and the
reclaim victim rule; the swap sizes the paper states for each placement
(layer-major S to mS, slab-major fixed kS, layer-group-major kS to mkS) as
properties of the runs; and the invariant checks of the slab state, each
shown to reject a state that breaks it.
"""
import numpy as np
import pytest

import oracle
from oracle import (FREE, LENDER, STAGING, LOCAL, BORROWED, GROUP_MAJOR, LAYER_MAJOR, SLAB_MAJOR,
                    InvariantError, SlabSliceOracle)

HKV, D, BS = 1, 128, 16
BB = 2 * BS * HKV * D * 2


def make(n_local, n_slabs, L=4, S=2, k=2, layout=GROUP_MAJOR, extra_slots=0, data=False):
    return SlabSliceOracle(HKV, D, BS, "f16", 0, n_local * BB, (n_slabs * L * S + extra_slots) * BB,
                           layers=L, slab_blocks=S, group=k, slab_layout=layout,
                           with_data=data)


# ---- placement -------------------------------------------------------------------------

def test_slot_formulas_on_a_hand_drawn_example():
    # L = 4 layers, S = 2 positions, k = 2 layers per group, 3 slabs: 24 slots.
    # Layer-major: slot = (l*3 + i)*2 + p -> (slab 1, layer 2, pos 1) = (6+1)*2+1 = 15.
    # Slab-major:  slot = (i*4 + l)*2 + p -> (4+2)*2+1 = 13.
    # Group-major: slot = ((l//2*3 + i)*2 + l%2)*2 + p -> ((3+1)*2+0)*2+1 = 17.
    assert make(0, 3, layout=LAYER_MAJOR).slot(1, 2, 1) == 15
    assert make(0, 3, layout=SLAB_MAJOR).slot(1, 2, 1) == 13
    assert make(0, 3, layout=GROUP_MAJOR).slot(1, 2, 1) == 17
    # Group-major order of the first 12 slots: group 0 of slab 0 (layers 0,1 x
    # positions 0,1), then group 0 of slab 1, then of slab 2; group 1 starts at 12.
    st = make(0, 3, layout=GROUP_MAJOR)
    first = [(i, l, p) for i in range(3) for l in (0, 1) for p in (0, 1)]
    assert [st.slot(*t) for t in first] == list(range(12))
    assert st.slot(0, 2, 0) == 12


@pytest.mark.parametrize("layout", [LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR])
@pytest.mark.parametrize("L,S,k,n", [(4, 2, 2, 3), (6, 3, 3, 2), (8, 5, 4, 4), (4, 1, 1, 5)])
def test_every_placement_is_a_bijection_onto_the_slabbed_slots(layout, L, S, k, n):
    st = make(0, n, L=L, S=S, k=k, layout=layout)
    slots = sorted(st.slot(i, l, p) for i in range(n) for l in range(L) for p in range(S))
    assert slots == list(range(n * L * S))


def test_slots_past_the_last_whole_slab_are_never_lent():
    st = make(0, 2, extra_slots=5)              # 16 slabbed slots + 5 spare
    assert st.n_slabs == 2
    assert list(st.own_slice[16:]) == [LENDER] * 5
    oracle.check_slab_tags(st)


# ---- allocation, free, lend --------------------------------------------------------------

def test_alloc_fills_borrowed_slabs_then_takes_the_lowest_free_slab():
    st = make(4, 3)                              # S = 2
    # seq 7 needs 3 blocks: slab 0 taken (positions 0, 1), then slab 1 (position 2)
    assert list(st.slab_alloc([7, 7, 7])) == [0, 1, 2]
    assert list(st.slab_tag) == [BORROWED, BORROWED, FREE]
    # seq 8 fills position 3 of slab 1 and takes slab 2
    assert list(st.slab_alloc([8, 8])) == [3, 4]
    # every layer of position 4 (slab 2, p 0) belongs to seq 8
    assert all(st.owner(st.block_id(4, l)) == 8 for l in range(4))
    before = (st.slab_tag.copy(), st.pos_owner.copy())
    with pytest.raises(oracle.OracleError) as e:              # one position left, two wanted
        st.slab_alloc([9, 9])
    assert e.value.code == oracle.ERR_NOMEM
    assert np.array_equal(before[0], st.slab_tag) and np.array_equal(before[1], st.pos_owner)
    oracle.check_slab_tags(st)


def test_free_returns_an_emptied_slab_and_alloc_reuses_the_lowest_position():
    st = make(4, 3)
    st.slab_alloc([7, 7, 8, 8, 9])               # slabs 0, 1, 2 (slab 2 half used)
    st.slab_free([2, 3])                         # slab 1 empties -> back to the slice
    assert list(st.slab_tag) == [BORROWED, FREE, BORROWED]
    st.slab_free([0])                            # slab 0 keeps position 1
    assert st.slab_tag[0] == BORROWED
    # lowest free position of a borrowed slab first (0), then slab 2's free 5,
    # then the lowest free slab (1)
    assert list(st.slab_alloc([4, 4, 4])) == [0, 5, 2]
    with pytest.raises(oracle.OracleError) as e:
        st.slab_free([3, 3])
    assert e.value.code == oracle.ERR_INVAL
    with pytest.raises(oracle.OracleError) as e:
        st.slab_free([3])                          # free position of slab 1
    assert e.value.code == oracle.ERR_OWNER
    oracle.check_slab_tags(st)


def test_slice_blocks_only_through_slab_calls():
    st = make(4, 2)
    with pytest.raises(oracle.OracleError):
        st.alloc_blocks(oracle.SLICE, [1])
    pos = st.slab_alloc([1])
    with pytest.raises(oracle.OracleError):
        st.free_blocks([st.block_id(pos[0], 0)])
    assert list(st.alloc_blocks(LOCAL, [1, STAGING])) == [0, 1]


def test_lend_returns_the_lowest_lender_slabs():
    st = make(2, 4)
    r = st.reclaim(3)                            # nothing borrowed: free slabs 3, 2, 1 taken
    assert r["slabs"] == [3, 2, 1] and r["victims"] == []
    assert list(st.slab_tag) == [FREE, LENDER, LENDER, LENDER]
    assert st.lend(2) == 2
    assert list(st.slab_tag) == [FREE, FREE, FREE, LENDER]
    assert st.lend(5) == 1
    oracle.check_slab_tags(st)


# ---- reclaim: the slab with the fewest active requests -------------------------------------

def test_reclaim_takes_free_slabs_first_then_the_slab_with_fewest_requests():
    # S = 4 positions, L = 2, k = 1, 3 slabs, 6 local blocks.
    st = make(6, 3, L=2, S=4, k=1)
    # slab 0: seqs 1, 2, 3, 3 (three requests); slab 1: seqs 4, 4, 5, 5 (two);
    # slab 2: seq 6 only (one request, one position used).
    st.slab_alloc([1, 2, 3, 3, 4, 4, 5, 5, 6])
    local = st.alloc_blocks(LOCAL, [6, 4, 1])    # local blocks 0, 1, 2
    tables = np.full((2, 7, 4), -1)
    for pos, seq in enumerate([1, 2, 3, 3, 4, 4, 5, 5, 6]):
        j = int(np.sum(tables[0, seq] >= 0))
        for l in range(2):
            tables[l, seq, j] = st.block_id(pos, l)
    for u, seq in zip(local, [6, 4, 1]):
        tables[0, seq, int(np.sum(tables[0, seq] >= 0))] = u
    oracle.check_ownership(st, tables)
    # Reclaim 2 slabs. No free slab: slab 2 has the fewest requests (1) ->
    # seq 6 preempted: its position 8 and its local block 0 are released, slab 2
    # goes to the lender. Second slab: slabs 0 (3 requests) and 1 (2) ->
    # slab 1: seqs 4 and 5 preempted (local block 1 of seq 4 released too).
    r = st.reclaim(2, tables)
    assert r["slabs"] == [2, 1]
    assert r["victims"] == [6, 4, 5]
    assert list(st.slab_tag) == [BORROWED, LENDER, LENDER]
    assert list(st.own_local[:3]) == [FREE, FREE, 1]
    assert np.all(tables[:, [4, 5, 6]] == -1)
    assert tables[0, 1, 1] == 2                  # seq 1's local block kept
    oracle.check_ownership(st, tables)
    oracle.check_slab_tags(st)
    # reclaim everything: slab 0 last; the lender holds every slab again
    r = st.reclaim(10, tables)
    assert r["slabs"] == [0] and r["victims"] == [1, 2, 3]
    oracle.check_slab_sd_symmetry(st, tables)


def test_reclaim_tie_goes_to_the_highest_slab_and_emptied_slabs_return_first():
    # S = 2, L = 2, k = 1, 3 slabs: slab 0 = seq 1 x2, slab 1 = seq 2 x2, slab 2 = seq 1 x2.
    st = make(0, 3, L=2, S=2, k=1)
    st.slab_alloc([1, 1, 2, 2, 1, 1])
    # all have one request: tie -> slab 2; preempting seq 1 also empties slab 0,
    # which returns to the slice and is the next slab taken, without a victim.
    r = st.reclaim(2)
    assert r["slabs"] == [2, 0] and r["victims"] == [1]
    assert list(st.slab_tag) == [LENDER, BORROWED, LENDER]


# ---- the swap of a layer group ------------------------------------------------------------

def _run_lengths(st, g, stage_first=0):
    return [r[2] for r in st.group_runs(g, stage_first)]


def test_layer_group_major_swaps_adjacent_slabs_in_one_run():
    # L = 4, S = 2, k = 2, 4 slabs; borrowed slabs 0, 1, 3 (slab 2 free).
    st = make(40, 4, L=4, S=2, k=2, layout=GROUP_MAJOR)
    st.slab_alloc([1] * 8)                       # slabs 0..3
    st.slab_free([4, 5])                         # slab 2 back to the slice
    # group 1 of slab 0 starts at ((1*4 + 0)*2)*2 = 16: slabs 0 and 1 are one
    # run of 2*k*S = 8 blocks (slots 16..23), slab 3 one of 4 (slots 28..31).
    runs = st.group_runs(1, 100)
    assert [(s - st.n_local, d, n) for s, d, n in runs] == [(16, 100, 8), (28, 108, 4)]


@pytest.mark.parametrize("borrowed", [[0], [0, 1], [0, 1, 2], [0, 2, 3], [1, 3]])
def test_swap_sizes_match_the_paper_per_placement(borrowed):
    L, S, k, n = 8, 3, 2, 4
    for layout in (LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR):
        st = make(200, n, L=L, S=S, k=k, layout=layout)
        st.slab_alloc([5] * (n * S))
        st.slab_free([i * S + p for i in range(n) if i not in borrowed for p in range(S)])
        # maximal sets of adjacent borrowed slabs
        blocks, cur = [], 1
        for a, b in zip(borrowed, borrowed[1:]):
            if b == a + 1:
                cur += 1
            else:
                blocks.append(cur)
                cur = 1
        blocks.append(cur)
        for g in range(L // k):
            lens = _run_lengths(st, g)
            assert sum(lens) == len(borrowed) * k * S       # every slab's group moves
            if layout == SLAB_MAJOR:
                assert lens == [k * S] * len(borrowed)      # fixed kS
            elif layout == GROUP_MAJOR:
                assert lens == [m * k * S for m in blocks]  # kS .. mkS
            else:
                # S .. mS per layer (runs of adjacent slabs in one layer), layer
                # after layer; the last run of a layer continues into the first
                # of the next when slab n-1 and slab 0 are both borrowed (layer
                # l's slab n-1 ends where layer l+1's slab 0 starts)
                want = [m * S for m in blocks]
                if borrowed[0] == 0 and borrowed[-1] == n - 1 and len(blocks) > 1:
                    merged = list(want)
                    for _ in range(k - 1):
                        merged[-1] += want[0]
                        merged += want[1:]
                    want = merged
                elif borrowed[0] == 0 and borrowed[-1] == n - 1:
                    want = [n * S * k]
                else:
                    want = want * k
                assert lens == want


@pytest.mark.parametrize("layout", [LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR])
def test_group_prefetch_copies_whole_slabs_into_the_staging_image(layout):
    rng = np.random.default_rng(4)
    L, S, k = 4, 3, 2
    st = make(64, 3, L=L, S=S, k=k, layout=layout, data=True)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)
    st.slab_alloc([1, 1, 2, 2, 2, 3, 3])           # slabs 0, 1, 2 (slab 2 has 1 used)
    st.slab_free([3, 4, 5])                         # slab 1 returns: borrowed 0 and 2
    stage = st.alloc_blocks(LOCAL, [STAGING] * (2 * k * S))
    assert list(stage) == list(range(2 * k * S))
    for g in range(L // k):
        st.prefetch_group(g, 0)
        for pos in [0, 1, 2, 6, 7, 8]:               # every position, used or not
            for j in range(k):
                l = g * k + j
                d = st.staged_id(pos, l, 0)
                assert np.array_equal(st.local[d], st.slice[st.block_id(pos, l) - st.n_local])
    with pytest.raises(oracle.OracleError):
        st.prefetch_group(0, 1)                     # runs past the staging area


# ---- invariant checks of the slab state, pinned by violating states --------------------------

def _valid():
    st = make(4, 3)
    st.slab_alloc([1, 1, 2])                     # slab 0 (seq 1 x2), slab 1 (seq 2, one free)
    st.reclaim(1)                                # free slab 2 -> lender
    return st


def test_slab_tag_check_accepts_a_valid_state():
    oracle.check_slab_tags(_valid())


@pytest.mark.parametrize("break_it,what", [
    (lambda st: st.slab_tag.__setitem__(1, 7), "has tag"),
    (lambda st: st.own_slice.__setitem__(st.slot(1, 3, 1), 2), "has tag 2"),          # stray owner
    (lambda st: st.own_slice.__setitem__(st.slot(2, 0, 0), FREE), "not -3"),          # lender slot freed
    (lambda st: st.pos_owner.__setitem__(5, 4), "not borrowed"),                      # block in lender slab
    (lambda st: (st.pos_owner.__setitem__(2, FREE),
                 [st.own_slice.__setitem__(st.slot(1, l, 0), FREE) for l in range(4)]),
     "holds no block"),                                                               # empty borrowed slab
    (lambda st: st.own_slice.__setitem__(st.slot(0, 2, 0), 2), "not 1"),              # one layer re-owned
])
def test_slab_tag_check_rejects_each_violation(break_it, what):
    st = _valid()
    break_it(st)
    with pytest.raises(InvariantError, match=what):
        oracle.check_slab_tags(st)


def test_slab_sd_symmetry_rejects_a_lender_short_of_its_slabs():
    st = _valid()
    with pytest.raises(InvariantError, match="still lent"):
        oracle.check_slab_sd_symmetry(st)
    st.reclaim(10)
    oracle.check_slab_sd_symmetry(st)
    st.own_slice[0] = 1
    with pytest.raises(InvariantError, match="not the lender"):
        oracle.check_slab_sd_symmetry(st)
    st.own_slice[0] = LENDER
    with pytest.raises(InvariantError, match="names a slice"):
        oracle.check_slab_sd_symmetry(st, np.array([[[st.n_local + 3]]]))


def test_random_slab_traces_keep_every_invariant():
    rng = np.random.default_rng(11)
    for layout in (LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR):
        L, S, k, B = 4, 3, 2, 6
        st = make(40, 6, L=L, S=S, k=k, layout=layout)
        tables = np.full((L, B, 12), -1)
        held = {b: [] for b in range(B)}                  # positions per sequence
        for _ in range(120):
            op = rng.integers(4)
            b = int(rng.integers(B))
            if op == 0:
                n = int(rng.integers(1, 4))
                try:
                    pos = st.slab_alloc([b] * n)
                except oracle.OracleError:
                    continue
                for p in pos:
                    j = int(np.sum(tables[0, b] >= 0))
                    if j >= tables.shape[2]:
                        st.slab_free([p])
                        continue
                    for l in range(L):
                        tables[l, b, j] = st.block_id(p, l)
                    held[b].append(int(p))
            elif op == 1 and held[b]:
                p = held[b].pop()
                j = int(np.nonzero(tables[0, b] == st.block_id(p, 0))[0][0])
                tables[:, b, j:-1] = tables[:, b, j + 1:]
                tables[:, b, -1] = -1
                st.slab_free([p])
            elif op == 2:
                r = st.reclaim(int(rng.integers(1, 3)), tables)
                for v in r["victims"]:
                    held[v] = []
                    tables[:, v] = -1                     # rewritten to -1 already
            else:
                st.lend(int(rng.integers(1, 3)))
            oracle.check_slab_tags(st)
            oracle.check_ownership(st, tables)
        st.reclaim(100, tables)
        oracle.check_slab_sd_symmetry(st, tables)


# ---- the paper's worked example (tests/golden/layer_group_example.json) --------------------

def test_layer_group_major_placement_reproduces_the_papers_example():
    import json
    import os
    ex = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "layer_group_example.json")))
    k, L = ex["group_size"], ex["layers"]
    S, n = 3, 4
    st = make(200, n, L=L, S=S, k=k, layout=GROUP_MAJOR)
    # layer groups are runs of k consecutive layers
    for g, layers in enumerate(ex["layer_groups"]):
        assert [l for l in range(L) if l // k == g] == layers
    # slab 0 of the group's layers, then slab 1 of the same layers, back to back
    adj = ex["adjacent_slabs"]
    a, b = adj["first_slab"], adj["next_slab"]
    first = [st.slot(a, l, p) for l in adj["layers"] for p in range(S)]
    second = [st.slot(b, l, p) for l in adj["layers"] for p in range(S)]
    assert first == list(range(first[0], first[0] + k * S))
    assert second == list(range(first[-1] + 1, first[-1] + 1 + k * S))
    # with those two slabs borrowed, the group's swap is a single transfer
    sw = ex["combined_swap"]
    st.slab_alloc([7] * (n * S))
    st.slab_free([i * S + p for i in range(n) if i not in sw["borrowed_slabs"] for p in range(S)])
    runs = st.group_runs(sw["group"], 0)
    assert len(runs) == sw["transfers"]
    assert runs[0][2] == len(sw["borrowed_slabs"]) * k * S

"""Pins of the oracle's invariant checks: each must reject a state that breaks
the invariant it encodes.

The states are built by hand (owner tags and tables written directly, never
produced by the oracle's operations), one violation each, beside the same
state without the violation, which must pass:

* I1 exactly-once ownership (section 4: a segment belongs to one user at a
  time, enforced by the mapping table): a block referenced twice, an owned
  block missing from every table, an entry owned by another row, an entry
  naming a free or staging block;
* I2 conservation of tags: a lender tag below lim, a borrower or free tag at
  or above lim, a staging or lender tag in the wrong pool, an unknown tag;
* I3 static-dynamic symmetry (sections 3 and 4.1: each GPU always keeps at
  least the memory it contributed): after reclaiming everything, lim above
  zero, a borrower block or a free slot left in the slice, a table still
  naming a slice slot;
* I4 logical view: invariant under a layout change of a block, sensitive to
  one changed element.
"""
import numpy as np
import pytest

import oracle
from oracle import FREE, STAGING, LENDER, InvariantError
from synth import LAYOUT_ATTN, LAYOUT_NHD, pack_block, random_16bit

HKV, D, BS = 1, 128, 16
BB = 2 * BS * HKV * D * 2


def state(local, slc, lim):
    """An oracle slice with the given owner tags (hand-written)."""
    st = oracle.SliceOracle(HKV, D, BS, "f16", LAYOUT_ATTN, len(local) * BB, len(slc) * BB,
                            with_data=False)
    st.own_local[:] = local
    st.own_slice[:] = slc
    st.lim = lim
    return st


# A valid state: 4 local blocks, 4 slice slots, lim 3 (slot 3 is the lender's).
# Sequence 0 holds local 0 and slice slot 1 (unified 5); sequence 1 holds local
# 2 and slice slot 0 (unified 4). Local 1 is staging, local 3 and slot 2 free.
LOCAL = [0, STAGING, 1, FREE]
SLICE = [1, 0, FREE, LENDER]
TABLES = np.array([[[0, 5], [2, 4]]])        # [layer][row][block]


def test_valid_state_passes_every_check():
    st = state(LOCAL, SLICE, 3)
    oracle.check_ownership(st, TABLES)
    oracle.check_conservation(st)


# ---- I1 ------------------------------------------------------------------------

def test_ownership_rejects_a_block_referenced_twice():
    st = state(LOCAL, SLICE, 3)
    t = np.array([[[0, 5], [2, 4]], [[0, -1], [-1, -1]]])     # block 0 again in layer 1
    with pytest.raises(InvariantError, match="referenced twice"):
        oracle.check_ownership(st, t)


def test_ownership_rejects_an_owned_block_missing_from_every_table():
    st = state(LOCAL, SLICE, 3)
    t = np.array([[[0, -1], [2, 4]]])                          # slot 1 (unified 5) dropped
    with pytest.raises(InvariantError, match="not referenced"):
        oracle.check_ownership(st, t)


def test_ownership_rejects_an_entry_owned_by_another_row():
    st = state(LOCAL, SLICE, 3)
    t = np.array([[[0, 4], [2, 5]]])                           # slots swapped between rows
    with pytest.raises(InvariantError, match="owned by"):
        oracle.check_ownership(st, t)


@pytest.mark.parametrize("entry", [1, 3, 6])                   # staging, free local, free slot
def test_ownership_rejects_an_entry_naming_an_unowned_block(entry):
    st = state(LOCAL, SLICE, 3)
    t = np.array([[[0, 5, entry], [2, 4, -1]]])
    with pytest.raises(InvariantError, match="owned by"):
        oracle.check_ownership(st, t)


def test_ownership_respects_the_row_owner_map():
    st = state(LOCAL, SLICE, 3)
    rows_swapped = np.array([[[2, 4], [0, 5]]])
    oracle.check_ownership(st, rows_swapped, row_owner=[1, 0])
    with pytest.raises(InvariantError):
        oracle.check_ownership(st, rows_swapped)


# ---- I2 ------------------------------------------------------------------------

@pytest.mark.parametrize("local,slc,lim,what", [
    (LOCAL, [1, LENDER, FREE, LENDER], 3, "below lim"),        # lender tag below lim
    (LOCAL, [1, 0, FREE, 7], 3, "not the lender"),             # borrower tag above lim
    (LOCAL, [1, 0, FREE, FREE], 3, "not the lender"),          # free slot above lim
    (LOCAL, [1, 0, STAGING, LENDER], 3, "below lim"),          # staging in the slice
    ([0, LENDER, 1, FREE], SLICE, 3, "local block"),           # lender tag in the local pool
    ([0, -9, 1, FREE], SLICE, 3, "local block"),               # unknown tag
    (LOCAL, SLICE, 5, "outside"),                              # lim beyond the pool
])
def test_conservation_rejects_misplaced_tags(local, slc, lim, what):
    with pytest.raises(InvariantError, match=what):
        oracle.check_conservation(state(local, slc, lim))


def test_conservation_accepts_every_lim():
    # the same slot tags are valid for lim = 0 when all are the lender's
    oracle.check_conservation(state(LOCAL, [LENDER] * 4, 0))
    oracle.check_conservation(state(LOCAL, [1, 0, FREE, FREE], 4))


# ---- I3 ------------------------------------------------------------------------

def test_sd_symmetry_accepts_a_fully_reclaimed_slice():
    st = state([0, 1, FREE, FREE], [LENDER] * 4, 0)
    oracle.check_sd_symmetry(st, np.array([[[0, -1], [1, -1]]]))


@pytest.mark.parametrize("slc,lim,what", [
    ([LENDER, LENDER, LENDER, FREE], 1, "lim is 1"),           # something still lent
    ([LENDER, 3, LENDER, LENDER], 0, "still has tag"),         # borrower block left behind
    ([LENDER, LENDER, FREE, LENDER], 0, "still has tag"),      # a free slot not returned
])
def test_sd_symmetry_rejects_a_lender_short_of_its_contribution(slc, lim, what):
    with pytest.raises(InvariantError, match=what):
        oracle.check_sd_symmetry(state([0, 1, FREE, FREE], slc, lim))


def test_sd_symmetry_rejects_a_table_still_naming_the_slice():
    st = state([0, 1, FREE, FREE], [LENDER] * 4, 0)
    with pytest.raises(InvariantError, match="still names slice"):
        oracle.check_sd_symmetry(st, np.array([[[0, 6], [1, -1]]]))


def test_checks_hold_without_assertions():
    # the checks raise, they do not assert: python -O keeps them
    import inspect
    import oracle.invariants as inv
    assert "assert " not in inspect.getsource(inv)


# ---- I4 ------------------------------------------------------------------------

def test_logical_view_is_layout_independent_and_element_exact():
    rng = np.random.default_rng(1)
    K = random_16bit(rng, (HKV, BS, D), "f16")
    V = random_16bit(rng, (HKV, BS, D), "f16")
    st = oracle.SliceOracle(HKV, D, BS, "f16", LAYOUT_NHD, 2 * BB, 2 * BB)
    st.own_local[:] = [0, FREE]
    st.own_slice[:] = [0, FREE]
    st.local[0] = pack_block(K, V, LAYOUT_ATTN)
    st.slice[0] = pack_block(K, V, LAYOUT_NHD)
    a = oracle.logical_view(st, np.array([[[0]]]))[(0, 0, 0)]
    b = oracle.logical_view(st, np.array([[[2]]]))[(0, 0, 0)]   # the slice copy, other layout
    assert np.array_equal(a[0], K) and np.array_equal(a[1], V)
    assert np.array_equal(b[0], K) and np.array_equal(b[1], V)
    V2 = V.copy()
    V2[0, BS - 1, D - 1] ^= 1
    st.slice[0] = pack_block(K, V2, LAYOUT_NHD)
    c = oracle.logical_view(st, np.array([[[2]]]))[(0, 0, 0)]
    assert not np.array_equal(c[1], V)

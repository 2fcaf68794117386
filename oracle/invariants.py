"""Invariants of the slice state.

I1 exactly-once ownership (section 4: a segment is assigned to a single user
   and the mapping table enforces it): every block owned by a sequence appears
   in exactly one canonical table entry, in that sequence's row, and every
   table entry points at a block its row owns.
I2 conservation: every physical block carries exactly one valid tag; slice
   slots at or above lim are the lender's, none below it is.
I3 static-dynamic symmetry (section 3 and 4.1): after reclaiming everything
   lent, the lender holds all of its slots and no borrower block is left in
   the slice.
I4 logical view: the K/V content of every surviving logical block is unchanged
   by block movement (compared layout-independently).
"""
import numpy as np

from .layout import decode_block
from .slice_state import FREE, STAGING, LENDER


def check_ownership(st, tables, row_owner=None):
    """I1. tables: int [L][B][maxblk] canonical tables of unified ids (-1 pad)."""
    tables = np.asarray(tables)
    L, B, _ = tables.shape
    row_owner = np.arange(B) if row_owner is None else np.asarray(row_owner)
    seen = {}
    for l in range(L):
        for b in range(B):
            for u in tables[l, b]:
                u = int(u)
                if u < 0:
                    continue
                o = st.owner(u)
                assert o == int(row_owner[b]), f"entry {u} of row {b} owned by {o}"
                assert u not in seen, f"block {u} referenced twice"
                seen[u] = (l, b)
    owned = [u for u in range(st.n_local + st.n_slice) if st.owner(u) >= 0]
    missing = [u for u in owned if u not in seen]
    assert not missing, f"owned blocks not referenced by any table: {missing[:8]}"


def check_conservation(st):
    """I2."""
    assert np.all((st.own_local >= 0) | (st.own_local == FREE) | (st.own_local == STAGING))
    below = st.own_slice[:st.lim]
    assert np.all((below >= 0) | (below == FREE)), "lender tag below lim"
    assert np.all(st.own_slice[st.lim:] == LENDER), "non-lender tag at or above lim"
    n = (np.sum(st.own_local == FREE) + np.sum(st.own_local == STAGING)
         + np.sum(st.own_local >= 0) + np.sum(st.own_slice == FREE)
         + np.sum(st.own_slice >= 0) + np.sum(st.own_slice == LENDER))
    assert n == st.n_local + st.n_slice


def check_sd_symmetry(st):
    """I3 (call after reclaiming all lent slots)."""
    assert st.lim == 0
    assert np.all(st.own_slice == LENDER)


def logical_view(st, tables):
    """I4 helper: {(l, b, j): (K, V)} of every referenced block, as logical
    uint16 arrays [kv_head][token][channel], independent of pool layout."""
    tables = np.asarray(tables)
    view = {}
    for (l, b, j), u in np.ndenumerate(tables):
        if u < 0:
            continue
        view[(l, b, j)] = decode_block(st.read_block(u), st.layout_of(int(u)), st.kv_heads,
                                       st.head_dim, st.block_size)
    return view

"""Invariants of the slice state.

I1 exactly-once ownership (section 4: a segment is assigned to a single user
   and the mapping table enforces it): every block owned by a sequence appears
   in exactly one canonical table entry, in that sequence's row, and every
   table entry points at a block its row owns.
I2 conservation: every physical block carries exactly one valid tag (local
   blocks: a sequence, FREE or STAGING; slice slots below lim: a sequence or
   FREE; slice slots at or above lim: LENDER).
I3 static-dynamic symmetry (section 3 and 4.1): after reclaiming everything
   lent, the lender holds all of its slots and no borrower block is left in
   the slice (nor referenced by a table, when tables are given).
I4 logical view: the K/V content of every surviving logical block is unchanged
   by block movement (compared layout-independently).

Each check raises InvariantError (an OracleError) naming the first violation;
they use no `assert`, so they hold under `python -O` as well.
"""
import numpy as np

from .layout import decode_block
from .slice_state import ERR_INVAL, FREE, LENDER, STAGING, OracleError


class InvariantError(OracleError):
    """A slice state that breaks one of I1-I3."""

    def __init__(self, msg):
        super().__init__(ERR_INVAL, "invariant: " + msg)


def _require(cond, msg):
    if not cond:
        raise InvariantError(msg)


def check_ownership(st, tables, row_owner=None):
    """I1. tables: int [L][B][maxblk] canonical tables of unified ids (-1 pad);
    row b belongs to sequence row_owner[b] (default: b)."""
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
                _require(o == int(row_owner[b]),
                         f"entry {u} of row {b} (layer {l}) is owned by {o}, not {int(row_owner[b])}")
                _require(u not in seen, f"block {u} referenced twice: {seen.get(u)} and {(l, b)}")
                seen[u] = (l, b)
    owned = [u for u in range(st.n_local + st.n_slice) if st.owner(u) >= 0]
    missing = [u for u in owned if u not in seen]
    _require(not missing, f"owned blocks not referenced by any table: {missing[:8]}")


def check_conservation(st):
    """I2."""
    loc = st.own_local
    bad = np.nonzero(~((loc >= 0) | (loc == FREE) | (loc == STAGING)))[0]
    _require(len(bad) == 0, f"local block {bad[:1].tolist()} has tag "
                            f"{loc[bad[:1]].tolist()} (a local block is owned, FREE or STAGING)")
    _require(0 <= st.lim <= st.n_slice, f"lim {st.lim} outside [0, {st.n_slice}]")
    below = st.own_slice[:st.lim]
    bad = np.nonzero(~((below >= 0) | (below == FREE)))[0]
    _require(len(bad) == 0, f"slice slot {bad[:1].tolist()} below lim {st.lim} has tag "
                            f"{below[bad[:1]].tolist()}")
    above = st.own_slice[st.lim:]
    bad = np.nonzero(above != LENDER)[0]
    _require(len(bad) == 0, f"slice slot {(bad[:1] + st.lim).tolist()} at or above lim "
                            f"{st.lim} is not the lender's")
    n = (np.sum(loc == FREE) + np.sum(loc == STAGING) + np.sum(loc >= 0)
         + np.sum(below == FREE) + np.sum(below >= 0) + np.sum(above == LENDER))
    _require(n == st.n_local + st.n_slice, f"{n} tagged blocks, {st.n_local + st.n_slice} exist")


def check_sd_symmetry(st, tables=None):
    """I3 (call after reclaiming all lent slots): lim is 0, every slice slot is
    the lender's, and no table entry (if tables are given) names a slice slot."""
    _require(st.lim == 0, f"lim is {st.lim} after reclaiming everything")
    bad = np.nonzero(st.own_slice != LENDER)[0]
    _require(len(bad) == 0, f"slice slot {bad[:1].tolist()} still has tag "
                            f"{st.own_slice[bad[:1]].tolist()}: the lender does not hold its "
                            "whole contribution")
    if tables is not None:
        t = np.asarray(tables)
        left = t[t >= st.n_local]
        _require(left.size == 0, f"a table still names slice block {left[:1].tolist()}")


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

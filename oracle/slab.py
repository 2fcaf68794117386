"""Oracle of a slab-managed memory slice (section 4.2.1-4.2.3). TEST
INFRASTRUCTURE ONLY.

The slice is cut into slabs: a slab is ``slab_blocks`` (S) KV-block positions,
the same positions in every one of the cache's L layers, so one slab spans
L x S layer-blocks (slabs are allocated alike in every layer).
A slab belongs to one user at a time: the lender (LENDER), nobody (FREE, lent
but unused) or the borrower (BORROWED). Inside a borrowed slab each position
holds one logical block of one sequence -- in every layer at once -- or is
free. When a sequence needs a block and its slabs are full, the borrower takes
another free slab; a slab whose last position is freed returns to the slice.

Physical placement of layer-block (slab i, layer l, position p) among the
slice slots, with n = number of slabs and k = layers per group:
    layer-major        (l * n + i) * S + p             (section 4.2.1)
    slab-major         (i * L + l) * S + p             (section 4.2.2)
    layer-group-major  ((l // k * n + i) * k + l % k) * S + p   (section 4.2.3)
so a layer group of one slab is k x S contiguous slots in the last two, and in
the layer-group-major layout the same group of the next slab follows it.

Reclaim (section 4.2.1): for each slab the lender takes back it returns a free
slab if there is one (the highest-indexed first), else it picks the borrowed
slab that holds the fewest active requests (ties: the highest index) and
preempts every request with a block in it; a preempted request releases every
block it holds, local or in any slab (the dependency chain of section 4.1),
slabs left empty return to the slice, and the picked slab goes to the lender.

The swap of a layer group (prefetch) copies every borrowed slab's blocks of
the group's layers -- used and unused positions alike, the internal
fragmentation of section 4.2.1 -- into a staging area that is a compact image
of the borrowed slabs in the slice layout's own order: staging block of
(borrowed-slab rank r of m, group layer j, position p) is
    layer-major        (j * m + r) * S + p
    slab-major and layer-group-major   (r * k + j) * S + p.
A swap is issued as maximal runs that are contiguous on both sides.
"""
import numpy as np

from .slice_state import (ERR_INVAL, ERR_NOMEM, ERR_OWNER, FREE, LENDER, LOCAL, STAGING,
                          OracleError, SliceOracle)

LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR = 0, 1, 2
BORROWED = -4          # slab tag: the borrower's


class SlabSliceOracle(SliceOracle):
    def __init__(self, kv_heads, head_dim, block_size, dtype, slice_layout, local_bytes,
                 lent_bytes, layers, slab_blocks, group, slab_layout, with_data=True):
        super().__init__(kv_heads, head_dim, block_size, dtype, slice_layout, local_bytes,
                         lent_bytes, with_data=with_data)
        if layers < 1 or slab_blocks < 1 or group < 1 or layers % group:
            raise OracleError(ERR_INVAL, "slab shape")
        if slab_layout not in (LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR):
            raise OracleError(ERR_INVAL, "slab layout")
        self.L, self.S, self.k, self.slab_layout = layers, slab_blocks, group, slab_layout
        self.n_slabs = self.n_slice // (layers * slab_blocks)
        self.slab_tag = np.full(self.n_slabs, FREE, dtype=np.int64)       # everything lent
        self.pos_owner = np.full(self.n_slabs * slab_blocks, FREE, dtype=np.int64)
        # slots past the last whole slab are never lent
        self.own_slice[self.n_slabs * layers * slab_blocks:] = LENDER
        self.lim = self.n_slice          # per-slot tags carry the state; lim is unused

    # ---- placement ---------------------------------------------------------------
    def slot(self, i, l, p):
        """Slice slot of (slab i, layer l, position p)."""
        n, S, L, k = self.n_slabs, self.S, self.L, self.k
        if self.slab_layout == LAYER_MAJOR:
            return (l * n + i) * S + p
        if self.slab_layout == SLAB_MAJOR:
            return (i * L + l) * S + p
        return ((l // k * n + i) * k + l % k) * S + p

    def block_id(self, pos, layer):
        """Unified id of layer `layer`'s block at slab position `pos` (= i*S + p)."""
        i, p = divmod(int(pos), self.S)
        return self.n_local + self.slot(i, int(layer), p)

    def _set_pos(self, pos, o):
        self.pos_owner[pos] = o
        i, p = divmod(int(pos), self.S)
        for l in range(self.L):
            self.own_slice[self.slot(i, l, p)] = o

    def _set_slab(self, i, tag):
        self.slab_tag[i] = tag
        t = FREE if tag in (FREE, BORROWED) else LENDER
        for l in range(self.L):
            for p in range(self.S):
                self.own_slice[self.slot(i, l, p)] = t
                self.pos_owner[i * self.S + p] = FREE

    def borrowed(self):
        return [i for i in range(self.n_slabs) if self.slab_tag[i] == BORROWED]

    # ---- allocation ----------------------------------------------------------------
    def alloc_blocks(self, where, owners):
        if where != LOCAL:
            raise OracleError(ERR_INVAL, "slab mode: slice blocks come from slab_alloc")
        return super().alloc_blocks(where, owners)

    def free_blocks(self, ids):
        if any(int(u) >= self.n_local for u in ids):
            raise OracleError(ERR_INVAL, "slab mode: slice blocks are freed by slab_free")
        super().free_blocks(ids)

    def slab_alloc(self, owners):
        """One slab position (a logical block in every layer) per owner, in
        order: the lowest free position of the borrowed slabs, slabs in index
        order; when they are full, the lowest-indexed free slab is taken.
        All or nothing. Returns positions i * S + p."""
        owners = [int(o) for o in owners]
        if any(o < 0 for o in owners):
            raise OracleError(ERR_INVAL, "slab owners are sequences")
        free_pos = [i * self.S + p for i in self.borrowed() for p in range(self.S)
                    if self.pos_owner[i * self.S + p] == FREE]
        free_slabs = [i for i in range(self.n_slabs) if self.slab_tag[i] == FREE]
        if len(owners) > len(free_pos) + self.S * len(free_slabs):
            raise OracleError(ERR_NOMEM, "not enough slab positions")
        out = []
        for o in owners:
            if not free_pos:
                i = free_slabs.pop(0)
                self._set_slab(i, BORROWED)
                free_pos = [i * self.S + p for p in range(self.S)]
            pos = free_pos.pop(0)
            self._set_pos(pos, o)
            out.append(pos)
        return np.array(out, dtype=np.int64)

    def _release_empty(self):
        for i in self.borrowed():
            if np.all(self.pos_owner[i * self.S:(i + 1) * self.S] == FREE):
                self._set_slab(i, FREE)

    def slab_free(self, positions):
        """Positions back to free; a borrowed slab left empty returns to the slice."""
        positions = [int(p) for p in positions]
        if len(set(positions)) != len(positions):
            raise OracleError(ERR_INVAL, "duplicate positions")
        for pos in positions:
            if not 0 <= pos < self.n_slabs * self.S:
                raise OracleError(ERR_INVAL, f"position {pos} out of range")
            if self.pos_owner[pos] < 0:
                raise OracleError(ERR_OWNER, f"position {pos} not allocated")
        for pos in positions:
            self._set_pos(pos, FREE)
        self._release_empty()

    def lend(self, n):
        """The lender contributes up to n more slabs (lowest-indexed first)."""
        if n < 0:
            raise OracleError(ERR_INVAL, "n < 0")
        mine = [i for i in range(self.n_slabs) if self.slab_tag[i] == LENDER]
        add = mine[:int(n)]
        for i in add:
            self._set_slab(i, FREE)
        return len(add)

    def active_requests(self, i):
        """Distinct sequences with a block in slab i."""
        own = self.pos_owner[i * self.S:(i + 1) * self.S]
        return sorted({int(o) for o in own if o >= 0})

    def reclaim(self, n, tables=None):
        """The lender takes back n slabs (see the module docstring). Returns
        the slabs taken in order, the preempted requests in order, and the
        rewritten tables (in place): every entry naming a preempted request's
        block becomes -1."""
        n = int(n)
        if n < 0:
            raise OracleError(ERR_INVAL, "n < 0")
        lent = [i for i in range(self.n_slabs) if self.slab_tag[i] != LENDER]
        n_eff = min(n, len(lent))
        taken, victims, released = [], [], []
        for _ in range(n_eff):
            free = [i for i in range(self.n_slabs) if self.slab_tag[i] == FREE]
            if free:
                i = free[-1]
            else:
                cand = self.borrowed()
                i = min(cand, key=lambda s: (len(self.active_requests(s)), -s))
                for r in self.active_requests(i):
                    victims.append(r)
                    for u in range(self.n_local):
                        if self.own_local[u] == r:
                            self.own_local[u] = FREE
                            released.append(u)
                    for pos in np.nonzero(self.pos_owner == r)[0]:
                        released.extend(self.block_id(pos, l) for l in range(self.L))
                        self._set_pos(int(pos), FREE)
                self._release_empty()
            self._set_slab(i, LENDER)
            taken.append(i)
        if tables is not None:
            gone = set(released)
            flat = tables.reshape(-1)
            for e in range(flat.size):
                if int(flat[e]) in gone:
                    flat[e] = -1
        return {"reclaimed": n_eff, "slabs": taken, "victims": victims,
                "released": sorted(released)}

    # ---- layer-group swaps ------------------------------------------------------------
    def stage_index(self, r, m, j, p):
        """Staging offset of (borrowed-slab rank r of m, group layer j, position p)."""
        if self.slab_layout == LAYER_MAJOR:
            return (j * m + r) * self.S + p
        return (r * self.k + j) * self.S + p

    def group_pairs(self, g, stage_first):
        """(source unified id, staging id) of every block the swap of layer
        group g moves, in staging order."""
        slabs = self.borrowed()
        m = len(slabs)
        pairs = []
        for r, i in enumerate(slabs):
            for j in range(self.k):
                for p in range(self.S):
                    src = self.n_local + self.slot(i, g * self.k + j, p)
                    pairs.append((src, stage_first + self.stage_index(r, m, j, p)))
        pairs.sort(key=lambda t: t[1])
        return pairs

    def group_runs(self, g, stage_first):
        """The swap of layer group g as maximal runs (src_first, dst_first,
        length) contiguous on both sides, in staging order."""
        runs = []
        for s, d in self.group_pairs(g, stage_first):
            if runs and runs[-1][0] + runs[-1][2] == s and runs[-1][1] + runs[-1][2] == d:
                runs[-1][2] += 1
            else:
                runs.append([s, d, 1])
        return [tuple(r) for r in runs]

    def prefetch_group(self, g, stage_first):
        """Copy layer group g of every borrowed slab into the staging area
        starting at local block stage_first (which must be STAGING blocks)."""
        if not 0 <= g < self.L // self.k:
            raise OracleError(ERR_INVAL, f"group {g} out of range")
        pairs = self.group_pairs(g, stage_first)
        for _, d in pairs:
            if not (0 <= d < self.n_local) or self.own_local[d] != STAGING:
                raise OracleError(ERR_INVAL, f"staging block {d} is not a staging block")
        for s, d in pairs:
            self._copy(s, d)

    def staged_id(self, pos, layer, stage_first):
        """Where the swap of `layer`'s group puts the block at slab position pos."""
        i, p = divmod(int(pos), self.S)
        slabs = self.borrowed()
        r = slabs.index(i)
        return stage_first + self.stage_index(r, len(slabs), int(layer) % self.k, p)


# ---- invariants of the slab state (raise InvariantError) ------------------------------

def check_slab_tags(st):
    """Every slab is the lender's, free or borrowed; the slots of a lender's
    slab are LENDER and those of a free slab FREE; a borrowed slab holds at
    least one block, and each of its positions carries one owner (or FREE) in
    every layer; slots past the last whole slab are the lender's."""
    from .invariants import InvariantError
    for i in range(st.n_slabs):
        tag = int(st.slab_tag[i])
        if tag not in (LENDER, FREE, BORROWED):
            raise InvariantError(f"slab {i} has tag {tag}")
        own = st.pos_owner[i * st.S:(i + 1) * st.S]
        if tag != BORROWED and np.any(own != FREE):
            raise InvariantError(f"slab {i} is not borrowed but holds blocks")
        if tag == BORROWED and np.all(own == FREE):
            raise InvariantError(f"borrowed slab {i} holds no block")
        for l in range(st.L):
            for p in range(st.S):
                want = LENDER if tag == LENDER else int(own[p])
                got = int(st.own_slice[st.slot(i, l, p)])
                if got != want:
                    raise InvariantError(f"slot of slab {i} layer {l} position {p} has tag "
                                         f"{got}, not {want}")
    tail = st.own_slice[st.n_slabs * st.L * st.S:]
    if np.any(tail != LENDER):
        raise InvariantError("a slot past the last whole slab is lent")


def check_slab_sd_symmetry(st, tables=None):
    """After the lender reclaims every slab: all slabs and slots are the
    lender's, and no table entry names the slice (sections 3 and 4.1)."""
    from .invariants import InvariantError
    if np.any(st.slab_tag != LENDER):
        raise InvariantError(f"slab {int(np.nonzero(st.slab_tag != LENDER)[0][0])} is still lent")
    if np.any(st.own_slice != LENDER):
        raise InvariantError("a slice slot is not the lender's")
    if tables is not None and np.any(np.asarray(tables) >= st.n_local):
        raise InvariantError("a table still names a slice block")

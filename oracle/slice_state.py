"""Oracle of one memory slice plus the local paged KV cache.

Model (EMA section 4, "Memory Slice"): the borrower's local pool and the slice
(the lender's contribution, here a separate region) are arrays of fixed-size
layer-blocks. Every physical block carries one owner tag at a time -- the
mapping table of section 4 guarantees a segment is used by a single user:

    owner >= 0   a sequence (request) of the borrower
    FREE         unused, allocatable
    STAGING      a local block holding a prefetched copy (the swap buffer of
                 section 4.2.2: prefetched data is a copy, placement of the
                 logical block does not change)
    LENDER       a slice slot the lender holds back for itself

``lim`` is how many slice slots are currently lent; slots at or above it are
LENDER. Unified block ids: u < n_local is local block u, u >= n_local is slice
slot u - n_local, -1 is padding.

Operations (each all-or-nothing; on error nothing changes):
* alloc_blocks: take the lowest-index FREE slots (slice: below lim) -- "first
  attempt to allocate from free memory" (section 4.1).
* free_blocks / lend: give blocks back; lend raises lim (the lender contributes
  memory again, section 6.6).
* prefetch: copy slice blocks into STAGING local blocks before use (section 5.1,
  the slice process prefetches ahead of access).
* migrate: move a logical block between pools (copy to a block of the same
  owner).
* kv_append / writeback: a decode step stores each sequence's new token in the
  block holding its position (a slice-resident block is written through its
  staged copy), and the modified staged copies are copied back into their
  slice blocks -- the swap-out that matches the swap-in (section 4: data
  swapped in must be balanced by data swapped out; here only blocks written
  since their prefetch need to travel).
* reclaim(n): the lender takes back n lent slots (section 4.1). It operates on
  logical ownership: borrowed blocks in the returned range move to free space
  when there is room; otherwise whole requests are preempted, and a preempted
  request releases every block it holds, local and remote (the dependency
  chain of section 4.1). See ``reclaim`` for the exact reading.
"""
from collections import Counter
import numpy as np

from .layout import LAYOUT_ATTN, block_bytes, convert_block, decode_block, encode_block

FREE, STAGING, LENDER = -1, -2, -3
LOCAL, SLICE = 0, 1
ERR_INVAL, ERR_NOMEM, ERR_OWNER = -1, -2, -3


class OracleError(Exception):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class SliceOracle:
    def __init__(self, kv_heads, head_dim, block_size, dtype, slice_layout, local_bytes,
                 lent_bytes, with_data=True):
        if dtype not in ("f16", "bf16"):
            raise OracleError(ERR_INVAL, "dtype")
        self.kv_heads, self.head_dim, self.block_size = kv_heads, head_dim, block_size
        self.dtype, self.slice_layout = dtype, slice_layout
        self.bb = block_bytes(kv_heads, head_dim, block_size)
        self.n_local = int(local_bytes // self.bb)
        self.n_slice = int(lent_bytes // self.bb)
        self.lim = self.n_slice
        self.own_local = np.full(self.n_local, FREE, dtype=np.int64)
        self.own_slice = np.full(self.n_slice, FREE, dtype=np.int64)
        self.with_data = with_data
        if with_data:
            self.local = np.zeros((self.n_local, self.bb), dtype=np.uint8)
            self.slice = np.zeros((self.n_slice, self.bb), dtype=np.uint8)

    # ---- helpers -------------------------------------------------------------
    def owner(self, u):
        u = int(u)
        if 0 <= u < self.n_local:
            return int(self.own_local[u])
        s = u - self.n_local
        if 0 <= s < self.n_slice:
            return int(self.own_slice[s])
        raise OracleError(ERR_INVAL, f"id {u} out of range")

    def _set_owner(self, u, o):
        if u < self.n_local:
            self.own_local[u] = o
        else:
            self.own_slice[u - self.n_local] = o

    def layout_of(self, u):
        return LAYOUT_ATTN if u < self.n_local else self.slice_layout

    def read_block(self, u):
        """Bytes of block u in its own pool's layout."""
        u = int(u)
        return self.local[u] if u < self.n_local else self.slice[u - self.n_local]

    def write_block(self, u, data):
        u = int(u)
        if u < self.n_local:
            self.local[u] = data
        else:
            self.slice[u - self.n_local] = data

    def _copy(self, src, dst):
        """dst <- src, re-laid into the destination pool's layout."""
        if not self.with_data:
            return
        data = convert_block(self.read_block(src), self.layout_of(src), self.layout_of(dst),
                             self.kv_heads, self.head_dim, self.block_size)
        self.write_block(dst, data)

    def _in_range(self, u):
        return 0 <= u < self.n_local + self.n_slice

    def free_counts(self):
        return (int(np.sum(self.own_local == FREE)),
                int(np.sum(self.own_slice[:self.lim] == FREE)))

    # ---- allocation ----------------------------------------------------------
    def alloc_blocks(self, where, owners):
        """Allocate len(owners) blocks; the i-th lowest FREE slot gets owners[i].
        STAGING is allowed only in the local pool. Returns unified ids."""
        owners = [int(o) for o in owners]
        for o in owners:
            if o < 0 and o != STAGING:
                raise OracleError(ERR_INVAL, f"bad owner {o}")
            if o == STAGING and where != LOCAL:
                raise OracleError(ERR_INVAL, "staging blocks are local")
        if where == LOCAL:
            free = [u for u in range(self.n_local) if self.own_local[u] == FREE]
        elif where == SLICE:
            free = [self.n_local + s for s in range(self.lim) if self.own_slice[s] == FREE]
        else:
            raise OracleError(ERR_INVAL, f"bad pool {where}")
        if len(free) < len(owners):
            raise OracleError(ERR_NOMEM, f"need {len(owners)} have {len(free)}")
        ids = free[:len(owners)]
        for u, o in zip(ids, owners):
            self._set_owner(u, o)
        return np.array(ids, dtype=np.int64)

    def free_blocks(self, ids):
        ids = [int(u) for u in ids]
        if len(set(ids)) != len(ids):
            raise OracleError(ERR_INVAL, "duplicate ids")
        for u in ids:
            if not self._in_range(u):
                raise OracleError(ERR_INVAL, f"id {u} out of range")
            o = self.owner(u)
            if o == FREE or o == LENDER:
                raise OracleError(ERR_OWNER, f"block {u} not allocated")
        for u in ids:
            self._set_owner(u, FREE)

    def lend(self, n):
        """The lender contributes up to n more slots: lim <- min(n_slice, lim+n)."""
        if n < 0:
            raise OracleError(ERR_INVAL, "n < 0")
        new = min(self.n_slice, self.lim + int(n))
        self.own_slice[self.lim:new] = FREE
        added = new - self.lim
        self.lim = new
        return added

    # ---- copies --------------------------------------------------------------
    def _check_pairs(self, src, dst):
        src = [int(u) for u in src]
        dst = [int(u) for u in dst]
        if len(src) != len(dst):
            raise OracleError(ERR_INVAL, "length mismatch")
        if len(set(dst)) != len(dst):
            raise OracleError(ERR_INVAL, "duplicate destination")
        if set(src) & set(dst):
            raise OracleError(ERR_INVAL, "source and destination overlap")
        for u in src + dst:
            if not self._in_range(u):
                raise OracleError(ERR_INVAL, f"id {u} out of range")
        return src, dst

    def prefetch(self, src, dst):
        """Copy slice blocks src[i] into STAGING local blocks dst[i], in order.
        The slice block is re-laid into the local (ATTN) layout."""
        src, dst = self._check_pairs(src, dst)
        for u in src:
            if u < self.n_local or self.owner(u) < 0:
                raise OracleError(ERR_INVAL, f"prefetch source {u} is not an owned slice block")
        for u in dst:
            if u >= self.n_local or self.owner(u) != STAGING:
                raise OracleError(ERR_INVAL, f"prefetch destination {u} is not a staging block")
        for s, d in zip(src, dst):
            self._copy(s, d)

    def migrate(self, src, dst):
        """Copy owned blocks src[i] into blocks dst[i] of the same owner (any pools)."""
        src, dst = self._check_pairs(src, dst)
        for s, d in zip(src, dst):
            o = self.owner(s)
            if o < 0 or self.owner(d) != o:
                raise OracleError(ERR_INVAL, f"migrate {s}->{d}: owners differ or unowned")
        for s, d in zip(src, dst):
            self._copy(s, d)

    def writeback(self, src, dst):
        """Swap-out of modified staged copies: copy STAGING local blocks src[i]
        back into owned slice blocks dst[i], re-laid into the slice layout (the
        inverse of prefetch; only blocks written since their prefetch need it)."""
        src, dst = self._check_pairs(src, dst)
        for u in src:
            if u >= self.n_local or self.owner(u) != STAGING:
                raise OracleError(ERR_INVAL, f"writeback source {u} is not a staging block")
        for u in dst:
            if u < self.n_local or self.owner(u) < 0:
                raise OracleError(ERR_INVAL, f"writeback destination {u} is not an owned slice block")
        for s, d in zip(src, dst):
            self._copy(s, d)

    def kv_append(self, k16, v16, table, lens):
        """Store the new decode token of every sequence: for sequence b with
        lens[b] > 0 the token at position p = lens[b] - 1 (lens already count
        it) gets K = k16[b], V = v16[b] (uint16 [kv_head][channel]) in row
        p % block_size of local block table[b][p // block_size]. Every target
        must be a local block; nothing is written otherwise."""
        table = np.asarray(table)
        targets = []
        for b, n in enumerate(np.asarray(lens)):
            n = int(n)
            if n <= 0:
                continue
            p = n - 1
            j = p // self.block_size
            if j >= table.shape[1]:
                raise OracleError(ERR_INVAL, f"append: sequence {b} needs block {j}")
            u = int(table[b, j])
            if not (0 <= u < self.n_local):
                raise OracleError(ERR_INVAL, f"append: block {u} of sequence {b} is not local")
            targets.append((b, u, p % self.block_size))
        for b, u, r in targets:
            K, V = decode_block(self.local[u], LAYOUT_ATTN, self.kv_heads, self.head_dim,
                                self.block_size)
            K[:, r, :] = k16[b]
            V[:, r, :] = v16[b]
            self.local[u] = encode_block(K, V, LAYOUT_ATTN)

    # ---- reclaim -------------------------------------------------------------
    def _movers(self, cut):
        return [self.n_local + s for s in range(cut, self.lim) if self.own_slice[s] >= 0]

    def _destinations(self, cut):
        fs = [self.n_local + s for s in range(cut) if self.own_slice[s] == FREE]
        fl = [u for u in range(self.n_local) if self.own_local[u] == FREE]
        return fs + fl

    def reclaim(self, n, tables=None):
        """The lender takes back n lent slots.

        Reading (block-granular, the paper's reclaim is logical):
          1. n' = min(n, lim); the returned range is the top [cut, lim), cut = lim - n'.
          2. movers M: slots in the range owned by a sequence, ascending.
          3. destinations F: FREE slice slots below cut ascending (compaction),
             then FREE local blocks ascending (write-back).
          4. while |M| > |F|: preempt the owner with the most movers (tie: the
             larger owner id); it releases every block it holds anywhere;
             recompute M and F.
          5. copy M[i] -> F[i]; F[i] takes M[i]'s owner.
          6. the range becomes LENDER and lim = cut; every table entry t is
             rewritten to remap(t): a mover's id to its destination, a victim's
             block to -1, anything else unchanged.
        ``tables`` (any int array of unified ids) is rewritten in place.
        """
        n = int(n)
        if n < 0:
            raise OracleError(ERR_INVAL, "n < 0")
        n_eff = min(n, self.lim)
        cut = self.lim - n_eff
        victims, victim_blocks = [], []
        M, F = self._movers(cut), self._destinations(cut)
        while len(M) > len(F):
            counts = Counter(self.owner(u) for u in M)
            victim = max(counts.items(), key=lambda kv: (kv[1], kv[0]))[0]
            victims.append(victim)
            held = [u for u in range(self.n_local + self.n_slice) if self.owner(u) == victim]
            victim_blocks.extend(held)
            for u in held:
                self._set_owner(u, FREE)
            M, F = self._movers(cut), self._destinations(cut)
        moves = list(zip(M, F[:len(M)]))
        for s, d in moves:
            self._copy(s, d)
            self._set_owner(d, self.owner(s))
        remap = {s: d for s, d in moves}
        for u in victim_blocks:
            remap[u] = -1
        self.own_slice[cut:self.lim] = LENDER
        self.lim = cut
        if tables is not None:
            flat = tables.reshape(-1)
            for i in range(flat.size):
                t = int(flat[i])
                if t in remap:
                    flat[i] = remap[t]
        return {
            "reclaimed": n_eff,
            "moved": len(moves),
            "written_back": sum(1 for _, d in moves if d < self.n_local),
            "victims": victims,
            "lim": self.lim,
            "moves": moves,
            "remap": remap,
        }

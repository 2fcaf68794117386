"""Host bookkeeping of the C-ABI library against the oracle, on the CPU.

The library is created host-only (no device memory): allocation, freeing,
lending, copy-list validation and the reclaim planner are the same C++ code
the GPU path runs. Random traces drive the library and the oracle side by side;
ids, error codes, owner tags, lent limit, reclaim plans and rewritten tables
must match exactly after every operation.
"""
import os

import numpy as np
import pytest

import oracle
from slice_trace import Cache, OracleBackend, random_trace

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2609_27040_amd", "lib", "libema_slice.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")

HKV, D, BS = 2, 128, 16
BB = 2 * BS * HKV * D * 2


class LibHostBackend:
    """The library in host-only mode. Table rewriting is the device's job, so
    this adapter applies the returned plan to host tables itself."""

    validating = True     # host-only slices validate every id list

    def __init__(self, n_local, n_slice, layout=0):
        from paper_2609_27040_amd import ema
        self.ema = ema
        self.h = ema.slice_create(HKV, D, BS, "f16", layout, n_local * BB, n_slice * BB,
                                  host_only=True)
        self.n_local = n_local

    def close(self):
        self.ema.slice_destroy(self.h)

    def alloc_blocks(self, where, owners):
        return self.ema.slice_alloc_blocks(self.h, where, owners).astype(np.int64)

    def free_blocks(self, ids):
        self.ema.slice_free_blocks(self.h, ids)

    def lend(self, n):
        return self.ema.slice_lend(self.h, n)

    def migrate(self, src, dst):
        self.ema.slice_migrate(self.h, np.asarray(src), np.asarray(dst))

    def prefetch(self, src, dst):
        self.ema.slice_prefetch(self.h, np.asarray(src), np.asarray(dst))

    def writeback(self, src, dst):
        self.ema.slice_writeback(self.h, np.asarray(src), np.asarray(dst))

    def reclaim(self, n, tables):
        own_l, own_s, _ = self.ema.slice_owners(self.h)
        owners_before = np.concatenate([own_l, own_s])
        r = self.ema.slice_reclaim(self.h, n)
        remap = {int(s): int(d) for s, d in r["moves"]}
        victims = set(r["victims"])
        flat = tables.reshape(-1)
        for i, t in enumerate(flat):
            if t < 0:
                continue
            if int(owners_before[t]) in victims:
                flat[i] = -1
            elif int(t) in remap:
                flat[i] = remap[int(t)]
        return {k: r[k] for k in ("reclaimed", "moved", "written_back", "victims", "lim",
                                  "moves")}

    def owners(self):
        return self.ema.slice_owners(self.h)


def compare_owners(st, lib):
    own_l, own_s, lim = lib.owners()
    assert np.array_equal(own_l, st.own_local) and np.array_equal(own_s, st.own_slice)
    assert lim == st.lim


@pytest.mark.parametrize("seed", range(12))
def test_library_bookkeeping_matches_oracle_on_random_traces(seed):
    rng = np.random.default_rng(1000 + seed)
    n_local, n_slice = int(rng.integers(6, 30)), int(rng.integers(4, 24))
    st = oracle.SliceOracle(HKV, D, BS, "f16", 0, n_local * BB, n_slice * BB, with_data=False)
    lib = LibHostBackend(n_local, n_slice)
    try:
        cache = Cache([OracleBackend(st), lib], layers=3, batch=6, maxblk=5, rng=rng)
        random_trace(cache, 300, rng, on_step=lambda step, op: compare_owners(st, lib))
        cache.reclaim(int(rng.integers(0, n_slice + 3)))
        compare_owners(st, lib)
    finally:
        lib.close()


def test_error_codes_match_the_oracle():
    st = oracle.SliceOracle(HKV, D, BS, "f16", 0, 4 * BB, 4 * BB, with_data=False)
    lib = LibHostBackend(4, 4)
    try:
        cache = Cache([OracleBackend(st), lib], layers=1, batch=2, maxblk=4,
                      rng=np.random.default_rng(0))
        cases = [("alloc_blocks", 0, [0] * 5), ("alloc_blocks", 1, [-2]), ("alloc_blocks", 3, [0]),
                 ("alloc_blocks", 0, [-7]), ("free_blocks", [0]), ("free_blocks", [99]),
                 ("lend", -1), ("migrate", [0], [1]), ("prefetch", [4], [0])]
        for name, *args in cases:
            _, err = cache._all(name, *args)
            assert err is not None, (name, args)
    finally:
        lib.close()


def test_large_pool_reclaim_plan_matches_oracle():
    """A big, fragmented slice: one reclaim of most of the lent range."""
    rng = np.random.default_rng(7)
    n_local, n_slice = 400, 600
    st = oracle.SliceOracle(HKV, D, BS, "f16", 0, n_local * BB, n_slice * BB, with_data=False)
    lib = LibHostBackend(n_local, n_slice)
    try:
        cache = Cache([OracleBackend(st), lib], layers=2, batch=40, maxblk=12, rng=rng)
        for _ in range(300):
            cache.grow(int(rng.integers(2)), int(rng.integers(40)), int(rng.integers(2)),
                       int(rng.integers(1, 6)))
        for b in rng.choice(40, 8, replace=False):
            cache.finish(int(b))
        r = cache.reclaim(450)
        assert r["moved"] > 0
        compare_owners(st, lib)
        oracle.check_ownership(st, cache.tables)
    finally:
        lib.close()


def test_library_reclaim_victim_order_hand_worked():
    """Step 4 of reclaim on the library: owners ranked by movers in the
    returned range, ties to the larger id, preempted until the rest fit."""
    lib = LibHostBackend(3, 6)
    ema = lib.ema
    try:
        lib.alloc_blocks(ema.POOL_LOCAL, [7, 7, 7])
        lib.free_blocks([0, 1])                                    # local 0, 1 free
        lib.alloc_blocks(ema.POOL_SLICE, [5, 6, 2, 2, 3, 3])       # slots 0..5
        r = lib.reclaim(4, np.full((1, 1), -1))                    # range: slots 2..5
        # owners 2 and 3 hold two movers each, two destinations (local 0, 1):
        # the larger id is preempted, owner 2's blocks are written back
        assert r["victims"] == [3] and r["moved"] == 2 and r["written_back"] == 2
        assert np.asarray(r["moves"]).tolist() == [[5, 0], [6, 1]]
        own_l, own_s, lim = lib.owners()
        assert own_l.tolist() == [2, 2, 7] and lim == 2
        assert own_s.tolist()[:2] == [5, 6]
    finally:
        lib.close()
    lib = LibHostBackend(1, 8)
    ema = lib.ema
    try:
        lib.alloc_blocks(ema.POOL_LOCAL, [4])
        lib.alloc_blocks(ema.POOL_SLICE, [1, 4, 9, 9, 4, 1, 1, 1])  # slots 0..7
        r = lib.reclaim(6, np.full((1, 1), -1))                    # range: slots 2..7
        # movers: owner 1 x3, 9 x2, 4 x1; no destinations. Owner 1 goes
        # first (which frees slot 0), then 9; owner 4's mover at slot 4 takes
        # slot 0, and owner 4 keeps its local block
        assert r["victims"] == [1, 9] and r["moves"].tolist() == [[5, 1]]
        own_l, own_s, lim = lib.owners()
        assert own_l.tolist() == [4] and own_s.tolist()[:2] == [4, 4]
    finally:
        lib.close()


def test_library_run_prefetch_validation_host_only():
    """Run prefetches expand to block lists that go through the same checks as
    a prefetch (host-only library: the check runs, no copy)."""
    lib = LibHostBackend(12, 8, layout=1)
    ema = lib.ema
    try:
        lib.alloc_blocks(ema.POOL_SLICE, [0] * 8)                    # slots 12..19
        dst = lib.alloc_blocks(ema.POOL_LOCAL, [ema.STAGING] * 4)    # local 0..3
        ema.slice_prefetch_runs(lib.h, [12, 16], [0, 2], [2, 2])     # valid: 4 blocks
        bad = [([12], [int(dst[0])], [2], ema.ENGINE_DMA),           # engines need the local layout
               ([12], [int(dst[0])], [9], ema.ENGINE_KERNEL),        # run past the pool
               ([12, 13], [0, 0], [1, 1], ema.ENGINE_KERNEL),        # a staging block twice
               ([0], [int(dst[0])], [1], ema.ENGINE_KERNEL),         # source not a slice block
               ([12], [0], [-1], ema.ENGINE_KERNEL),                 # negative run
               ([12], [0], [1], 7)]                                  # unknown engine
        for s, d, k, eng in bad:
            with pytest.raises(ema.EmaError) as e:
                ema.slice_prefetch_runs(lib.h, s, d, k, engine=eng)
            assert e.value.code == ema.ERR_INVAL, (s, d, k, eng)
    finally:
        lib.close()


def test_binding_refuses_arrays_the_kernels_could_not_read():
    """Device entry points take GPU tensors only: the binding refuses host
    arrays, CPU tensors, other dtypes, non-contiguous views and short inputs
    before any pointer reaches the library (a kernel would dereference it)."""
    import torch
    from paper_2609_27040_amd import ema
    ok = torch.zeros(8, dtype=torch.int32)                 # right dtype, but on the CPU
    for bad in (np.zeros(8, np.int32), ok, ok.to(torch.int64), ok[::2]):
        with pytest.raises(ema.EmaError) as e:
            ema._i32_dev(bad, "ids", 4)
        assert e.value.code == ema.ERR_INVAL
    lib = LibHostBackend(4, 4)
    try:
        with pytest.raises(ema.EmaError) as e:                 # host-only: fewer ids than n
            ema.slice_prefetch(lib.h, np.array([4], np.int32), np.array([0], np.int32), 2)
        assert e.value.code == ema.ERR_INVAL
    finally:
        lib.close()

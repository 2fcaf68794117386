"""GPU parity of block movement: prefetch, migrate and reclaim, bit for bit.

Every test compares the whole of both device pools with the oracle's after the
operation (so a stray write anywhere fails), plus owners, lent limit and the
rewritten tables. Everything runs through the C ABI.
"""
import numpy as np
import pytest
import torch

import oracle
from slice_trace import Cache, OracleBackend, random_trace

pytestmark = pytest.mark.gpu

HKV, D = 2, 128


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


def i32(a):
    return torch.as_tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")


class GpuBackend:
    """The library on the GPU, mirrored step by step against the oracle."""

    def __init__(self, ema, bs, layout, dtype, n_local, n_slice, rng, hkv=HKV):
        self.ema = ema
        self.bb = 2 * bs * hkv * D * 2
        self.h = ema.slice_create(hkv, D, bs, dtype, layout, n_local * self.bb, n_slice * self.bb)
        self.n_local = n_local
        self.lv = ema.pool_view(self.h, ema.POOL_LOCAL)
        self.sv = ema.pool_view(self.h, ema.POOL_SLICE)
        self.init_local = rng.integers(0, 256, (n_local, self.bb), dtype=np.uint8)
        self.init_slice = rng.integers(0, 256, (n_slice, self.bb), dtype=np.uint8)
        self.lv.copy_(torch.from_numpy(self.init_local))
        self.sv.copy_(torch.from_numpy(self.init_slice))
        torch.cuda.synchronize()

    def close(self):
        self.lv = self.sv = None
        torch.cuda.synchronize()
        self.ema.slice_destroy(self.h)

    def alloc_blocks(self, where, owners):
        return self.ema.slice_alloc_blocks(self.h, where, owners).astype(np.int64)

    def free_blocks(self, ids):
        self.ema.slice_free_blocks(self.h, ids)

    def lend(self, n):
        return self.ema.slice_lend(self.h, n)

    def migrate(self, src, dst):
        self.ema.slice_migrate(self.h, i32(src), i32(dst))

    def prefetch(self, src, dst):
        self.ema.slice_prefetch(self.h, i32(src), i32(dst))

    def writeback(self, src, dst):
        self.ema.slice_writeback(self.h, i32(src), i32(dst))

    def reclaim(self, n, tables):
        t = i32(tables.reshape(-1))
        r = self.ema.slice_reclaim(self.h, n, t)
        tables.reshape(-1)[:] = t.cpu().numpy()
        return {k: r[k] for k in ("reclaimed", "moved", "written_back", "victims", "lim",
                                  "moves")}

    def pools(self):
        torch.cuda.synchronize()
        return self.lv.cpu().numpy(), self.sv.cpu().numpy()


def make_pair(ema, bs, layout, dtype, n_local, n_slice, seed, hkv=HKV):
    rng = np.random.default_rng(seed)
    gpu = GpuBackend(ema, bs, layout, dtype, n_local, n_slice, rng, hkv)
    st = oracle.SliceOracle(hkv, D, bs, dtype, layout, n_local * gpu.bb, n_slice * gpu.bb)
    st.local[:] = gpu.init_local
    st.slice[:] = gpu.init_slice
    return gpu, st


def assert_pools_equal(gpu, st):
    loc, sli = gpu.pools()
    bad_l = np.nonzero((loc != st.local).any(axis=1))[0]
    bad_s = np.nonzero((sli != st.slice).any(axis=1))[0]
    assert len(bad_l) == 0 and len(bad_s) == 0, f"local blocks {bad_l[:8]}, slice {bad_s[:8]}"
    assert gpu.ema.slice_device_errors(gpu.h) == 0


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("bs,hkv,dtype", [(16, 2, "f16"), (32, 1, "bf16"), (64, 8, "bf16"),
                                          (128, 4, "bf16"), (256, 2, "f16"), (16, 8, "bf16")])
def test_prefetch_matches_oracle_bit_for_bit(ema, layout, bs, hkv, dtype):
    print(f"prefetch layout={layout} bs={bs} hkv={hkv} {dtype}", flush=True)
    n_local, n_slice = 40, 30
    gpu, st = make_pair(ema, bs, layout, dtype, n_local, n_slice, seed=bs + layout, hkv=hkv)
    try:
        rng = np.random.default_rng(5)
        owners = rng.integers(0, 5, n_slice - 3)
        src_all = gpu.alloc_blocks(1, owners)
        st.alloc_blocks(1, owners)
        n = 13                                          # ragged: not a multiple of anything
        dst = gpu.alloc_blocks(0, [-2] * n)
        st.alloc_blocks(0, [-2] * n)
        src = rng.choice(src_all, n, replace=False)
        gpu.prefetch(src, dst[::-1])
        st.prefetch(src, dst[::-1])
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()


@pytest.mark.parametrize("layout", [0, 1])
def test_migrate_both_directions_matches_oracle(ema, layout):
    gpu, st = make_pair(ema, 16, layout, "bf16", 24, 24, seed=11)
    try:
        a = gpu.alloc_blocks(0, [3] * 6); st.alloc_blocks(0, [3] * 6)
        b = gpu.alloc_blocks(1, [3] * 6); st.alloc_blocks(1, [3] * 6)
        gpu.migrate(a, b); st.migrate(a, b)             # local -> slice (re-laid if NHD)
        c = gpu.alloc_blocks(0, [3] * 6); st.alloc_blocks(0, [3] * 6)
        gpu.migrate(b, c); st.migrate(b, c)             # slice -> local
        assert_pools_equal(gpu, st)
        for u, w in zip(a, c):                          # round trip restores the bytes
            assert np.array_equal(st.local[u], st.local[w])
    finally:
        gpu.close()


def test_empty_copy_lists_are_no_ops(ema):
    gpu, st = make_pair(ema, 16, 0, "f16", 8, 8, seed=12)
    try:
        empty = torch.empty(0, dtype=torch.int32, device="cuda")
        ema.slice_prefetch(gpu.h, empty, empty, 0)
        ema.slice_migrate(gpu.h, empty, empty, 0)
        r = ema.slice_reclaim(gpu.h, 0, torch.empty(0, dtype=torch.int32, device="cuda"))
        assert r["reclaimed"] == 0 and r["moved"] == 0
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()


def test_out_of_range_ids_are_skipped_and_counted(ema):
    gpu, st = make_pair(ema, 16, 0, "f16", 8, 8, seed=13)
    try:
        src = gpu.alloc_blocks(1, [0, 0]); st.alloc_blocks(1, [0, 0])
        dst = gpu.alloc_blocks(0, [-2, -2]); st.alloc_blocks(0, [-2, -2])
        ema.slice_prefetch(gpu.h, i32([src[0], 999, src[1]]), i32([dst[0], dst[1], -5]))
        st.prefetch([src[0]], [dst[0]])
        torch.cuda.synchronize()
        assert ema.slice_device_errors(gpu.h) == 2
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()


def test_checked_mode_rejects_invalid_prefetch(ema):
    bb = 2 * 16 * HKV * D * 2
    h = ema.slice_create(HKV, D, 16, "f16", 0, 8 * bb, 8 * bb, checked=True)
    try:
        src = ema.slice_alloc_blocks(h, 1, [0, 0])
        owned = ema.slice_alloc_blocks(h, 0, [1])
        with pytest.raises(ema.EmaError) as e:
            ema.slice_prefetch(h, i32(src[:1]), i32(owned))        # destination not staging
        assert e.value.code == ema.ERR_INVAL
        with pytest.raises(ema.EmaError):
            ema.slice_prefetch(h, i32(src), i32([0, 0]))            # duplicate destination
    finally:
        torch.cuda.synchronize()
        ema.slice_destroy(h)


@pytest.mark.parametrize("seed,layout,bs", [(0, 0, 16), (1, 1, 16), (2, 1, 32), (3, 0, 64)])
def test_random_trace_with_reclaim_matches_oracle(ema, seed, layout, bs):
    print(f"trace seed={seed} layout={layout} bs={bs}", flush=True)
    rng = np.random.default_rng(200 + seed)
    gpu, st = make_pair(ema, bs, layout, "bf16", 28, 20, seed=seed)
    try:
        cache = Cache([OracleBackend(st), gpu], layers=2, batch=5, maxblk=6, rng=rng)
        random_trace(cache, 120, rng)
        cache.reclaim(st.lim)                          # the lender takes everything back
        oracle.check_sd_symmetry(st)
        assert_pools_equal(gpu, st)
        moved = sum(e[2] for e in cache.log if e[0] == "reclaim")
        assert moved > 0
    finally:
        gpu.close()


def test_reclaim_with_writeback_and_preemption_large(ema):
    """Many blocks, reclaim most of the slice: compaction, write-back and
    preemption in one call, tables rewritten on the device."""
    rng = np.random.default_rng(21)
    gpu, st = make_pair(ema, 16, 1, "f16", 300, 400, seed=21, hkv=8)
    try:
        cache = Cache([OracleBackend(st), gpu], layers=2, batch=30, maxblk=16, rng=rng)
        for _ in range(400):
            cache.grow(int(rng.integers(2)), int(rng.integers(30)), int(rng.integers(2)),
                       int(rng.integers(1, 6)))
        r = cache.reclaim(380)
        assert r["moved"] > 0 and r["written_back"] > 0
        assert_pools_equal(gpu, st)
        oracle.check_ownership(st, cache.tables)
    finally:
        gpu.close()


@pytest.mark.parametrize("engine", [0, 1])
def test_prefetch_runs_match_oracle_bit_for_bit(ema, engine):
    """Contiguous runs copied by the gather kernel or the copy engines give the
    same bytes as the oracle's block-by-block prefetch (runs of 1, 3 and 5)."""
    gpu, st = make_pair(ema, 16, 0, "bf16", 30, 20, seed=40 + engine, hkv=2)
    try:
        owners = np.arange(20) % 4
        gpu.alloc_blocks(1, owners)
        st.alloc_blocks(1, owners)
        dst = gpu.alloc_blocks(0, [-2] * 12)
        st.alloc_blocks(0, [-2] * 12)
        nl = st.n_local
        src_first = np.array([nl + 2, nl + 9, nl + 15])
        dst_first = np.array([dst[0], dst[1], dst[4]])
        runs = np.array([1, 3, 5])
        ema.slice_prefetch_runs(gpu.h, src_first, dst_first, runs, engine=engine)
        for a, b, k in zip(src_first, dst_first, runs):
            st.prefetch(list(range(a, a + k)), list(range(b, b + k)))
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()


def test_prefetch_runs_validation(ema):
    gpu, st = make_pair(ema, 16, 1, "bf16", 12, 8, seed=44)
    try:
        gpu.alloc_blocks(1, [0] * 8)
        dst = gpu.alloc_blocks(0, [-2] * 4)
        nl = 12
        cases = [([nl], [dst[0]], [2], 1),            # copy engines need the local layout
                 ([nl], [dst[0]], [9], 0),            # run past the pool
                 ([nl, nl + 1], [dst[0], dst[0]], [1, 1], 0),   # a staging block twice
                 ([0], [dst[0]], [1], 0)]             # source not a slice block
        for s, d, k, eng in cases:
            with pytest.raises(ema.EmaError) as e:
                ema.slice_prefetch_runs(gpu.h, s, d, k, engine=eng)
            assert e.value.code == ema.ERR_INVAL
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()


@pytest.mark.parametrize("first", ["prefetch", "reclaim"])
def test_plan_uploads_on_two_streams_stay_ordered(ema, first):
    """A run prefetch and a reclaim that both upload their plans through the
    handle's shared upload area, issued on two streams with no host
    synchronisation between them; the first call is queued behind a long copy,
    so its kernel has not started when the second call plans and uploads. Both
    pools and the rewritten table must equal the oracle's, which runs the two
    calls one after the other."""
    print(f"two-stream uploads, first={first}", flush=True)
    n_local, n_slice = 34000, 30000
    gpu, st = make_pair(ema, 16, 0, "bf16", n_local, n_slice, seed=77, hkv=1)
    try:
        nl = st.n_local
        owners = np.arange(n_slice) % 50
        ids = gpu.alloc_blocks(1, owners)
        assert np.array_equal(ids, st.alloc_blocks(1, owners))
        # every third slot below the top 3000 freed: the reclaim compacts into
        # scattered slots (3000 runs of one block: its plan is uploaded)
        free = ids[:27000:3]
        gpu.free_blocks(free)
        st.free_blocks(free)
        stage = gpu.alloc_blocks(0, [-2] * 8000)
        assert np.array_equal(stage, st.alloc_blocks(0, [-2] * 8000))
        # 4000 runs of two used slice blocks each into contiguous staging
        # (more runs than the launch arguments carry: the list is uploaded)
        j = np.arange(4000)
        src_first, dst_first, runs = nl + 1 + 3 * j, stage[0] + 2 * j, np.full(4000, 2)
        table = np.setdiff1d(ids, free).astype(np.int64)
        tdev = i32(table)
        big = torch.empty(8 << 30, dtype=torch.uint8, device="cuda")
        big2 = torch.empty_like(big)
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            big2.copy_(big)                            # keeps s1 busy for milliseconds
        pf = lambda s: ema.slice_prefetch_runs(gpu.h, src_first, dst_first, runs, stream=s)
        rc = lambda s: ema.slice_reclaim(gpu.h, 3000, tdev, stream=s)
        if first == "prefetch":
            pf(s1)
            r = rc(s2)
        else:
            r = rc(s1)
            pf(s2)
        torch.cuda.synchronize()
        del big, big2
        for a, b in zip(src_first, dst_first):
            st.prefetch([a, a + 1], [b, b + 1])
        ro = st.reclaim(3000, table)
        assert r["moved"] == ro["moved"] == 3000 and r["victims"] == ro["victims"] == []
        assert np.array_equal(tdev.cpu().numpy(), table)
        assert_pools_equal(gpu, st)
    finally:
        gpu.close()

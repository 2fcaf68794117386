"""Slab-managed slices on the GPU, through the C ABI, against the slab oracle.

A cache of a few sequences whose logical blocks live either locally (every
layer) or at a slab position (every layer, section 4.2.1), with holes: freed
positions and a slab returned to the slice between borrowed ones. For each
placement (layer-, slab-, layer-group-major) and slice layout, every layer
group's swap (both engines where the layout allows the copy engines) is
compared with the oracle's, both pools byte for byte; then decode attention
of every layer through the staged tables against the float64 oracle over the
canonical tables; then slab reclaims (free slabs first, then the slab with the
fewest requests, preempting) with the device table rewrite against the
oracle's tables.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from harness import TORCH_DT, rel_err

pytestmark = pytest.mark.gpu

D = 128


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


def i32(a):
    return torch.as_tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")


class SlabCache:
    """Library handle and oracle side by side, with canonical tables."""

    def __init__(self, ema, layout, slice_layout, L=4, S=3, k=2, n_slabs=16, hkv=2, bs=16,
                 dtype="bf16", B=5, seed=0):
        self.ema, self.L, self.S, self.k, self.hkv, self.bs, self.dtype = \
            ema, L, S, k, hkv, bs, dtype
        rng = np.random.default_rng(seed)
        self.rng = rng
        bb = oracle.block_bytes(hkv, D, bs)
        self.lens = rng.integers(1, 6 * bs, B)
        self.lens[0] = bs                     # one exactly full block
        nb = (self.lens + bs - 1) // bs
        self.maxblk = int(nb.max())
        n_local = int(nb.sum()) * L + n_slabs * k * S * 2 + 8
        n_slice = n_slabs * L * S + 5
        self.h = ema.slice_create(hkv, D, bs, dtype, slice_layout, n_local * bb, n_slice * bb)
        ema.slab_init(self.h, L, S, k, layout)
        self.st = st = oracle.SlabSliceOracle(hkv, D, bs, dtype, slice_layout, n_local * bb,
                                              n_slice * bb, layers=L, slab_blocks=S, group=k,
                                              slab_layout=layout)
        st.local[:] = synth.random_16bit(rng, (n_local, bb // 2), dtype).view(np.uint8) \
            .reshape(n_local, bb)
        st.slice[:] = synth.random_16bit(rng, (n_slice, bb // 2), dtype).view(np.uint8) \
            .reshape(n_slice, bb)
        self.lv = ema.pool_view(self.h, ema.POOL_LOCAL)
        self.sv = ema.pool_view(self.h, ema.POOL_SLICE)
        self.lv.copy_(torch.from_numpy(st.local))
        self.sv.copy_(torch.from_numpy(st.slice))
        # logical blocks in a seeded random order, ~60 % at slab positions
        self.tables = np.full((L, B, self.maxblk), -1, dtype=np.int64)
        self.pos = {}
        order = [(b, j) for b in range(B) for j in range(nb[b])]
        order = [order[i] for i in rng.permutation(len(order))]
        for b, j in order:
            if rng.random() < 0.6:
                p = int(ema.slab_alloc(self.h, [b])[0])
                assert p == int(st.slab_alloc([b])[0])
                self.pos[(b, j)] = p
                self.tables[:, b, j] = [st.block_id(p, l) for l in range(L)]
            else:
                ids = ema.slice_alloc_blocks(self.h, ema.POOL_LOCAL, [b] * L)
                assert np.array_equal(ids, st.alloc_blocks(oracle.LOCAL, [b] * L))
                self.tables[:, b, j] = ids
        # holes: one sequence's slab positions freed, and extra positions
        # allocated then freed to leave a free slab between borrowed ones
        extra = ema.slab_alloc(self.h, [B] * (2 * S))
        assert np.array_equal(extra, st.slab_alloc([B] * (2 * S)))
        ema.slab_free(self.h, extra[:S + 1])
        st.slab_free(extra[:S + 1])
        self.extra = extra[S + 1:]
        self.q16 = synth.random_16bit(rng, (B, 4 * hkv, D), dtype)
        self.q = torch.from_numpy(self.q16.view(np.int16)).cuda().view(TORCH_DT[dtype])
        self.lens_dev = i32(self.lens)
        self.B = B
        torch.cuda.synchronize()

    def staging(self):
        """A staging image per group slot (two), contiguous local blocks."""
        m = len(self.st.borrowed())
        n = m * self.k * self.S
        ids = self.ema.slice_alloc_blocks(self.h, self.ema.POOL_LOCAL, [self.ema.STAGING] * (2 * n))
        assert np.array_equal(ids, self.st.alloc_blocks(oracle.LOCAL, [oracle.STAGING] * (2 * n)))
        assert np.array_equal(np.diff(ids), np.ones(len(ids) - 1)) if len(ids) > 1 else True
        return [int(ids[0]), int(ids[0]) + n] if n else [0, 0]

    def attn_table(self, l, first):
        t = self.tables[l].copy()
        for (b, j), p in self.pos.items():
            t[b, j] = self.ema.slab_block_ids(self.h, [p], l, first)[0]
        return t

    def close(self):
        self.lv = self.sv = None
        torch.cuda.synchronize()
        self.ema.slice_destroy(self.h)


def _reader(st):
    return lambda u: oracle.convert_block(st.read_block(u), st.layout_of(int(u)),
                                          oracle.LAYOUT_ATTN, st.kv_heads, st.head_dim,
                                          st.block_size)


@pytest.mark.parametrize("layout", [oracle.LAYER_MAJOR, oracle.SLAB_MAJOR, oracle.GROUP_MAJOR])
@pytest.mark.parametrize("slice_layout", [0, 1])
def test_group_swaps_attention_and_reclaim_match_the_oracle(ema, layout, slice_layout):
    print(f"slab layout={layout} slice_layout={slice_layout}", flush=True)
    c = SlabCache(ema, layout, slice_layout, seed=10 * layout + slice_layout)
    st = c.st
    try:
        firsts = c.staging()
        engines = [ema.ENGINE_KERNEL] + ([ema.ENGINE_DMA] if slice_layout == 0 else [])
        out = torch.empty((c.B, 4 * c.hkv, D), device="cuda")
        for eng in engines:
            for g in range(c.L // c.k):
                first = firsts[g % 2]
                # runs agree with the oracle's
                a, d, n = ema.slab_group_runs(c.h, g, first)
                assert list(zip(a.tolist(), d.tolist(), n.tolist())) == st.group_runs(g, first)
                ema.slab_prefetch_group(c.h, g, first, eng)
                st.prefetch_group(g, first)
                for l in range(g * c.k, (g + 1) * c.k):
                    tab = c.attn_table(l, first)
                    ema.paged_decode_attention(c.h, c.q, i32(tab), c.lens_dev, out)
                    torch.cuda.synchronize()
                    ref = oracle.paged_decode_attention(c.q16, c.tables[l], c.lens, _reader(st),
                                                        c.hkv, D, c.bs, c.dtype)
                    assert rel_err(out.cpu().numpy(), ref) <= 2e-3, (eng, l)
            torch.cuda.synchronize()
            assert np.array_equal(c.lv.cpu().numpy(), st.local), eng
            assert np.array_equal(c.sv.cpu().numpy(), st.slice), eng
        # reclaims: the device rewrites the tables as the oracle does (the
        # positions held outside the tables are returned first)
        ema.slab_free(c.h, c.extra)
        st.slab_free(c.extra)
        oracle.check_ownership(st, c.tables)
        tables_dev = i32(c.tables)
        for n in (1, 2, 10 ** 6):
            r = ema.slab_reclaim(c.h, n, tables_dev.view(-1))
            ro = st.reclaim(n, c.tables)
            assert r["slabs"] == ro["slabs"] and r["victims"] == ro["victims"]
            torch.cuda.synchronize()
            assert np.array_equal(tables_dev.cpu().numpy(), c.tables)
            oracle.check_ownership(st, c.tables)
            oracle.check_slab_tags(st)
        oracle.check_slab_sd_symmetry(st, c.tables)
        assert ema.slice_device_errors(c.h) == 0
    finally:
        c.close()


def test_swap_lists_follow_the_borrowed_set(ema):
    """The device keeps every group's source list; after the borrowed set
    changes (a slab returned, another borrowed) the next swap must use the new
    one: staging compared with the oracle after each change."""
    print("slab lists rebuild", flush=True)
    c = SlabCache(ema, oracle.GROUP_MAJOR, 0, seed=3)
    st = c.st
    try:
        first = c.staging()[0]
        ema.slab_prefetch_group(c.h, 1, first)
        st.prefetch_group(1, first)
        # return the extra sequence's last positions (a slab empties), then
        # borrow one more slab for a new sequence
        ema.slab_free(c.h, c.extra)
        st.slab_free(c.extra)
        p = ema.slab_alloc(c.h, [7] * c.S)
        assert np.array_equal(p, st.slab_alloc([7] * c.S))
        m = len(st.borrowed())
        need = m * c.k * c.S
        ids = ema.slice_alloc_blocks(c.h, ema.POOL_LOCAL, [ema.STAGING] * need)
        st.alloc_blocks(oracle.LOCAL, [oracle.STAGING] * need)
        ema.slab_prefetch_group(c.h, 0, int(ids[0]))
        st.prefetch_group(0, int(ids[0]))
        torch.cuda.synchronize()
        assert np.array_equal(c.lv.cpu().numpy(), st.local)
        assert ema.slice_device_errors(c.h) == 0
    finally:
        c.close()


@pytest.mark.parametrize("mode", ["serial", "overlap"])
@pytest.mark.parametrize("engine", [0, 1])
@pytest.mark.parametrize("S,k", [(1, 1), (3, 2), (10, 4)])
def test_slab_step_matches_the_oracle(ema, engine, S, k, mode):
    """The bench's slab step (workloads.slabs) on a scaled-down 8B-shaped
    cache with interleaved free slabs: one full step (every group's swap and
    every layer's attention, on one stream or with the swaps on a second),
    whose last layer's output is checked, then every layer's attention through
    its staged table against the float64 oracle over the canonical blocks."""
    from paper_2609_27040_amd.step import StepRunner
    from workloads.slabs import slab_cache
    print(f"slab step engine={engine} S={S} k={k} mode={mode}", flush=True)
    cfg = synth.LLAMA8B.scaled(layers=4, batch=6, lens=("uniform", 40, 300))
    c = slab_cache(cfg, S, k, engine=engine, seed=100 + S)
    try:
        runs = [c.group_runs(g) for g in range(len(c.groups))]
        assert all(int(r[2].sum()) == c.swap_blocks() for r in runs)
        runner = StepRunner(c, mode)
        out = c.new_out()
        lv = c.local_view.cpu().numpy()
        sv = c.slice_view.cpu().numpy()

        def read(u):
            return lv[u] if u < c.n_local else sv[u - c.n_local]
        runner.run(out)
        torch.cuda.synchronize()
        last = c.L - 1
        ref = oracle.paged_decode_attention(c.q16, c.tables[last], c.lens, read, c.hkv, D,
                                            c.bs, c.dtype)
        assert rel_err(out.cpu().numpy(), ref) <= 2e-3, "step output of the last layer"
        for l in range(c.L):
            # an image holds the last group swapped into it: swap l's group again
            c.prefetch_group(l // k)
            ema.paged_decode_attention(c.h, c.q, c.attn_dev[l], c.lens_dev, out)
            torch.cuda.synchronize()
            ref = oracle.paged_decode_attention(c.q16, c.tables[l], c.lens, read, c.hkv, D,
                                                c.bs, c.dtype)
            assert rel_err(out.cpu().numpy(), ref) <= 2e-3, l
        assert ema.slice_device_errors(c.h) == 0
    finally:
        c.close()


def test_slab_step_full_size_sampled(ema):
    """The slab sweep's configuration at its real size (the 8B-shaped cache,
    32 layers, batch 64, 10-block slabs, groups of 4, layer-group-major, a
    seeded half of the slabs set aside): one full step on one stream, then for
    three layers the attention through the staged tables on sampled sequences
    against the float64 oracle over the canonical blocks, and the staged copies
    of those sequences' slab blocks equal to their slice blocks."""
    from paper_2609_27040_amd.step import StepRunner
    from harness import read_blocks
    from workloads.slabs import slab_cache
    print("slab step full size", flush=True)
    c = slab_cache(synth.LLAMA8B, 10, 4)
    rng = np.random.default_rng(9)
    try:
        runner = StepRunner(c, "serial")
        out = c.new_out()
        runner.run(out)
        torch.cuda.synchronize()
        for l in (0, 17, 31):
            c.prefetch_group(l // c.group)
            ema.paged_decode_attention(c.h, c.q, c.attn_dev[l], c.lens_dev, out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            for b in rng.choice(c.B, size=3, replace=False):
                nb = (int(c.lens[b]) + c.bs - 1) // c.bs
                canon = c.tables[l, b, :nb]
                staged = c.attn_tables[l, b, :nb]
                loc = read_blocks(c.local_view, canon[canon < c.n_local])
                sli = read_blocks(c.slice_view, canon[canon >= c.n_local] - c.n_local)

                def read(u, loc=loc, sli=sli):
                    return loc[int(u)] if u < c.n_local else sli[int(u) - c.n_local]
                ref = oracle.paged_decode_attention(c.q16[b:b + 1], c.tables[l, b:b + 1],
                                                    c.lens[b:b + 1], read, c.hkv, D, c.bs,
                                                    c.dtype)
                assert rel_err(got[b:b + 1], ref) <= 2e-3, (l, b)
                st = read_blocks(c.local_view, staged[canon >= c.n_local])
                for u, s in zip(staged[canon >= c.n_local], canon[canon >= c.n_local]):
                    assert np.array_equal(st[int(u)], sli[int(s) - c.n_local]), (l, b, u)
        assert ema.slice_device_errors(c.h) == 0
    finally:
        c.close()

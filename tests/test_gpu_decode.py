"""Decode steps that grow the cache, through the C ABI: every step each
sequence gains one token (a new block, local or in the slice, when it crosses a
block boundary); per layer the slice-resident blocks are prefetched into
staging, the new token's K/V is appended through the attention table (into the
staged copy when its block lives in the slice), attention runs, and the
modified staged copies are written back to the slice. An oracle replays the
same operations; attention is compared every layer and step, both pools byte
for byte at the end. Plus append parity and validation on their own.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from harness import TORCH_DT, Workload, oracle_mirror, rel_err

pytestmark = pytest.mark.gpu

HKV, D, BS = 2, 128, 16


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


def i32(a):
    return torch.as_tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")


def u16_dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(TORCH_DT[dtype])


def _pair(ema, dtype="bf16", n_local=20, n_slice=6, checked=False, seed=0):
    bb = oracle.block_bytes(HKV, D, BS)
    h = ema.slice_create(HKV, D, BS, dtype, 0, n_local * bb, n_slice * bb, checked=checked)
    st = oracle.SliceOracle(HKV, D, BS, dtype, 0, n_local * bb, n_slice * bb)
    rng = np.random.default_rng(seed)
    st.local[:] = rng.integers(0, 256, st.local.shape, dtype=np.uint8)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)
    lv, sv = ema.pool_view(h, ema.POOL_LOCAL), ema.pool_view(h, ema.POOL_SLICE)
    lv.copy_(torch.from_numpy(st.local))
    sv.copy_(torch.from_numpy(st.slice))
    torch.cuda.synchronize()
    return h, st, lv, sv, rng


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_kv_append_matches_oracle_bit_for_bit(ema, dtype):
    h, st, lv, sv, rng = _pair(ema, dtype)
    try:
        B = 6
        table = np.full((B, 3), -1, dtype=np.int64)
        for b in range(B):
            table[b] = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [b] * 3)
            st.alloc_blocks(oracle.LOCAL, [b] * 3)
        lens = np.array([0, 1, 16, 17, 33, 48])      # empty, rows 0, 15, 0, 0, 15
        k = synth.random_16bit(rng, (B, HKV, D), dtype)
        v = synth.random_16bit(rng, (B, HKV, D), dtype)
        ema.kv_append(h, u16_dev(k, dtype), u16_dev(v, dtype), i32(table), i32(lens))
        st.kv_append(k, v, table, lens)
        torch.cuda.synchronize()
        assert np.array_equal(lv.cpu().numpy(), st.local)
        assert np.array_equal(sv.cpu().numpy(), st.slice)
        assert ema.slice_device_errors(h) == 0
    finally:
        lv = sv = None
        torch.cuda.synchronize()
        ema.slice_destroy(h)


def test_kv_append_invalid_targets(ema):
    # checked mode: rejected on the host, nothing written
    h, st, lv, sv, rng = _pair(ema, checked=True, seed=1)
    try:
        loc = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [0])
        sli = ema.slice_alloc_blocks(h, ema.POOL_SLICE, [1])
        k = synth.random_16bit(rng, (2, HKV, D), "bf16")
        for table, lens in (([[loc[0]], [sli[0]]], [1, 1]),       # a slice block
                            ([[loc[0]], [loc[0]]], [1, BS + 1])):  # past the table
            with pytest.raises(ema.EmaError) as e:
                ema.kv_append(h, u16_dev(k, "bf16"), u16_dev(k, "bf16"), i32(table), i32(lens))
            assert e.value.code == ema.ERR_INVAL
        torch.cuda.synchronize()
        assert np.array_equal(lv.cpu().numpy(), st.local)
    finally:
        lv = sv = None
        torch.cuda.synchronize()
        ema.slice_destroy(h)
    # unchecked: the kernel skips and counts them, valid rows are still written
    h, st, lv, sv, rng = _pair(ema, seed=2)
    try:
        loc = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [0, 1])
        st.alloc_blocks(oracle.LOCAL, [0, 1])
        sli = ema.slice_alloc_blocks(h, ema.POOL_SLICE, [2])
        st.alloc_blocks(oracle.SLICE, [2])
        k = synth.random_16bit(rng, (3, HKV, D), "bf16")
        table = np.array([[loc[0]], [sli[0]], [loc[1]]])
        lens = np.array([3, 1, BS + 2])                # ok, slice id, past the table
        ema.kv_append(h, u16_dev(k, "bf16"), u16_dev(k, "bf16"), i32(table), i32(lens))
        st.kv_append(k[:1], k[:1], table[:1], lens[:1])
        torch.cuda.synchronize()
        assert ema.slice_device_errors(h) == 2
        assert np.array_equal(lv.cpu().numpy(), st.local)
        assert np.array_equal(sv.cpu().numpy(), st.slice)
    finally:
        lv = sv = None
        torch.cuda.synchronize()
        ema.slice_destroy(h)


@pytest.mark.parametrize("layout", [0, 1])
def test_writeback_matches_oracle_bit_for_bit(ema, layout):
    bb = oracle.block_bytes(HKV, D, BS)
    h = ema.slice_create(HKV, D, BS, "bf16", layout, 16 * bb, 12 * bb)
    st = oracle.SliceOracle(HKV, D, BS, "bf16", layout, 16 * bb, 12 * bb)
    rng = np.random.default_rng(7 + layout)
    st.local[:] = rng.integers(0, 256, st.local.shape, dtype=np.uint8)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)
    lv, sv = ema.pool_view(h, ema.POOL_LOCAL), ema.pool_view(h, ema.POOL_SLICE)
    lv.copy_(torch.from_numpy(st.local))
    sv.copy_(torch.from_numpy(st.slice))
    try:
        owners = rng.integers(0, 4, 9)
        dst = ema.slice_alloc_blocks(h, ema.POOL_SLICE, owners)
        st.alloc_blocks(oracle.SLICE, owners)
        src = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [ema.STAGING] * 9)
        st.alloc_blocks(oracle.LOCAL, [oracle.STAGING] * 9)
        perm = rng.permutation(9)
        ema.slice_writeback(h, i32(src[perm]), i32(dst))
        st.writeback(src[perm], dst)
        torch.cuda.synchronize()
        assert np.array_equal(lv.cpu().numpy(), st.local)
        assert np.array_equal(sv.cpu().numpy(), st.slice)
        assert ema.slice_device_errors(h) == 0
    finally:
        lv = sv = None
        torch.cuda.synchronize()
        ema.slice_destroy(h)


@pytest.mark.parametrize("layout", [0, 1])
def test_decode_steps_with_append_and_writeback_match_oracle(ema, layout):
    print(f"decode loop layout={layout}", flush=True)
    cfg = synth.LLAMA8B.scaled(layers=3, batch=6)
    L, B, steps = 3, 6, 24
    lens0 = [1, 15, 16, 17, 40, 100]
    grow = B * (steps // cfg.block_size + 2)          # new blocks per layer, at most
    w = Workload(cfg, layers=L, lens=lens0, slice_layout=layout, fill="host",
                 stage_n=grow + 64, extra_local=L * grow, extra_slice=L * grow)
    try:
        st = oracle_mirror(w)
        rng = np.random.default_rng(11 + layout)
        bs, nl = w.bs, w.n_local
        width = w.maxblk + steps // bs + 2
        tables = np.full((L, B, width), -1, dtype=np.int64)
        tables[:, :, :w.maxblk] = w.tables
        w.tables = tables
        w.tables_dev = torch.from_numpy(tables.astype(np.int32)).cuda()
        lens = np.asarray(lens0, dtype=np.int64)
        out = w.new_out()
        errs = []
        for step in range(steps):
            lens = lens + 1
            for b in range(B):
                j = (lens[b] - 1) // bs
                if (lens[b] - 1) % bs:
                    continue
                for l in range(L):                     # a new block, local or in the slice
                    pool = ema.POOL_SLICE if rng.random() < 0.5 else ema.POOL_LOCAL
                    u = ema.slice_alloc_blocks(w.h, pool, [b])
                    assert np.array_equal(u, st.alloc_blocks(pool, [b]))
                    tables[l, b, j] = int(u[0])
            w.lens = lens.copy()
            w.lens_dev = torch.from_numpy(lens.astype(np.int32)).cuda()
            w.restage()
            for l in range(L):
                w.prefetch(l)
                st.prefetch(w.pf_src[l], w.pf_dst[l])
                k = synth.random_16bit(rng, (B, w.hkv, w.D), cfg.dtype)
                v = synth.random_16bit(rng, (B, w.hkv, w.D), cfg.dtype)
                ema.kv_append(w.h, u16_dev(k, cfg.dtype), u16_dev(v, cfg.dtype), w.attn_dev[l],
                              w.lens_dev)
                st.kv_append(k, v, w.attn_tables[l], lens)
                w.attention(l, out)
                ref = oracle.paged_decode_attention(w.q16, w.attn_tables[l], lens,
                                                    lambda u: st.local[u], w.hkv, w.D, bs,
                                                    cfg.dtype)
                errs.append(rel_err(out.cpu().numpy(), ref))
                assert errs[-1] <= 2e-3, f"step {step} layer {l}: rel err {errs[-1]}"
                last = (lens - 1) // bs
                canon = tables[l, np.arange(B), last]
                dirty = canon >= nl
                src = w.attn_tables[l][np.arange(B), last][dirty]
                if dirty.any():
                    ema.slice_writeback(w.h, i32(src), i32(canon[dirty]))
                    st.writeback(src, canon[dirty])
        torch.cuda.synchronize()
        assert np.array_equal(w.local_view.cpu().numpy(), st.local)
        assert np.array_equal(w.slice_view.cpu().numpy(), st.slice)
        assert ema.slice_device_errors(w.h) == 0
        print(f"max rel err {max(errs):.2e} over {len(errs)} layer-steps", flush=True)
    finally:
        w.close()


@pytest.mark.parametrize("layout,mode,group", [(0, "overlap", 1), (1, "overlap", 1),
                                               (0, "serial", 2), (1, "overlap", 2)])
def test_step_runner_append_reaches_every_block(ema, layout, mode, group):
    """A step with append (either schedule, layer groups of 1 or 2): after one
    step every sequence's last block, in every layer, holds the new token's K/V
    at its row -- read from the slice block itself where the block lives in the
    slice (written back)."""
    from harness import StepRunner
    cfg = synth.LLAMA8B.scaled(layers=4, batch=5)
    w = Workload(cfg, layers=4, lens=[1, 16, 17, 40, 95], slice_layout=layout, fill="device",
                 frac=0.5, group=group, staging_slots=2 * group)
    try:
        runner = StepRunner(w, mode, append=True)
        out = w.new_out()
        runner.run(out)
        torch.cuda.synchronize()
        k_new, v_new = (t.view(torch.int16).cpu().numpy().view(np.uint16) for t in runner.kv_new)
        for l in range(w.L):
            for b in range(w.B):
                p = int(w.lens[b]) - 1
                u = int(w.tables[l, b, p // w.bs])
                if u >= w.n_local:
                    blk, lay = w.slice_view[u - w.n_local].cpu().numpy(), layout
                else:
                    blk, lay = w.local_view[u].cpu().numpy(), synth.LAYOUT_ATTN
                K, V = synth.unpack_block(blk, lay, w.hkv, w.bs, w.D)
                assert np.array_equal(K[:, p % w.bs], k_new[b]), (l, b)
                assert np.array_equal(V[:, p % w.bs], v_new[b]), (l, b)
        assert sum(len(s) for s in w.wb_src) > 0          # some blocks were written back
        assert ema.slice_device_errors(w.h) == 0
    finally:
        w.close()


def test_captured_step_replays_match_eager(ema):
    """The one-stream step (layer groups of 2, with append and write-back)
    captured as a HIP graph: every replay, with eager work and
    synchronisations between replays, leaves the same output and the same
    pools, byte for byte, as an eager step."""
    from harness import StepRunner, capture_step
    cfg = synth.LLAMA8B.scaled(layers=4, batch=6)
    w = Workload(cfg, layers=4, lens=[1, 16, 17, 40, 95, 300], fill="device", frac=0.5,
                 group=2, staging_slots=4)
    try:
        runner = StepRunner(w, "serial", append=True)
        out = w.new_out()
        for _ in range(2):
            runner.run(out)
        torch.cuda.synchronize()
        ref_out = out.clone()
        ref_local, ref_slice = w.local_view.clone(), w.slice_view.clone()
        g = capture_step(runner, out)
        other = w.new_out()
        for rep in range(3):
            out.zero_()
            w.attention(rep % w.L, other)                 # eager work between replays
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, ref_out), rep
            assert torch.equal(w.local_view, ref_local), rep
            assert torch.equal(w.slice_view, ref_slice), rep
        assert ema.slice_device_errors(w.h) == 0
        del g
    finally:
        w.close()



@pytest.mark.parametrize("bs", [16, 32, 64, 128, 256])
@pytest.mark.parametrize("hkv", [1, 8])
def test_relayout_both_directions_every_block_size(ema, bs, hkv):
    """Token-major slice: write-back (local layout -> slice layout), migration
    into the slice and migration out of it at every block size, both whole
    pools byte-equal to the oracle. The relayout units change shape with the
    block size (16-, 32- and 64-token units), so each size is its own case."""
    print(f"relayout bs={bs} hkv={hkv}", flush=True)
    bb = oracle.block_bytes(hkv, D, bs)
    n_l, n_s = 14, 12
    h = ema.slice_create(hkv, D, bs, "f16", 1, n_l * bb, n_s * bb)
    st = oracle.SliceOracle(hkv, D, bs, "f16", 1, n_l * bb, n_s * bb)
    rng = np.random.default_rng(bs * 10 + hkv)
    st.local[:] = rng.integers(0, 256, st.local.shape, dtype=np.uint8)
    st.slice[:] = rng.integers(0, 256, st.slice.shape, dtype=np.uint8)
    lv, sv = ema.pool_view(h, ema.POOL_LOCAL), ema.pool_view(h, ema.POOL_SLICE)
    lv.copy_(torch.from_numpy(st.local))
    sv.copy_(torch.from_numpy(st.slice))
    try:
        def both(call, *args):
            getattr(ema, call)(h, *[i32(a) for a in args])
            getattr(st, call.replace("slice_", ""))(*args)
        # write-back: 4 staged local blocks -> 4 slice blocks (scattered order)
        sdst = ema.slice_alloc_blocks(h, ema.POOL_SLICE, [0, 1, 2, 3])
        st.alloc_blocks(oracle.SLICE, [0, 1, 2, 3])
        stg = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [ema.STAGING] * 4)
        st.alloc_blocks(oracle.LOCAL, [oracle.STAGING] * 4)
        both("slice_writeback", stg[[2, 0, 3, 1]], sdst)
        # migrate into the slice: 3 local blocks of sequence 5
        lsrc = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [5, 5, 5])
        st.alloc_blocks(oracle.LOCAL, [5, 5, 5])
        sdst2 = ema.slice_alloc_blocks(h, ema.POOL_SLICE, [5, 5, 5])
        st.alloc_blocks(oracle.SLICE, [5, 5, 5])
        both("slice_migrate", lsrc, sdst2[::-1])
        # migrate out of the slice: sequence 1's and 2's slice blocks -> local
        ldst = ema.slice_alloc_blocks(h, ema.POOL_LOCAL, [1, 2])
        st.alloc_blocks(oracle.LOCAL, [1, 2])
        both("slice_migrate", sdst[[1, 2]], ldst)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(h) == 0
        assert np.array_equal(lv.cpu().numpy(), st.local)
        assert np.array_equal(sv.cpu().numpy(), st.slice)
    finally:
        lv = sv = None
        torch.cuda.synchronize()
        ema.slice_destroy(h)

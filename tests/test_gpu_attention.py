"""GPU parity of paged decode attention against the float64 oracle.

Bar: max over (sequence, query head) of ||o - ref||_inf / ||ref||_inf <= 2e-3
(16-bit inputs, fp32 accumulation and fp32 output). Unused tail token slots
hold NaN so masking is exercised; staging blocks start as a sentinel.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from harness import Workload, elem_err, oracle_mirror, read_blocks, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-3


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


@pytest.fixture(params=["stream-k", "grid"])
def impl(request):
    """Attention schedule, chosen when the slice is created: stream-K (the
    default for batches up to the work-list limit) or the grid form that
    larger batches take (EMA_CREATE_ATTN_GRID forces it)."""
    return request.param


def oracle_attention(w, st, l):
    return oracle.paged_decode_attention(w.q16, w.attn_tables[l], w.lens, st.read_block, w.hkv,
                                         w.D, w.bs, w.cfg.dtype)


@pytest.mark.parametrize("layout", [0, 1])
def test_tiny_config_end_to_end(ema, layout):
    """The tiny workload in full: prefetch the slice half into staging, decode
    one token per sequence, then reclaim every lent block."""
    print(f"tiny layout={layout}", flush=True)
    w = Workload(synth.TINY, slice_layout=layout, staging_slots=1, extra_local=200)
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got = out.cpu().numpy()
        assert np.all(np.isfinite(got))
        ref = oracle_attention(w, st, 0)
        assert rel_err(got, ref) <= TOL
        assert np.array_equal(w.local_view.cpu().numpy(), st.local)     # prefetch bit-exact
        # reclaim everything lent; tables rewritten on the device
        r = ema.slice_reclaim(w.h, 10 ** 9, w.tables_dev.view(-1))
        ro = st.reclaim(10 ** 9, w.tables)
        assert np.array_equal(r["moves"], np.asarray(ro["moves"], np.int64).reshape(-1, 2))
        assert r["victims"] == ro["victims"]
        assert r["lim"] == 0 and ro["lim"] == 0
        assert np.array_equal(w.tables_dev.cpu().numpy(), w.tables)
        torch.cuda.synchronize()
        assert np.array_equal(w.local_view.cpu().numpy(), st.local)
        oracle.check_sd_symmetry(st)
        oracle.check_ownership(st, w.tables)
    finally:
        w.close()


SHAPES = [  # (q_heads, kv_heads, block_size, dtype)
    (8, 8, 16, "f16"), (32, 8, 16, "bf16"), (8, 1, 32, "bf16"), (4, 2, 64, "f16"),
    (16, 1, 16, "bf16"), (2, 2, 256, "f16"), (16, 4, 128, "bf16"),
]
LENS = [0, 1, 15, 16, 17, 255, 256, 257, 511, 513, 1000, 2049]


@pytest.mark.parametrize("hq,hkv,bs,dtype", SHAPES)
def test_attention_shapes_and_ragged_lengths(ema, impl, hq, hkv, bs, dtype):
    print(f"attn {impl} hq={hq} hkv={hkv} bs={bs} {dtype}", flush=True)
    cfg = synth.KVConfig("grid", 1, hq, hkv, 128, dtype, bs, len(LENS), ("uniform", 0, 0), 0.4,
                         31 + bs)
    w = Workload(cfg, lens=LENS, staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got = out.cpu().numpy()
        ref = oracle_attention(w, st, 0)
        assert np.all(got[0] == 0.0)                    # empty sequence
        assert rel_err(got, ref) <= TOL, rel_err(got, ref)
        # elementwise with a floor of 1e-3 of the row's max: the probabilities
        # keep 16 significant bits, so an element's error stays below 2^-16
        # of the row max, i.e. 2^-16 / 1e-3 at the floor
        e = elem_err(got, ref)
        print(f"  normwise {rel_err(got, ref):.2e}, elementwise (floor 1e-3 of the row max) "
              f"{e:.2e}", flush=True)
        assert e <= 2.0 ** -16 / 1e-3, e
    finally:
        w.close()


@pytest.mark.parametrize("hq,hkv,bs,dtype,lens", [
    (8, 1, 32, "bf16", [16384, 12000, 5000, 513, 256, 1]),      # up to 64 splits merged
    (16, 1, 16, "f16", [9000, 4097, 31]),
])
def test_long_sequences_many_splits(ema, impl, hq, hkv, bs, dtype, lens):
    print(f"long {impl} hq={hq} hkv={hkv} bs={bs} {dtype}", flush=True)
    cfg = synth.KVConfig("long", 1, hq, hkv, 128, dtype, bs, len(lens), ("uniform", 0, 0), 0.5,
                         77 + bs)
    w = Workload(cfg, lens=lens, staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        for _ in range(3):                               # counters must reset between calls
            w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got = out.cpu().numpy()
        ref = oracle_attention(w, st, 0)
        assert rel_err(got, ref) <= TOL, rel_err(got, ref)
    finally:
        w.close()


def test_calls_with_different_cuts_on_one_handle(ema, impl):
    """Successive calls on one handle whose stream-K ranges cut different
    (sequence, KV head) pairs into different numbers of pieces (batch and
    lengths change between calls): the reused partial slots and merge records
    must never carry a previous call's pieces into the next."""
    print(f"rearm {impl}", flush=True)
    rng = np.random.default_rng(313)
    lens_a = rng.integers(200, 6000, 24)
    cfg = synth.KVConfig("rearm", 1, 8, 1, 128, "bf16", 32, 24, ("uniform", 0, 0), 0.5, 313)
    w = Workload(cfg, lens=lens_a.tolist(), staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        cases = [(24, lens_a), (24, lens_a // 3), (10, lens_a[:10]), (24, lens_a[::-1] % 700),
                 (24, lens_a)]
        for k, (nb, lens) in enumerate(cases):
            lens = np.minimum(lens, lens_a[:nb]).astype(np.int64)
            out = torch.full((nb, 8, 128), float("nan"), device="cuda")
            ema.paged_decode_attention(w.h, w.q[:nb], w.attn_dev[0][:nb],
                                       torch.as_tensor(lens.astype(np.int32), device="cuda"), out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            ref = oracle.paged_decode_attention(w.q16[:nb], w.attn_tables[0][:nb], lens,
                                                st.read_block, w.hkv, w.D, w.bs, w.cfg.dtype)
            assert rel_err(got, ref) <= TOL, (k, rel_err(got, ref))
        assert ema.slice_device_errors(w.h) == 0
    finally:
        w.close()


def test_empty_batch_and_all_empty_sequences(ema, impl):
    """Degenerate calls: a batch of zero sequences launches nothing and leaves
    the output alone; a batch whose sequences are all empty writes zeros (no
    tile anywhere, so no range cuts a pair); a normal call on the same handle
    afterwards still matches the oracle."""
    print(f"degenerate batches {impl}", flush=True)
    cfg = synth.KVConfig("degenerate", 1, 8, 2, 128, "bf16", 16, 12, ("uniform", 0, 0), 0.5, 77)
    lens = np.random.default_rng(77).integers(1, 900, 12)
    w = Workload(cfg, lens=lens.tolist(), staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = torch.full((12, 8, 128), float("nan"), device="cuda")
        empty = torch.zeros(0, dtype=torch.int32, device="cuda")
        ema.paged_decode_attention(w.h, w.q[:0], w.attn_dev[0][:0], empty, out[:0])
        zeros = torch.zeros(12, dtype=torch.int32, device="cuda")
        out2 = torch.full((12, 8, 128), float("nan"), device="cuda")
        ema.paged_decode_attention(w.h, w.q, w.attn_dev[0], zeros, out2)
        torch.cuda.synchronize()
        assert torch.isnan(out).all()
        assert (out2 == 0).all()
        w.attention(0, out)
        torch.cuda.synchronize()
        ref = oracle.paged_decode_attention(w.q16, w.attn_tables[0], w.lens, st.read_block,
                                            w.hkv, w.D, w.bs, w.cfg.dtype)
        assert rel_err(out.cpu().numpy(), ref) <= TOL
        assert ema.slice_device_errors(w.h) == 0
    finally:
        w.close()


def test_wide_batch_takes_the_long_chunk_path(ema, impl):
    """batch x kv heads >= 256 selects 512-token workgroups; full oracle check."""
    print(f"wide {impl}", flush=True)
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 3000, 32).tolist()
    lens[:4] = [0, 1, 512, 513]
    cfg = synth.KVConfig("wide", 1, 32, 8, 128, "bf16", 16, 32, ("uniform", 0, 0), 0.3, 91)
    w = Workload(cfg, lens=lens, staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got = out.cpu().numpy()
        assert np.all(got[0] == 0.0)
        ref = oracle_attention(w, st, 0)
        assert rel_err(got, ref) <= TOL, rel_err(got, ref)
    finally:
        w.close()


@pytest.mark.parametrize("batch,hi,hkv,hq", [(600, 100, 2, 8), (2100, 40, 1, 4),
                                             (4096, 24, 1, 4), (4200, 16, 1, 2),
                                             (2048, 20, 1, 16), (2100, 20, 1, 16)])
def test_many_short_sequences(ema, impl, batch, hi, hkv, hq):
    """Stream-K ranges then cover several whole sequences each (written
    directly) plus cut ones, and more segments than a range stages up front;
    above 4096 sequences (2048 with 16 query heads per KV head) the grid form
    takes over."""
    print(f"short {impl} batch={batch}", flush=True)
    rng = np.random.default_rng(batch)
    lens = rng.integers(0, hi + 1, batch).tolist()
    cfg = synth.KVConfig("short", 1, hq, hkv, 128, "f16", 16, batch, ("uniform", 0, 0), 0.4, 93)
    w = Workload(cfg, lens=lens, staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got = out.cpu().numpy()
        ref = oracle_attention(w, st, 0)
        assert rel_err(got, ref) <= TOL, rel_err(got, ref)
    finally:
        w.close()


@pytest.mark.parametrize("seed", range(12))
def test_random_configurations(ema, seed):
    """Seeded random shapes, block sizes, dtypes, slice layouts, slice
    fractions and length mixes (with the edge lengths 0, 1, bs and bs + 1
    sprinkled in), through the default matrix-core stream-K path: prefetch
    bit-exact, attention within the bar."""
    rng = np.random.default_rng(1000 + seed)
    hkv = int(rng.choice([1, 2, 4, 8]))
    hq = hkv * int(rng.choice([1, 2, 4, 8, 16]))
    bs = int(rng.choice([16, 32, 64, 128, 256]))
    dtype = str(rng.choice(["f16", "bf16"]))
    layout = int(rng.integers(2))
    batch = int(rng.integers(1, 48))
    lens = rng.integers(0, int(rng.choice([64, 600, 3000])) + 1, batch)
    for v in (0, 1, bs, bs + 1):
        lens[int(rng.integers(batch))] = v
    frac = float(rng.uniform(0.0, 0.9))
    print(f"random seed={seed} hq={hq} hkv={hkv} bs={bs} {dtype} layout={layout} "
          f"batch={batch} frac={frac:.2f}", flush=True)
    cfg = synth.KVConfig("random", 1, hq, hkv, 128, dtype, bs, batch, ("uniform", 0, 0), frac,
                         2000 + seed)
    w = Workload(cfg, lens=lens.tolist(), slice_layout=layout, staging_slots=1)
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        out = w.new_out()
        w.attention(0, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        assert np.array_equal(w.local_view.cpu().numpy(), st.local)
        got = out.cpu().numpy()
        ref = oracle_attention(w, st, 0)
        assert np.all(got[lens == 0] == 0.0)
        assert rel_err(got, ref) <= TOL, rel_err(got, ref)
    finally:
        w.close()


def test_staged_and_all_local_tables_give_identical_bits(ema):
    """Local-remote symmetry as a functional property: the same tokens read
    from staging copies or from other local blocks give the same bits."""
    cfg = synth.LLAMA8B.scaled(layers=1, batch=6)
    w = Workload(cfg, staging_slots=1, extra_local=4000, fill="device")
    try:
        w.prefetch(0)
        out_a = w.new_out()
        w.attention(0, out_a)
        # copy every block of layer 0 to fresh local blocks of the same owner
        tab = w.tables[0]
        valid = tab >= 0
        owners = np.nonzero(valid)[0]
        fresh = ema.slice_alloc_blocks(w.h, ema.POOL_LOCAL, owners)
        src = torch.as_tensor(tab[valid].astype(np.int32), device="cuda")
        dst = torch.as_tensor(fresh, device="cuda")
        ema.slice_migrate(w.h, src, dst)
        tab2 = np.full_like(tab, -1)
        tab2[valid] = fresh
        out_b = w.new_out()
        w.attention(0, out_b, table=torch.as_tensor(tab2.astype(np.int32), device="cuda"))
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        assert torch.equal(out_a, out_b)
    finally:
        w.close()


def test_checked_mode_rejects_slice_ids_in_attention_table(ema):
    cfg = synth.TINY.scaled(batch=2)
    w = Workload(cfg, staging_slots=1, checked=True)
    try:
        out = w.new_out()
        with pytest.raises(ema.EmaError) as e:
            w.attention(0, out, table=w.tables_dev[0])  # canonical table still has slice ids
        assert e.value.code == ema.ERR_INVAL
    finally:
        w.close()


def sampled_parity(ema, w, layer, samples, rng):
    w.prefetch(layer)
    out = w.new_out()
    w.attention(layer, out)
    torch.cuda.synchronize()
    assert ema.slice_device_errors(w.h) == 0
    got = out.cpu().numpy()
    bs = w.bs
    pick = rng.choice(w.B, size=min(samples, w.B), replace=False)
    for b in pick:
        nb = (int(w.lens[b]) + bs - 1) // bs
        ids = w.attn_tables[layer, b, :nb]
        blocks = read_blocks(w.local_view, ids)
        ref = oracle.paged_decode_attention(w.q16[b:b + 1], w.attn_tables[layer, b:b + 1],
                                            w.lens[b:b + 1], blocks.__getitem__, w.hkv, w.D, bs,
                                            w.cfg.dtype)
        assert rel_err(got[b:b + 1], ref) <= TOL, (b, rel_err(got[b:b + 1], ref))
        # the staged copies are the slice blocks, bit for bit
        canon = w.tables[layer, b, :nb]
        sl = canon >= w.n_local
        if sl.any():
            src = read_blocks(w.slice_view, canon[sl] - w.n_local)
            for u, s in zip(ids[sl], canon[sl] - w.n_local):
                if w.slice_layout == 0:
                    assert np.array_equal(blocks[int(u)], src[int(s)])
    return got


def test_llama8b_shaped_layer_sampled(ema):
    print("llama8b layer", flush=True)
    w = Workload(synth.LLAMA8B, layers=2, fill="device")
    try:
        sampled_parity(ema, w, 1, 6, np.random.default_rng(1))
    finally:
        w.close()


def test_ranges_too_long_to_stage(ema):
    """8B-shaped heads with lengths near 8k: every stream-K range holds more
    block ids than the kernel stages in LDS up front, so each segment takes
    the unstaged path (sampled sequences against the oracle)."""
    print("long ranges", flush=True)
    cfg = synth.LLAMA8B.scaled(layers=1, lens=("uniform", 7800, 8192))
    w = Workload(cfg, fill="device")
    try:
        tiles = sum((int(n) + 31) // 32 for n in w.lens) * w.hkv
        assert tiles * 2 // 256 > 512                   # ids per range (block size 16)
        sampled_parity(ema, w, 0, 4, np.random.default_rng(3))
    finally:
        w.close()


def test_70b_tp8_share_layer_sampled(ema):
    print("70b share layer", flush=True)
    w = Workload(synth.L70B_TP8, layers=2, fill="device")
    try:
        assert w.lens.max() > 4096                      # long tails exercise many splits
        sampled_parity(ema, w, 0, 6, np.random.default_rng(2))
    finally:
        w.close()


def _ordered16(bits):
    """16-bit float patterns as integers that step by one per ulp (+0 == -0)."""
    b = np.asarray(bits, np.int64)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


@pytest.mark.parametrize("hq,hkv,bs,dtype,out16", [
    (32, 8, 16, "bf16", "bf16"), (8, 1, 32, "bf16", "bf16"), (8, 8, 16, "f16", "f16"),
    (16, 4, 128, "bf16", "f16"),
])
def test_16bit_output_is_the_fp32_result_rounded_to_nearest_even(ema, impl, hq, hkv, bs, dtype,
                                                                 out16):
    """out_dtype bf16 / fp16: every element is the fp32 output of the same call
    rounded to nearest even (bit for bit), and within one ulp of the float64
    oracle rounded the same way wherever the element is at least 1/64 of its
    row's largest magnitude (below that, the fp32 result's own error, about
    1e-6 of the row maximum, can exceed an fp16 ulp); normwise within 2e-3
    plus the rounding bound everywhere."""
    print(f"out16 {impl} hq={hq} hkv={hkv} bs={bs} {dtype} -> {out16}", flush=True)
    cfg = synth.KVConfig("out16", 1, hq, hkv, 128, dtype, bs, len(LENS), ("uniform", 0, 0), 0.4,
                         55 + bs)
    w = Workload(cfg, lens=LENS, staging_slots=1, attn_grid=impl == "grid")
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        o32 = w.new_out()
        tdt = {"bf16": torch.bfloat16, "f16": torch.float16}[out16]
        o16 = torch.full(o32.shape, float("nan"), dtype=tdt, device="cuda")
        w.attention(0, o32)
        ema.paged_decode_attention(w.h, w.q, w.attn_dev[0], w.lens_dev, o16)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
        got16 = o16.view(torch.int16).cpu().numpy().view(np.uint16)
        got32 = o32.cpu().numpy()
        assert np.array_equal(got16, synth.round_to_16bit(got32, out16))
        ref = oracle_attention(w, st, 0)
        ref16 = synth.round_to_16bit(ref.astype(np.float32), out16)
        rowmax = np.abs(ref).max(axis=-1, keepdims=True)
        big = np.abs(ref) >= rowmax / 64
        ulps = np.abs(_ordered16(got16) - _ordered16(ref16))
        assert ulps[big].max(initial=0) <= 1, ulps[big].max(initial=0)
        as_f = o16.float().cpu().numpy()
        u = 2.0 ** -8 if out16 == "bf16" else 2.0 ** -11
        assert rel_err(as_f, ref) <= TOL + u
        assert np.all(as_f[0] == 0.0)
    finally:
        w.close()

"""The attention entry point that allocates nothing: through the C ABI, its
outputs equal the ordinary entry point's on the same inputs (the same kernels,
so bit for bit) and the float64 oracle within 2e-3, on two calls in a row
whose second is smaller, on two handles of different head shapes sharing the
GPU's fixed workspace, and with a 16-bit output; inputs past its limits are
refused on the host before anything is launched."""
import numpy as np
import pytest
import torch

import oracle
import synth
from harness import Workload, oracle_mirror, rel_err

pytestmark = pytest.mark.gpu
TOL = 2e-3


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


def _ref(w, st, nb, lens):
    return oracle.paged_decode_attention(w.q16[:nb], w.attn_tables[0][:nb], lens, st.read_block,
                                         w.hkv, w.D, w.bs, w.cfg.dtype)


@pytest.mark.parametrize("hq,hkv,bs,dtype,batch", [(32, 8, 16, "bf16", 40),
                                                   (8, 1, 32, "bf16", 48)])
def test_noalloc_equals_the_ordinary_call_on_two_calls_in_a_row(ema, hq, hkv, bs, dtype, batch):
    print(f"noalloc hq={hq} hkv={hkv} bs={bs} batch={batch}", flush=True)
    rng = np.random.default_rng(batch)
    lens = rng.integers(0, 3000, batch)
    lens[:3] = [0, 1, bs + 1]
    cfg = synth.KVConfig("noalloc", 1, hq, hkv, 128, dtype, bs, batch, ("uniform", 0, 0), 0.4,
                         700 + bs)
    w = Workload(cfg, lens=lens.tolist(), staging_slots=1)
    try:
        st = oracle_mirror(w)
        w.prefetch(0)
        st.prefetch(w.pf_src[0], w.pf_dst[0])
        small = max(1, batch // 4)
        for nb, ln in ((batch, lens), (small, lens[:small] // 2)):
            ln = ln.astype(np.int64)
            lens_dev = torch.as_tensor(ln.astype(np.int32), device="cuda")
            want = torch.full((nb, hq, 128), float("nan"), device="cuda")
            got = torch.full((nb, hq, 128), float("nan"), device="cuda")
            ema.paged_decode_attention(w.h, w.q[:nb], w.attn_dev[0][:nb], lens_dev, want)
            ema.paged_decode_attention_noalloc(w.h, w.q[:nb], w.attn_dev[0][:nb], lens_dev, got)
            torch.cuda.synchronize()
            assert torch.equal(got, want), nb
            g = got.cpu().numpy()
            assert rel_err(g, _ref(w, st, nb, ln)) <= TOL
            assert np.all(g[0] == 0.0)
        # a 16-bit output through the fixed workspace
        o16 = torch.empty((batch, hq, 128), dtype=torch.bfloat16, device="cuda")
        o32 = torch.empty((batch, hq, 128), device="cuda")
        ema.paged_decode_attention_noalloc(w.h, w.q, w.attn_dev[0], w.lens_dev, o16)
        ema.paged_decode_attention(w.h, w.q, w.attn_dev[0], w.lens_dev, o32)
        torch.cuda.synchronize()
        assert torch.equal(o16, o32.to(torch.bfloat16))
        assert ema.slice_device_errors(w.h) == 0
    finally:
        w.close()


def test_noalloc_refuses_inputs_beyond_its_limits(ema):
    print("noalloc limits", flush=True)
    cfg = synth.KVConfig("noalloc-lim", 1, 4, 1, 128, "f16", 16, 4097, ("uniform", 0, 0), 0.0,
                         709)
    w = Workload(cfg, lens=[1] * 4097, staging_slots=1)
    try:
        out = torch.zeros((4097, 4, 128), device="cuda")
        with pytest.raises(ema.EmaError) as e:
            ema.paged_decode_attention_noalloc(w.h, w.q, w.attn_dev[0], w.lens_dev, out)
        assert e.value.code == ema.ERR_INVAL
        torch.cuda.synchronize()
        assert torch.count_nonzero(out) == 0          # nothing ran
        # the ordinary call takes the same batch (grid form)
        ema.paged_decode_attention(w.h, w.q, w.attn_dev[0], w.lens_dev, out)
        torch.cuda.synchronize()
        assert ema.slice_device_errors(w.h) == 0
    finally:
        w.close()

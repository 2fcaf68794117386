"""Bursty elastic trace: the lender lends or reclaims 1-25 % of the slice every
step, the borrower's slice fraction follows a random walk in [0, 0.7], and a
full overlapped decode step runs on the result (tests/bursty.py).

Scaled down (4 layers, batch 8, values drawn on the host, both slice layouts,
and a local pool of 0.8 of the cache so that reclaims also preempt):
every step the owners, lent limit, reclaim results and rewritten tables are
compared with an oracle replaying the same operations; every 25 steps both
pools are compared byte for byte (staging blocks aside: the oracle does not
prefetch) and the last layer's attention output against the oracle's float64
attention over the canonical tables.

Full size (the 8B-shaped cache, 32 layers, batch 64, 200 steps): an oracle
without block data replays every allocation, free, lend, migration and
reclaim, and every step the owners, lent limit, reclaim moves, victims and
rewritten tables are compared with it (the device-rewritten tables also
against the host's own application of the plan), plus the ownership
invariants; at the end the content of every logical block of the sequences
never preempted (checksums taken before the trace) and the attention output
of sampled sequences against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from harness import oracle_mirror, owners_mirror, read_blocks, rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


def _local_attention_reader(st):
    return lambda u: oracle.convert_block(st.read_block(u), st.layout_of(int(u)),
                                          oracle.LAYOUT_ATTN, st.kv_heads, st.head_dim,
                                          st.block_size)


@pytest.mark.parametrize("layout,local_frac,mode,group", [(0, 1.0, "serial", 1),
                                                          (0, 1.0, "overlap", 2),
                                                          (1, 1.0, "overlap", 1),
                                                          (1, 0.8, "serial", 2)])
def test_bursty_trace_scaled_matches_oracle(ema, layout, local_frac, mode, group):
    from workloads.bursty import BurstyTrace
    print(f"bursty scaled layout={layout} local_frac={local_frac} mode={mode} group={group}",
          flush=True)
    tr = BurstyTrace(synth.BURSTY, layers=4, batch=8, fill="host", mirror=oracle_mirror,
                     slice_layout=layout, local_frac=local_frac, mode=mode, group=group)
    try:
        st = tr.mirror
        logical0 = oracle.logical_view(st, tr.w.tables)
        kinds = {"reclaim": 0, "lend": 0}
        victims = 0
        for k in range(200):
            rec = tr.step()
            tr.check_invariants()
            kinds["reclaim" if rec["reclaim"] else "lend"] += 1
            if (k + 1) % 25 == 0:
                torch.cuda.synchronize()
                loc = tr.w.local_view.cpu().numpy()
                sli = tr.w.slice_view.cpu().numpy()
                keep = st.own_local != oracle.STAGING
                assert np.array_equal(loc[keep], st.local[keep]), f"step {k}: local pool differs"
                assert np.array_equal(sli, st.slice), f"step {k}: slice pool differs"
                l = tr.L - 1
                ref = oracle.paged_decode_attention(tr.w.q16, tr.w.tables[l], tr.w.lens,
                                                    _local_attention_reader(st), tr.w.hkv,
                                                    tr.w.D, tr.w.bs, tr.cfg.dtype)
                err = rel_err(tr.out.cpu().numpy(), ref)
                assert err <= 2e-3, f"step {k}: attention rel err {err}"
        victims = sum(len(e[4]) for e in tr.log if e[0] == "reclaim")
        assert kinds["reclaim"] > 50 and kinds["lend"] > 50
        assert sum(e[2] for e in tr.log if e[0] == "reclaim") > 0      # blocks moved
        # I4 on the oracle: sequences never preempted kept their content
        logical1 = oracle.logical_view(st, tr.w.tables)
        for key, kv in logical0.items():
            if key[1] in tr.readmitted:
                continue
            assert np.array_equal(kv[0], logical1[key][0]) and \
                np.array_equal(kv[1], logical1[key][1]), f"block {key} changed"
        print(f"reclaims {kinds['reclaim']}, lends {kinds['lend']}, preempted {victims}, "
              f"waiting at the end {len(tr.waiting)}", flush=True)
        if local_frac < 1.0:
            assert victims > 0, "the tight local pool never forced a preemption"
        else:
            assert victims == 0
        assert ema.slice_device_errors(tr.w.h) == 0
    finally:
        tr.close()


def test_bursty_trace_full_size(ema):
    from workloads.bursty import BurstyTrace
    print("bursty full size", flush=True)
    tr = BurstyTrace(synth.BURSTY, fill="device", mirror=owners_mirror)
    try:
        fp0 = tr.fingerprints()
        ms = []
        fr = []
        for k in range(synth.BURSTY.extra["steps"]):
            rec = tr.step()
            tr.check_invariants()
            ms.append(rec["ms"])
            fr.append(rec["slice_frac"])
            if (k + 1) % 50 == 0:
                print(f"step {k + 1}: {rec}", flush=True)
        fp1 = tr.fingerprints()
        keep = np.ones(tr.w.tables.shape, dtype=bool)
        for b in tr.readmitted:
            keep[:, b, :] = False
        keep &= fp0 >= 0
        assert np.array_equal(fp0[keep], fp1[keep]), "block content changed by movement"
        # attention of sampled sequences, last layer, against the oracle
        l = tr.L - 1
        rng = np.random.default_rng(5)
        for b in rng.choice(tr.B, 4, replace=False):
            nb = int((tr.w.lens[b] + tr.w.bs - 1) // tr.w.bs)
            blocks = read_blocks(tr.w.local_view, tr.w.attn_tables[l, b, :nb])
            ref = oracle.paged_decode_attention(tr.w.q16[b:b + 1], tr.w.attn_tables[l, b:b + 1],
                                                tr.w.lens[b:b + 1], blocks.__getitem__,
                                                tr.w.hkv, tr.w.D, tr.w.bs, tr.cfg.dtype)
            err = rel_err(tr.out[b:b + 1].cpu().numpy(), ref)
            assert err <= 2e-3, f"sequence {b}: rel err {err}"
        assert max(fr) - min(fr) > 0.1, "the walk did not move the slice fraction"
        print(f"step ms p50 {np.median(ms):.3f} p90 {np.percentile(ms, 90):.3f} "
              f"max {max(ms):.3f}; slice fraction {min(fr):.2f}..{max(fr):.2f}; "
              f"preempted {len(tr.readmitted)}", flush=True)
        assert ema.slice_device_errors(tr.w.h) == 0
    finally:
        tr.close()

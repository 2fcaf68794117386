"""Large-block copy stress at full pool sizes (tests/stress.py): prefetch of every
slice block in one call, then reclaims of 1, 5, 25 and 100 % of the lent slots
with write-back and a migration back after each.

Checked: sampled blocks bit for bit after every copy (layout-independently for
a token-major slice), the device-rewritten tables against the host's
application of each reclaim plan, each plan (moves, victims, lent limit) and
the rewritten tables against an oracle without block data that replays every
allocation, free, lend, migration and reclaim, and the reclaim counts (the local pool has
room for every borrowed block, so every mover is written back and nothing is
preempted; the slice is full, so every slot of the returned range moves).
"""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ema():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_27040_amd import ema as m
    return m


@pytest.mark.parametrize("bs,layout,n_blocks", [(16, 0, None), (64, 0, None), (256, 0, None),
                                                (16, 1, 65536), (64, 1, 16384), (256, 1, 4096)])
def test_stress_prefetch_and_reclaim_sweep(ema, bs, layout, n_blocks):
    from harness import owners_mirror
    from workloads.stress import StressRun
    print(f"stress bs={bs} layout={layout} n_blocks={n_blocks}", flush=True)
    run = StressRun(bs, n_blocks=n_blocks, slice_layout=layout, mirror=owners_mirror)
    try:
        pf = run.prefetch_all(reps=1)
        assert pf["exact"], "prefetch: sampled blocks differ"
        run.free_staging()
        lim0 = ema.slice_get_info(run.w.h)["lim"]
        sweep = run.reclaim_sweep()
        for r in sweep:
            assert r["tables_ok"], f"{r['frac']}: device tables differ"
            assert r["oracle_ok"], f"{r['frac']}: plan or tables differ from the oracle's"
            assert r["exact"], f"{r['frac']}: sampled written-back blocks differ"
            assert r["moved"] == r["n"] == r["written_back"] and r["victims"] == 0, r
            assert ema.slice_get_info(run.w.h)["lim"] == lim0     # lent back after each
        print(f"prefetch {pf['GBps']:.0f} GB/s; reclaim "
              + ", ".join(f"{r['frac']:.0%} {r['GBps']:.0f} (back {r['migrate_back_GBps']:.0f})"
                          for r in sweep), flush=True)
        assert ema.slice_device_errors(run.w.h) == 0
    finally:
        run.close()
        torch.cuda.empty_cache()

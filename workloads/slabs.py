"""The slab step sweep: the 8B-shaped decode step on a slab-managed slice.

A slice is shared by two users, so over time the borrower's slabs interleave
with slabs the other user holds (section 4.2.1: slab contiguity drops as the
workload changes). The cache here is the 8B-shaped one (32 layers, batch 64,
lengths U[1024, 4096], bf16, block 16): a seeded 30 % of its logical blocks
live at slab positions (all 32 layers each), the rest locally, and slabs are
filled in a seeded random order of logical blocks; before the borrower's
blocks are placed, a seeded half of the slabs in the used range is set aside
(taken by a placeholder and released afterwards, so they are free, not the
borrower's), which leaves the borrower's slabs in runs of about two adjacent
slabs. One step = per layer group, the group's swap (whole borrowed slabs,
into one of two staging images) and the paged decode attention of its layers,
on one stream -- the same step as the block-granular one.

``slab_cache`` builds one configuration; ``run_point`` times steps on it and
reports the swap's runs (count, mean size) and rates.
"""
import numpy as np
import torch

import synth
from paper_2609_27040_amd import ema
from paper_2609_27040_amd.kvcache import TORCH_DT, SlabKVCache
from paper_2609_27040_amd.step import StepRunner
from workloads.synthetic import fill_device


def slab_cache(cfg, slab_blocks, group, layout=ema.SLAB_GROUP_MAJOR, engine=ema.ENGINE_KERNEL,
               gap_frac=0.5, seed=None, fill=True):
    seed = cfg.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    lens = synth.seq_lens(cfg, rng)
    nb = (lens + cfg.block_size - 1) // cfg.block_size
    maxblk = int(nb.max())
    valid = np.arange(maxblk)[None, :] < nb[:, None]
    fb, fj = np.nonzero(valid)
    n_l = len(fb)
    k = int(np.floor(cfg.slice_frac * n_l + 0.5))
    in_slab = np.zeros((len(lens), maxblk), dtype=bool)
    pick = rng.choice(n_l, size=k, replace=False)
    in_slab[fb[pick], fj[pick]] = True
    order = np.stack([fb, fj], axis=1)[rng.permutation(n_l)]
    need = -(-k // slab_blocks)
    gaps = int(round(gap_frac * need / (1.0 - gap_frac))) if gap_frac < 1 else 0
    cache = SlabKVCache(kv_heads=cfg.kv_heads, head_dim=cfg.head_dim, block_size=cfg.block_size,
                        dtype=cfg.dtype, slice_layout=ema.LAYOUT_ATTN, layers=cfg.layers,
                        lens=lens, maxblk=maxblk, in_slab=in_slab, order=order,
                        q_heads=cfg.q_heads, slab_blocks=slab_blocks, group=group,
                        slab_layout=layout, extra_slabs=gaps, engine=engine,
                        gap_slabs=_gap_pattern(rng, need, gaps))
    q16 = synth.q_values(cfg, rng, len(lens))
    cache.q = torch.from_numpy(q16.view(np.int16)).to("cuda").view(TORCH_DT[cfg.dtype])
    cache.q16 = q16
    if fill:
        fill_device(cache, cfg.dtype, seed)
    torch.cuda.synchronize()
    return cache


def _gap_pattern(rng, need, gaps):
    """Which of the first need + gaps slabs are set aside: `gaps` of them,
    seeded, never the first."""
    total = need + gaps
    mark = np.zeros(total, dtype=bool)
    if gaps:
        mark[1 + rng.choice(total - 1, size=gaps, replace=False)] = True
    return mark


def run_point(cache, steps=5, warmup=2):
    """Times `steps` one-stream steps (after `warmup`); every group's swap and
    every layer's attention calls are bracketed by one event pair each, on one
    step, for the per-kind rates."""
    runner = StepRunner(cache, "serial")
    out = cache.new_out()
    for _ in range(warmup):
        runner.run(out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(runner.s1)
    for _ in range(steps):
        runner.run(out)
    e1.record(runner.s1)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    timers = runner.new_timers(layers=[], groups=list(range(len(cache.groups))))
    runner.run(out, timers)
    torch.cuda.synchronize()
    pf_ms = sum(a.elapsed_time(b) for a, b in timers["pf"].values())
    runs = [cache.group_runs(g) for g in range(len(cache.groups))]
    n_runs = sum(len(r[2]) for r in runs)
    moved = sum(int(r[2].sum()) for r in runs)
    pf_bytes = 2 * moved * cache.bb
    useful = int((cache.pos >= 0).sum()) * cache.L
    return {"slab_blocks": cache.S, "group": cache.group,
            "engine": "kernel" if cache.engine == ema.ENGINE_KERNEL else "copy-engines",
            "ms_per_step": ms, "tokens_per_s": cache.B / (ms / 1e3),
            "swap_GBps": pf_bytes / (pf_ms / 1e3) / 1e9, "swap_ms_per_step": pf_ms,
            "runs_per_step": n_runs, "mean_run_KiB": pf_bytes / 2 / max(n_runs, 1) / 1024,
            "moved_blocks": moved, "used_blocks": useful, "borrowed_slabs": cache.m}

#!/usr/bin/env python3
"""Benchmark of the memory-slice hot path on one MI355X.

One step = one decode iteration over every layer of a synthetic paged KV cache
(Llama-3-8B-shaped by default: 32 layers, 32/8 heads, head dim 128, bf16,
block 16, batch 64, lengths U[1024, 4096], 30 % of each layer's blocks in the
slice). Per layer group (``--group`` consecutive layers, 4 by default), one
call prefetches the group's slice-resident blocks into a staging area, and
paged decode attention of each of its layers reads them from there. Two
schedules: ``--mode serial`` (the default) runs prefetches and attention on
one stream; ``--mode overlap`` runs the prefetches on a second stream, ahead of
attention by up to ``--slots`` / ``--group`` − 1 groups. On one GPU the slice
shares the HBM with attention, so both schedules are bound by the same bytes;
the other schedule's steps are timed after the headline ones and reported as
``alt_mode``. ``--append`` also stores a new token per sequence before each
layer's attention and writes the modified staged blocks back to the slice
after it. Every event costs device time, so each step times one layer group
(rotating): one event pair around its prefetch and one around its
consecutive attention calls (with ``--append``, two layers' calls one by one).

After the timed steps, untimed by the step clock:
  * symmetry: attention over every layer through the staged tables versus
    through all-local tables holding the same tokens (each slice-resident block
    migrated to a fresh local block), interleaved A B A B; the outputs of one
    layer are compared bit for bit;
  * cpu_baseline: the oracle on a bounded sample, on this host's cores (before
    reclaim, which rewrites blocks the sample reads);
  * reclaim: the lender takes part of the slice back a few times (compaction /
    write-back / preemption plus the device table rewrite), timed on the device
    behind a blocking copy so that host planning is not counted.

Prints one JSON line. ``value`` is decode tokens/s of the whole step
(batch / step time; attention only, no projections or MLP). The roofline
object is for the attention entry point (its kernels' algorithmic HBM bytes
over their mean duration per call, from HIP events on the attention stream
during the timed steps); its ``traffic`` comes from the committed counter summary of the
same workload and is null when the kernel sources no longer match it.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# Sources whose code runs in one attention call; a counter record is valid for
# the digest of exactly these files.
ATTN_SOURCES = ("paper_2609_27040_amd/csrc/paged_attention_mfma.hip",
                "paper_2609_27040_amd/csrc/kernels.h")
COPY_SOURCES = ("paper_2609_27040_amd/csrc/block_copy.hip",
                "paper_2609_27040_amd/csrc/kernels.h")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b-kv",
                    choices=["llama3-8b-kv", "llama-70b-tp8-share", "bursty-8b", "stress",
                             "run-sweep", "slab-sweep"])
    ap.add_argument("--mode", default="serial", choices=["serial", "overlap"],
                    help="serial: prefetches and attention on one stream; overlap: prefetches "
                         "on a second stream, ahead of attention")
    ap.add_argument("--no-alt-mode", action="store_true",
                    help="skip the steps in the other mode that are reported alongside")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the graph-captured steps that are reported alongside")
    ap.add_argument("--group", type=int, default=4,
                    help="layers per layer group: one prefetch call per group")
    ap.add_argument("--slots", type=int, default=None,
                    help="staging slots, a multiple of the group size (default: two groups)")
    ap.add_argument("--timed-layers", type=int, default=2,
                    help="with --append: layers per step whose attention calls get their own "
                         "timing events (rotating); without it each step times one layer "
                         "group's consecutive attention calls between one event pair")
    ap.add_argument("--append", action="store_true",
                    help="each layer also appends the new token's K/V and writes the modified "
                         "staged blocks back to the slice")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--reclaim-reps", type=int, default=4)
    ap.add_argument("--symmetry-reps", type=int, default=6,
                    help="A/B pairs of the staged vs all-local attention passes (0: skip)")
    ap.add_argument("--no-legs", action="store_true",
                    help="skip the other workloads' compact legs reported beside the headline "
                         "(70B TP-8 share step, stress prefetch, token-major slice, bursty "
                         "trace, slab sweep, copy ceilings)")
    ap.add_argument("--legs", default="c3,stress,nhd,bursty,slabs,ceiling",
                    help="which compact legs to run (comma-separated)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def attention_bytes(w, layer=0):
    """Algorithmic HBM bytes of one attention call: the K and V of every cached
    token, q in and fp32 out, the block-table entries in use and the lengths."""
    e = 2
    toks = int(w.lens.sum())
    nblk = int(((w.lens + w.bs - 1) // w.bs).sum())
    hq = w.cfg.q_heads
    return (toks * 2 * w.hkv * w.D * e + w.B * hq * w.D * (e + 4) + 4 * nblk + 4 * w.B)


def sources_digest(sources=ATTN_SOURCES):
    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_record(name, sources):
    """The traffic record of a committed counter summary, or None when there is
    none or it was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-record:"):
                rec = json.loads(line.split(":", 1)[1])
                if rec.get("sources") == sources_digest(sources):
                    return rec
    return None


def counter_traffic(workload):
    """HBM bytes per attention call from the committed counter summary."""
    return counter_record(f"paged_attention_{workload}_counters.md", ATTN_SOURCES)


def pct(a, q):
    return float(np.percentile(np.asarray(a), q))


def step_timers(runner, args, k):
    """Timing events for step k. Without append, one layer group per step
    (rotating over the groups) gets one event pair around its consecutive
    attention calls and one around its prefetch: each event packet costs a
    few microseconds of device time, which a pair per call would add to
    every timed call. With append, a call's append sits between the
    attention calls, so a few layers per step are timed call by call."""
    w = runner.w
    if runner.kv_new is None:
        u = k % len(w.groups)
        return runner.new_timers(layers=[], groups=[u], attn_groups=[u])
    nt = max(1, min(w.L, args.timed_layers))
    return runner.new_timers([(nt * k + i) % w.L for i in range(nt)])


def attention_samples(timers, w):
    """Per-call attention times (ms) of every timed unit (a call, or a group's
    run of calls divided by its length) and the number of calls covered."""
    per_call, calls = [], 0
    for tm in timers:
        for e0, e1 in tm["at"].values():
            per_call.append(e0.elapsed_time(e1))
            calls += 1
        for u, (e0, e1) in tm["atg"].items():
            n = len(w.groups[u])
            per_call.append(e0.elapsed_time(e1) / n)
            calls += n
    return np.array(per_call), calls


def _host_blocks(w, ids):
    """Host copies (uint8 [n][block bytes]) of unified blocks of a workload."""
    import torch
    ids = np.asarray(ids, dtype=np.int64)
    out = np.empty((len(ids), w.bb), dtype=np.uint8)
    loc = ids < w.n_local
    for mask, view, off in ((loc, w.local_view, 0), (~loc, w.slice_view, w.n_local)):
        if mask.any():
            sel = torch.from_numpy(ids[mask] - off).to(view.device)
            out[mask] = view[sel].cpu().numpy()
    return out


def _oracle_layer(w, layer, min_s):
    """The oracle's float64 attention of every sequence of one layer over the
    canonical table, then that layer's prefetch (one block at a time, slice
    layout -> local layout), each repeated until it has run min_s seconds.
    Returns (seconds per attention pass, seconds per prefetch pass, passes)."""
    import oracle
    tab = w.tables[layer]
    used = np.unique(tab[tab >= 0])
    data = _host_blocks(w, used)
    row = {int(u): i for i, u in enumerate(used)}
    slice_layout = w.slice_layout

    def read(u):
        blk = data[row[int(u)]]
        if int(u) >= w.n_local and slice_layout != oracle.LAYOUT_ATTN:
            return oracle.convert_block(blk, slice_layout, oracle.LAYOUT_ATTN, w.hkv, w.D, w.bs)
        return blk
    n_a, t0 = 0, time.perf_counter()
    while n_a == 0 or time.perf_counter() - t0 < min_s:
        oracle.paged_decode_attention(w.q16, tab, w.lens, read, w.hkv, w.D, w.bs, w.cfg.dtype)
        n_a += 1
    t_a = (time.perf_counter() - t0) / n_a
    src = np.asarray(w.pf_src[layer], dtype=np.int64)
    sdata = data[[row[int(u)] for u in src]] if len(src) else np.empty((0, w.bb), np.uint8)
    dst = np.empty_like(sdata)
    n_p, t0 = 0, time.perf_counter()
    while n_p == 0 or time.perf_counter() - t0 < min_s / 4:
        for i in range(len(sdata)):
            dst[i] = oracle.convert_block(sdata[i], slice_layout, oracle.LAYOUT_ATTN, w.hkv,
                                          w.D, w.bs)
        n_p += 1
    t_p = (time.perf_counter() - t0) / n_p
    return t_a, t_p, len(src), n_a


def cpu_baseline(w, seconds):
    """The oracle timed on this host's cores (one thread) on the parts the
    baseline plan names: the tiny config in full; one layer of the 8B-shaped
    cache, its attention over every sequence plus that layer's prefetch; one
    layer of the 70B TP-8 share; 4 GiB of single-block copies of the stress
    pools' shape (64 KiB blocks). `value` is the 8B layer extrapolated to a
    whole decode step (every layer's prefetch and attention): batch / (layers
    x (attention + prefetch of one layer))."""
    import torch
    import synth
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    from workloads.synthetic import Workload

    per = max(0.5, seconds / 4)
    res = {"unit": "tokens/s", "cores": 1, "kind": "oracle",
           "host_cores_available": len(os.sched_getaffinity(0)),
           "blas_threads_default": [p.get("num_threads") for p in threadpool_info()],
           "blas_threads_used": 1}
    with threadpool_limits(1):
        t_a, t_p, n_pf, reps = _oracle_layer(w, 0, per)
        tok_s = w.B / (w.L * (t_a + t_p))
        res["value"] = tok_s
        res[f"{w.cfg.name}_layer"] = {
            "attention_s": t_a, "prefetch_s": t_p, "prefetch_blocks": n_pf,
            "attention_GBps": attention_bytes(w) / t_a / 1e9,
            "prefetch_GBps": 2 * n_pf * w.bb / t_p / 1e9 if t_p > 0 else None,
            "tokens_per_s_extrapolated": tok_s, "attention_passes": reps}
        others = [(c, k) for c, k in ((synth.TINY, "tiny_full"),
                                      (synth.LLAMA8B, "llama3-8b-kv_layer"),
                                      (synth.L70B_TP8, "llama-70b-tp8-share_layer"))
                  if c.name != w.cfg.name]
        for cfg, key in others:
            v = Workload(cfg, layers=1, fill="device", staging_slots=1)
            try:
                ta, tp, n, reps = _oracle_layer(v, 0, per if cfg is not synth.TINY else 0.5)
                res[key] = {"attention_s": ta, "prefetch_s": tp, "prefetch_blocks": n,
                            "attention_GBps": attention_bytes(v) / ta / 1e9,
                            "tokens_per_s_layer": v.B / (ta + tp), "attention_passes": reps,
                            "layers_in_config": cfg.layers}
            finally:
                v.close()
                torch.cuda.empty_cache()
        # 4 GiB of 64 KiB blocks (the stress pools at block size 16), one
        # oracle block copy at a time
        bb = 64 << 10
        n_blk = (4 << 30) // bb
        src = np.empty((n_blk, bb), dtype=np.uint8)
        src[:] = np.arange(bb, dtype=np.uint64).astype(np.uint8)
        dst = np.empty_like(src)
        t0 = time.perf_counter()
        for i in range(n_blk):
            dst[i] = oracle.convert_block(src[i], oracle.LAYOUT_ATTN, oracle.LAYOUT_ATTN, 8,
                                          128, 16)
        t_c = time.perf_counter() - t0
        del src, dst
        res["stress_copy_4GiB"] = {"blocks": n_blk, "seconds": t_c,
                                   "GBps": 2 * n_blk * bb / t_c / 1e9}
    res["sample"] = (
        f"one thread: {w.cfg.name} layer 0 (all {w.B} sequences, float64 attention, "
        f"{reps} passes) plus its prefetch of {n_pf} blocks, extrapolated to {w.L} layers; "
        "layer 0 of the other full-size shape; the tiny config in full; 4 GiB of single-block "
        f"copies ({n_blk} x 64 KiB)")
    return res


def cpu_copy_baseline(rows, layout, hkv, D, bs, seconds):
    """The oracle's block copy (slice layout -> local layout) on this host,
    one thread, over host copies of sampled slice blocks (rows: uint8
    [n][block bytes]) for about `seconds`; GB/s of read + write."""
    import oracle
    from threadpoolctl import threadpool_limits

    dst = np.empty_like(rows)
    n_cp = 0
    with threadpool_limits(1):
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            i = n_cp % len(rows)
            dst[i] = oracle.convert_block(rows[i], layout, oracle.LAYOUT_ATTN, hkv, D, bs)
            n_cp += 1
        t = time.perf_counter() - t0
    return {"value": 2 * n_cp * rows.shape[1] / t / 1e9, "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": (f"{n_cp} single-block copies of {rows.shape[1] >> 10} KiB by the oracle "
                       f"({t:.1f} s, one thread), cycling over {len(rows)} slice blocks read "
                       f"back from the device"),
            "host_cores_available": len(os.sched_getaffinity(0))}


def symmetry(w, out, s, reps, ema, torch):
    """Staged versus all-local attention tables over the same tokens.

    Every slice-resident block of every layer is migrated to a fresh local
    block (allocated in a seeded random order, so ids are as scattered as the
    canonical local ones). Pass A runs attention over all layers through the
    staged tables, pass B through the all-local tables; passes alternate.
    Layer 0 is prefetched first and its two outputs must match bit for bit.
    The timed passes read whatever the staging slots hold (the same bytes and
    access pattern as a step; only layer 0's values are compared). The fresh
    blocks are freed again at the end."""
    L = w.L
    sl = w.tables >= w.n_local
    src = w.tables[sl].astype(np.int32)
    owners = np.nonzero(sl)[1]
    perm = np.random.default_rng(w.cfg.seed + 1).permutation(len(src))
    fresh = ema.slice_alloc_blocks(w.h, ema.POOL_LOCAL, owners[perm])
    dst = np.empty(len(src), dtype=np.int32)
    dst[perm] = fresh
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a, dtype=np.int32), device="cuda")
    ema.slice_migrate(w.h, i32(src), i32(dst), stream=s)
    local_tabs = w.tables.copy()
    local_tabs[sl] = dst
    local_dev = i32(local_tabs)
    # bitwise check on layer 0
    w.prefetch(0, stream=s)
    out_b = w.new_out()
    w.attention(0, out, stream=s)
    w.attention(0, out_b, table=local_dev[0], stream=s)
    torch.cuda.synchronize()
    identical = bool(torch.equal(out, out_b))

    def run(tabs):
        for l in range(L):
            w.attention(l, out, table=tabs[l], stream=s)

    run(w.attn_dev)
    run(local_dev)
    ms = {"staged": [], "local": []}
    for _ in range(reps):
        for kind, tabs in (("staged", w.attn_dev), ("local", local_dev)):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            run(tabs)
            e1.record(s)
            e1.synchronize()
            ms[kind].append(e0.elapsed_time(e1))
    torch.cuda.synchronize()
    ema.slice_free_blocks(w.h, fresh)
    med = {k: float(np.median(v)) for k, v in ms.items()}
    return {"outputs_identical": identical,
            "staged_ms_per_step": med["staged"], "local_ms_per_step": med["local"],
            "staged_p10_p90": [pct(ms["staged"], 10), pct(ms["staged"], 90)],
            "local_p10_p90": [pct(ms["local"], 10), pct(ms["local"], 90)],
            "ratio": med["staged"] / med["local"],
            "attention_us_per_layer": med["staged"] * 1e3 / L,
            "reps": reps, "moved_blocks": int(len(src))}


def alt_mode_steps(w, out, mode, args, attn_b):
    """The same steps in the other schedule, timed the same way (reported beside
    the headline, not part of it)."""
    import torch
    from paper_2609_27040_amd.step import StepRunner
    log(f"{mode} steps for comparison")
    runner = StepRunner(w, mode)
    for _ in range(args.warmup):
        runner.run(out)
    timers = [step_timers(runner, args, k) for k in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        runner.run(out, timers[k])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    at_us = float(attention_samples(timers, w)[0].mean()) * 1e3
    return {"mode": mode, "ms_per_step": ms_step, "tokens_per_s": w.B / (ms_step / 1e3),
            "attention_mean_us": at_us, "attention_GBps": attn_b / at_us / 1e3}


def graph_steps(w, out, runner, args):
    """The one-stream step captured once as a HIP graph and replayed (reported
    beside the headline: timing events cannot be captured here, so the
    roofline stays with the eager steps). The replay's output must equal an
    eager step's bit for bit."""
    import torch
    from paper_2609_27040_amd.step import capture_step
    log("graph-captured steps for comparison")
    runner.run(out)
    torch.cuda.synchronize()
    ref = out.clone()
    g = capture_step(runner, out)
    with torch.cuda.stream(runner.s1):           # a graph replays on the current stream
        for _ in range(args.warmup):
            g.replay()
    torch.cuda.synchronize()
    same = bool(torch.equal(out, ref))
    t0 = time.perf_counter()
    with torch.cuda.stream(runner.s1):
        for _ in range(args.steps):
            g.replay()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    same = same and bool(torch.equal(out, ref))
    del g
    return {"ms_per_step": ms_step, "tokens_per_s": w.B / (ms_step / 1e3),
            "replay_matches_eager": same}


def calib_lib():
    """The calibration kernels (libema_calib.so, built with the library)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2609_27040_amd", "lib", "libema_calib.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build with __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    for f in (lib.ema_calib_read, lib.ema_calib_copy):
        f.restype = ctypes.c_int
    lib.ema_calib_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                   ctypes.c_void_p]
    lib.ema_calib_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_void_p]
    return lib


def hbm_context(torch, gib=4, reps=5):
    """What plain streaming gives on this GPU in the same run, as context for
    the fractions of 8 TB/s: the calibration kernels' contiguous read and
    copy (16-byte non-temporal accesses, whole chunks in flight; a copy counts
    read + write) and torch's device-to-device copy."""
    n = (gib << 30) // 2
    x = torch.randn(n, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    y = torch.empty_like(x)
    res = {}
    lib = calib_lib()
    sink = torch.empty(2 * n // 4096, device="cuda", dtype=torch.int32)

    def calib(rc):
        if rc != 0:
            raise RuntimeError(f"calibration launch failed ({rc})")
    stream = lambda: torch.cuda.current_stream().cuda_stream
    for name, fn, nbytes in (
            ("calib_read_GBps",
             lambda: calib(lib.ema_calib_read(x.data_ptr(), 2 * n, sink.data_ptr(), stream())),
             2 * n),
            ("calib_copy_GBps",
             lambda: calib(lib.ema_calib_copy(x.data_ptr(), y.data_ptr(), 2 * n, stream())),
             4 * n),
            ("torch_copy_GBps", lambda: y.copy_(x), 4 * n)):
        fn()
        torch.cuda.synchronize()
        # `reps` launches back to back between one event pair: the host's
        # submission gap before the first launch is spread over all of them
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        e1.synchronize()
        res[name] = reps * nbytes / (e0.elapsed_time(e1) / 1e3) / 1e9
    del x, y, sink
    torch.cuda.empty_cache()
    return res


def reclaim_phase(w, s, reps, ema, torch):
    """The lender takes 5 % of its lent blocks back, ``reps`` times. Each call is
    queued behind a device copy long enough to outlast the call's host planning,
    so the events bracket only device work: upload of the plan, block copies,
    table rewrite. ``host_plan_ms`` is the call's host time; ``device_only``
    says whether the copy was indeed still running when the call returned."""
    from paper_2609_27040_amd.step import BlockedTimer
    timer = BlockedTimer()
    res = []
    for _ in range(reps):
        lim = ema.slice_get_info(w.h)["lim"]
        n = max(1, lim // 20)
        r, ms, hms, covered = timer.time(
            s, lambda: ema.slice_reclaim(w.h, n, w.tables_dev.view(-1), stream=s),
            host_ms=2.0 + 50e-6 * n)
        nb = 2 * r["moved"] * w.bb + 8 * w.tables_dev.numel()
        res.append({"n": n, "moved": r["moved"], "written_back": r["written_back"],
                    "victims": len(r["victims"]), "ms": ms, "host_plan_ms": hms,
                    "device_only": covered, "GBps": nb / (ms / 1e3) / 1e9})
    timer.close()
    return res


def bursty_run(mode="serial", group=4, steps=None):
    """The bursty elastic trace: every step the lender lends or reclaims 1-25 %
    of the slice, the borrower's slice fraction takes a random-walk step and
    blocks migrate, then one decode step runs; returns the per-step latency
    distribution (the invariants are checked after every step)."""
    import torch
    import synth
    from workloads.bursty import BurstyTrace
    from paper_2609_27040_amd import ema

    torch.cuda.set_device(0)
    cfg = synth.BURSTY
    log("setting up bursty-8b")
    tr = BurstyTrace(cfg, fill="device", mode=mode, group=group)
    w = tr.w
    steps = cfg.extra["steps"] if steps is None else steps
    recs, gbps = [], []
    try:
        for k in range(steps):
            rec = tr.step()
            tr.check_invariants()
            pf = sum(2 * len(s) * w.bb for s in w.pf_src)
            toks = int(w.lens.sum())
            attn = w.L * (toks * 2 * w.hkv * w.D * 2)
            gbps.append((attn + pf) / (rec["ms"] / 1e3) / 1e9)
            recs.append(rec)
            if (k + 1) % 50 == 0:
                log(f"step {k + 1}: {rec['ms']:.3f} ms, slice fraction {rec['slice_frac']:.2f}")
        errs = ema.slice_device_errors(w.h)
        if errs:
            raise RuntimeError(f"kernels skipped {errs} invalid ids")
        ms = np.array([r["ms"] for r in recs])
        fr = np.array([r["slice_frac"] for r in recs])
        res = {
            "value": w.B / (float(np.median(ms)) / 1e3), "unit": "tokens/s",
            "steps": steps, "ms_per_step": float(np.median(ms)),
            "config": {"workload": cfg.name, "layers": w.L, "batch": w.B,
                       "q_heads": cfg.q_heads, "kv_heads": cfg.kv_heads,
                       "head_dim": cfg.head_dim, "block_size": cfg.block_size,
                       "lens": list(cfg.lens), "frac_max": cfg.extra["frac_max"],
                       "step_frac": list(cfg.extra["step_frac"]), "mode": mode,
                       "layer_group": group},
            "step_ms": {"p10": pct(ms, 10), "p50": pct(ms, 50), "p90": pct(ms, 90),
                        "max": float(ms.max())},
            "step_GBps": {"p10": pct(gbps, 10), "p50": pct(gbps, 50), "p90": pct(gbps, 90)},
            "slice_frac": {"min": float(fr.min()), "max": float(fr.max())},
            "lender": {"reclaims": sum(1 for e in tr.log if e[0] == "reclaim"),
                       "lends": sum(1 for e in tr.log if e[0] == "lend"),
                       "moved_blocks": int(sum(e[2] for e in tr.log if e[0] == "reclaim")),
                       "preempted": int(sum(len(e[4]) for e in tr.log if e[0] == "reclaim"))},
            "migrated_blocks": int(sum(e[2] for e in tr.log if e[0] == "migrate")),
        }
    finally:
        tr.close()
        torch.cuda.empty_cache()
    return res


def bursty_main(args):
    """The bursty trace on its own: one JSON line."""
    r = bursty_run(args.mode, args.group)
    res = {"metric": "prefetch/reclaim GB/s + paged decode tokens/s, % of HBM roofline, 1 GPU",
           "value": r["value"], "unit": "tokens/s", "n_gpus": 1, "steps": r["steps"],
           "warmup": 0, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic"}
    res.update({k: v for k, v in r.items() if k not in res})
    print(json.dumps(res))


def bursty_leg(steps=100):
    """A compact bursty trace beside the headline; its roofline is the whole
    step's HBM rate (attention plus prefetch bytes over the step time, median
    over steps that also reclaim, lend and migrate)."""
    log(f"leg: bursty trace, {steps} steps")
    r = bursty_run(steps=steps)
    r["roofline"] = roofline_obj(r["step_GBps"]["p50"], None,
                                 "decode step (prefetch + paged decode attention) under "
                                 "reclaims, lends and migrations")
    return r


def stress_main(args):
    """Large-block copy stress: per block size, prefetch of every slice block in
    one call, then reclaims of 1, 5, 25 and 100 % of the lent slots (write-back
    to local), each followed by a migration back; prints one JSON line."""
    import torch
    import synth
    from workloads.stress import StressRun, stress_blocks

    torch.cuda.set_device(0)
    cfg = synth.STRESS
    out = {}
    cpu = None
    for bs in cfg.extra["block_sizes"]:
        log(f"stress block size {bs}: {stress_blocks(cfg, bs)} blocks")
        run = StressRun(bs)
        try:
            pf = run.prefetch_all()
            if cpu is None and not args.no_cpu_baseline:
                log("cpu baseline (oracle block copies)")
                ids = run.w.pf_src[0][run._sample(len(run.w.pf_src[0]))]
                cpu = cpu_copy_baseline(run._rows(ids), run.layout, run.w.hkv, run.w.D, bs,
                                        args.cpu_seconds / 2)
                cpu["block_size"] = bs
            run.free_staging()
            rc = run.reclaim_sweep()
        finally:
            run.close()
        torch.cuda.empty_cache()
        out[str(bs)] = {"blocks": run.N, "block_bytes": run.w.bb, "prefetch": pf,
                        "reclaim": rc}
        log(f"bs {bs}: prefetch {pf['GBps']:.0f} GB/s, reclaim "
            + ", ".join(f"{r['frac']:.0%} {r['GBps']:.0f}" for r in rc))
    bad = [k for k, v in out.items() if not v["prefetch"]["exact"]
           or not all(r["exact"] and r["tables_ok"] for r in v["reclaim"])]
    if bad:
        raise RuntimeError(f"sampled copies differ at block sizes {bad}")
    best_bs = max(out, key=lambda k: out[k]["prefetch"]["GBps"])
    best = out[best_bs]["prefetch"]["GBps"]
    rec = counter_record("block_copy_stress_counters.md", COPY_SOURCES)
    traffic = None
    if rec is not None and best_bs in rec.get("per_block_size", {}):
        traffic = rec["per_block_size"][best_bs]["bytes_per_launch"]
    res = {"metric": "prefetch/reclaim GB/s + paged decode tokens/s, % of HBM roofline, 1 GPU",
           "value": best, "unit": "GB/s", "n_gpus": 1, "steps": 1, "warmup": 0,
           "ms_per_step": None, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f16", "data": "synthetic",
           "config": {"workload": "stress", "kv_heads": cfg.kv_heads,
                      "head_dim": cfg.head_dim, "slice_frac": cfg.slice_frac,
                      "block_sizes": list(cfg.extra["block_sizes"])},
           "roofline": {"bound": "hbm", "achieved": best, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                        "frac": best / HBM_PEAK_GBPS, "traffic": traffic,
                        "kernel": f"block_copy_same_kernel (prefetch of every slice block, "
                                  f"block size {best_bs})"},
           "sweep": out}
    if rec is not None:
        res["roofline"]["traffic_source"] = rec.get("note", "counter summary")
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res))


def run_sweep_main(args):
    """Copy efficiency against transfer size: prefetch of every slice block of a
    block-size-16 pool (8 GiB, 60 % slice) as contiguous runs of 1 to 400
    blocks, by the gather kernel and by the copy engines; one JSON line."""
    import torch
    from workloads.stress import run_sweep

    torch.cuda.set_device(0)
    log("slab sweep")
    rows = run_sweep()
    if not all(r["exact"] for r in rows):
        raise RuntimeError("sampled copies differ")
    best = max(r["kernel"]["GBps"] for r in rows)
    res = {"metric": "prefetch/reclaim GB/s + paged decode tokens/s, % of HBM roofline, 1 GPU",
           "value": best, "unit": "GB/s", "n_gpus": 1, "steps": 1, "warmup": 0,
           "ms_per_step": None, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f16", "data": "synthetic",
           "config": {"workload": "run-sweep", "block_size": 16, "kv_heads": 8,
                      "blocks": 1 << 17, "slice_frac": 0.6},
           "sweep": rows}
    for r in rows:
        log(f"run {r['run_blocks']:4d} blocks: kernel {r['kernel']['GBps']:.0f} GB/s, "
            f"copy engines {r['dma']['GBps']:.0f} GB/s (end to end {r['dma']['wall_GBps']:.0f})")
    print(json.dumps(res))


def measure_steps(w, runner, steps, warmup, timed_layers=2):
    """Times `steps` steps after `warmup`: whole-step wall time between two
    device synchronisations, attention per call and prefetch per group from
    event pairs (one layer group per step, rotating)."""
    import torch
    from types import SimpleNamespace
    a = SimpleNamespace(timed_layers=timed_layers)
    out = w.new_out()
    for _ in range(warmup):
        runner.run(out)
    torch.cuda.synchronize()
    timers = [step_timers(runner, a, k) for k in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        runner.run(out, timers[k])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    at_ms, at_calls = attention_samples(timers, w)
    pf_b = [2 * len(src) * w.bb for src in w.pf_src_grp]
    pf_ms = np.array([e0.elapsed_time(e1) for tm in timers for e0, e1 in tm["pf"].values()])
    pf_timed_b = float(sum(pf_b[k] for tm in timers for k in tm["pf"]))
    attn_b = attention_bytes(w)
    at_mean_s = float(at_ms.mean()) / 1e3
    attn_gbps = attn_b / at_mean_s / 1e9
    pf_gbps = pf_timed_b / (pf_ms.sum() / 1e3) / 1e9 if len(pf_ms) else 0.0
    step_bytes = attn_b * w.L + float(np.sum(pf_b))
    # Time of the step's attention and prefetch calls, each as timed on its
    # own, over the step's wall time: near 1, the device streams HBM for the
    # whole step and a second stream has no idle time left to fill.
    busy_s = at_mean_s * w.L + (float(np.sum(pf_b)) / (pf_gbps * 1e9) if pf_gbps else 0.0)
    return out, {
        "ms_per_step": ms_step, "tokens_per_s": w.B / (ms_step / 1e3),
        "attention": {"bytes_per_launch": attn_b, "timed_calls": int(at_calls),
                      "mean_us": at_mean_s * 1e6,
                      "tokens_per_s_attention_only": w.B / (w.L * at_mean_s),
                      "p10_us": pct(at_ms, 10) * 1e3, "p90_us": pct(at_ms, 90) * 1e3,
                      "GBps": attn_gbps, "frac": attn_gbps / HBM_PEAK_GBPS},
        "prefetch": {"bytes_per_step": float(np.sum(pf_b)),
                     "mean_us": float(pf_ms.mean()) * 1e3 if len(pf_ms) else 0.0,
                     "GBps": pf_gbps, "frac": pf_gbps / HBM_PEAK_GBPS},
        "step": {"bytes": step_bytes, "GBps": step_bytes / (ms_step / 1e3) / 1e9,
                 "frac": step_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBPS,
                 "kernel_time_share": busy_s / (ms_step / 1e3)}}


def roofline_obj(achieved, traffic_rec, kernel, key="bytes_per_call"):
    r = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
         "frac": achieved / HBM_PEAK_GBPS, "traffic": None, "kernel": kernel}
    if traffic_rec is not None:
        r["traffic"] = traffic_rec.get(key)
        r["traffic_source"] = traffic_rec.get("note", "counter summary")
    return r


def step_leg(cfg, steps, warmup, group=4, slice_layout=0, counters=None, sources=ATTN_SOURCES,
             roof="attention"):
    """One workload's one-stream step (compact: no other schedule, graph,
    symmetry or reclaim phase). The roofline is the attention entry point's,
    or with roof="prefetch" the group prefetch copy's."""
    import torch
    from paper_2609_27040_amd import ema
    from paper_2609_27040_amd.step import StepRunner
    from workloads.synthetic import Workload
    log(f"leg: {cfg.name}, slice layout {slice_layout}")
    w = Workload(cfg, fill="device", staging_slots=2 * group, group=group,
                 slice_layout=slice_layout)
    try:
        runner = StepRunner(w, "serial")
        _, rec = measure_steps(w, runner, steps, warmup)
        if ema.slice_device_errors(w.h):
            raise RuntimeError(f"{cfg.name}: kernels skipped invalid ids")
    finally:
        w.close()
        torch.cuda.empty_cache()
    log(f"  {rec['ms_per_step']:.3f} ms/step, attention {rec['attention']['mean_us']:.1f} us "
        f"({rec['attention']['GBps']:.0f} GB/s), prefetch {rec['prefetch']['GBps']:.0f} GB/s")
    crec = counter_record(counters, sources) if counters else None
    if roof == "attention":
        rec["roofline"] = roofline_obj(rec["attention"]["GBps"], crec,
                                       "paged_decode_attention (attn_mfma_streamk + "
                                       "attn_combine_streamk)")
    else:
        rec["roofline"] = roofline_obj(rec["prefetch"]["GBps"], crec,
                                       "block_copy_kernel (group prefetch, token-major slice "
                                       "re-laid into the local layout)", key="bytes_per_launch")
    rec["config"] = {"workload": cfg.name, "layers": w.L, "batch": w.B, "q_heads": cfg.q_heads,
                     "kv_heads": cfg.kv_heads, "block_size": cfg.block_size,
                     "lens": list(cfg.lens), "slice_frac": cfg.slice_frac, "layer_group": group,
                     "slice_layout": "token-major" if slice_layout else "local"}
    rec["steps"], rec["warmup"] = steps, warmup
    return rec


def stress_leg(block_sizes=(16, 64, 256)):
    """Prefetch of every slice block of the large-block stress pools (one
    call per block size) and one reclaim of 5 % of the lent slots with
    write-back, sampled blocks compared bit for bit."""
    import torch
    from workloads.stress import StressRun
    out = {}
    for bs in block_sizes:
        log(f"leg: stress block size {bs}")
        run = StressRun(bs)
        try:
            pf = run.prefetch_all(reps=3)
            run.free_staging()
            rc = run.reclaim_sweep(fractions=(0.05,))[0]
        finally:
            run.close()
            torch.cuda.empty_cache()
        if not (pf["exact"] and rc["exact"] and rc["tables_ok"]):
            raise RuntimeError(f"stress block size {bs}: sampled blocks or tables differ")
        log(f"  prefetch {pf['GBps']:.0f} GB/s, reclaim of 5 % {rc['GBps']:.0f} GB/s")
        out[str(bs)] = {"blocks": run.N, "block_bytes": run.w.bb, "prefetch_GBps": pf["GBps"],
                        "prefetch_ms": pf["ms"], "reclaim_5pct_GBps": rc["GBps"],
                        "reclaim_5pct_ms": rc["ms"], "reclaim_moved": rc["moved"]}
    best = max(out, key=lambda k: out[k]["prefetch_GBps"])
    crec = counter_record("block_copy_stress_counters.md", COPY_SOURCES)
    traffic = None
    if crec is not None and best in crec.get("per_block_size", {}):
        traffic = crec["per_block_size"][best]["bytes_per_launch"]
    roof = roofline_obj(out[best]["prefetch_GBps"], None,
                        f"block_copy_same_kernel (prefetch of every slice block, block size {best})")
    roof["traffic"] = traffic
    if crec is not None:
        roof["traffic_source"] = crec.get("note", "counter summary")
    return {"roofline": roof, "per_block_size": out}


def slab_leg(points, steps=3, warmup=1):
    """The 8B-shaped step on a slab-managed slice with interleaved free slabs
    (workloads.slabs), per (slab size, layer group, engine[, placement])."""
    import torch
    import synth
    from paper_2609_27040_amd import ema
    from workloads.slabs import run_point, slab_cache
    rows = []
    for pt in points:
        S, k, eng = pt[:3]
        layout = pt[3] if len(pt) > 3 else ema.SLAB_GROUP_MAJOR
        log(f"leg: slab step S={S} group={k} engine={eng} placement={layout}")
        c = slab_cache(synth.LLAMA8B, S, k, layout=layout, engine=eng)
        try:
            rows.append(run_point(c, steps=steps, warmup=warmup))
            rows[-1]["placement"] = ("layer-major", "slab-major", "layer-group-major")[layout]
            if ema.slice_device_errors(c.h):
                raise RuntimeError("slab step: kernels skipped invalid ids")
        finally:
            c.close()
            torch.cuda.empty_cache()
        r = rows[-1]
        log(f"  {r['ms_per_step']:.2f} ms/step, swap {r['swap_GBps']:.0f} GB/s, "
            f"{r['runs_per_step']} runs of {r['mean_run_KiB']:.0f} KiB")
    return rows


def slab_sweep_main(args):
    """The slab step sweep on its own (one JSON line): slabs of 1, 10 and 100
    blocks x groups of 1, 2 and 4 layers with the gather kernel, the copy
    engines at groups of 4, and the three placements at 10-block slabs and
    groups of 4 with both engines."""
    import torch
    from paper_2609_27040_amd import ema
    torch.cuda.set_device(0)
    K, D = ema.ENGINE_KERNEL, ema.ENGINE_DMA
    pts = [(S, k, K) for S in (1, 10, 100) for k in (1, 2, 4)]
    pts += [(S, 4, D) for S in (1, 10, 100)]
    pts += [(10, 4, e, lay) for lay in (ema.SLAB_LAYER_MAJOR, ema.SLAB_SLAB_MAJOR)
            for e in (K, D)]
    rows = slab_leg(pts, steps=max(1, args.steps // 4), warmup=max(1, args.warmup))
    best = max(rows, key=lambda r: r["tokens_per_s"])
    res = {"metric": "prefetch/reclaim GB/s + paged decode tokens/s, % of HBM roofline, 1 GPU",
           "value": best["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
           "steps": max(1, args.steps // 4), "warmup": max(1, args.warmup),
           "ms_per_step": best["ms_per_step"], "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "slab-sweep", "cache": "llama3-8b-kv", "slice_frac": 0.3,
                      "best": {k: best[k] for k in ("slab_blocks", "group", "engine",
                                                    "placement")}},
           "sweep": rows}
    print(json.dumps(res))


def ceiling_leg():
    """What this GPU's HBM gives the library's own copy on long contiguous
    runs (the kernel engine of the run prefetch, 400-block runs of 64 KiB),
    beside the calibration kernels' plain read and plain copy and torch's
    copy, in the same process."""
    import torch
    from workloads.stress import run_sweep
    log("leg: copy ceilings")
    rows = run_sweep(run_blocks=(400,), engines=("kernel",))
    res = {"library_copy_contiguous_GBps": rows[0]["kernel"]["GBps"],
           "library_copy_run_blocks": 400}
    res.update(hbm_context(torch))
    log("  " + ", ".join(f"{k} {v:.0f}" for k, v in res.items()))
    return res


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build runs on one GPU; the slice stands in for the peer's share "
              "on the same device, so there is no multi-GPU configuration (use --gpus 1).",
              file=sys.stderr)
        sys.exit(2)

    if args.workload == "bursty-8b":
        bursty_main(args)
        return
    if args.workload == "stress":
        stress_main(args)
        return
    if args.workload == "run-sweep":
        run_sweep_main(args)
        return
    if args.workload == "slab-sweep":
        slab_sweep_main(args)
        return
    import torch
    import synth
    from paper_2609_27040_amd.step import StepRunner
    from workloads.synthetic import Workload
    from paper_2609_27040_amd import ema

    torch.cuda.set_device(0)
    cfg = synth.CONFIGS[args.workload]
    log(f"setting up {cfg.name}")
    probe = synth.placement(cfg, synth.seq_lens(cfg, np.random.default_rng(cfg.seed)),
                            np.random.default_rng(cfg.seed))
    extra = len(probe.slice_order) if args.symmetry_reps > 0 else 0
    del probe
    g = max(1, args.group)
    slots = 2 * g if args.slots is None else args.slots
    w = Workload(cfg, fill="device", extra_local=extra, staging_slots=slots, group=g)
    L, B = w.L, w.B
    log(f"{L} layers, batch {B}, {w.n_local} local + {w.slice_view.shape[0]} slice blocks")
    runner = StepRunner(w, args.mode, append=args.append)
    s1 = runner.s1
    out = w.new_out()
    attn_b = attention_bytes(w)

    log(f"warmup {args.warmup}, timed {args.steps} steps ({args.mode})")
    out, core = measure_steps(w, runner, args.steps, args.warmup, timed_layers=args.timed_layers)
    ms_step = core["ms_per_step"]
    errs = ema.slice_device_errors(w.h)
    if errs:
        raise RuntimeError(f"kernels skipped {errs} invalid ids")
    attn_gbps = core["attention"]["GBps"]
    log(f"{ms_step:.3f} ms/step, attention {core['attention']['mean_us']:.1f} us/layer")

    alt = None
    if not args.no_alt_mode:
        alt = alt_mode_steps(w, out, "overlap" if args.mode == "serial" else "serial",
                             args, attn_b)
    graph = None
    if args.mode == "serial" and not args.no_graph:
        graph = graph_steps(w, out, runner, args)
        if not graph["replay_matches_eager"]:
            raise RuntimeError("graph replay differs from the eager step")

    traffic = None
    rec = counter_traffic(cfg.name)
    if rec is not None:
        traffic = rec["bytes_per_call"]

    res = {
        "metric": "prefetch/reclaim GB/s + paged decode tokens/s, % of HBM roofline, 1 GPU",
        "value": B / (ms_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "layers": L, "batch": B, "q_heads": cfg.q_heads,
                   "kv_heads": cfg.kv_heads, "head_dim": cfg.head_dim,
                   "block_size": cfg.block_size, "lens": list(cfg.lens),
                   "slice_frac": cfg.slice_frac, "mode": args.mode, "append": args.append,
                   "layer_group": w.group, "staging_slots": w.staging_slots},
        "roofline": {"bound": "hbm", "achieved": attn_gbps, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": attn_gbps / HBM_PEAK_GBPS, "traffic": traffic,
                     "kernel": "paged_decode_attention (attn_mfma_streamk + attn_combine_streamk)"},
        "attention": dict(core["attention"], timing=(
            "one event pair per call" if args.append else
            f"one event pair around each timed group's {w.group} consecutive calls")),
        "prefetch": core["prefetch"],
        "step": core["step"],
    }
    if rec is not None:
        res["roofline"]["traffic_source"] = rec.get("note", "counter summary")
    if alt is not None:
        res["alt_mode"] = alt
    if graph is not None:
        res["graph"] = graph

    if args.symmetry_reps > 0:
        log("symmetry: staged vs all-local tables")
        sym = symmetry(w, out, s1, args.symmetry_reps, ema, torch)
        sym["step_vs_all_local_attention"] = ms_step / sym["local_ms_per_step"]
        res["symmetry"] = sym
        iso = attn_b / (sym["attention_us_per_layer"] / 1e6) / 1e9
        res["attention"]["isolated_GBps"] = iso
        res["attention"]["isolated_frac"] = iso / HBM_PEAK_GBPS
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    if args.reclaim_reps > 0:
        log("reclaim")
        res["reclaim"] = reclaim_phase(w, s1, args.reclaim_reps, ema, torch)
    errs = ema.slice_device_errors(w.h)
    if errs:
        raise RuntimeError(f"kernels skipped {errs} invalid ids")
    w.close()
    del w, runner, out
    torch.cuda.empty_cache()
    if not args.no_legs and cfg.name == "llama3-8b-kv":
        res["legs"] = run_legs(args)
    elif not args.no_cpu_baseline:
        res["hbm_context"] = hbm_context(torch)
    print(json.dumps(res))


def run_legs(args):
    """The other workloads, compact, beside the headline (each with its own
    roofline object): the 70B TP-8 share's step, the stress pools' prefetch and
    reclaim, the 8B step with a token-major slice (the relayout copy), a
    100-step bursty trace, the slab step sweep, and the copy ceilings of this
    GPU."""
    import synth
    want = set(args.legs.split(","))
    legs = {}
    t0 = time.perf_counter()
    if "c3" in want:
        legs["llama-70b-tp8-share"] = step_leg(
            synth.L70B_TP8, steps=10, warmup=2,
            counters="paged_attention_llama-70b-tp8-share_counters.md")
    if "stress" in want:
        legs["stress"] = stress_leg()
    if "nhd" in want:
        legs["llama3-8b-kv-token-major-slice"] = step_leg(
            synth.LLAMA8B, steps=10, warmup=2, slice_layout=1,
            counters="block_copy_token_major_prefetch_counters.md", sources=COPY_SOURCES,
            roof="prefetch")
    if "bursty" in want:
        legs["bursty-8b"] = bursty_leg()
    if "slabs" in want:
        from paper_2609_27040_amd import ema
        pts = [(S, k, ema.ENGINE_KERNEL) for S in (1, 10, 100) for k in (1, 2, 4)]
        pts += [(S, 4, ema.ENGINE_DMA) for S in (1, 10, 100)]
        legs["slab-sweep"] = slab_leg(pts)
    if "ceiling" in want:
        legs["copy-ceilings"] = ceiling_leg()
    legs["seconds"] = time.perf_counter() - t0
    return legs


if __name__ == "__main__":
    main()

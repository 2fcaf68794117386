#!/usr/bin/env python3
"""Benchmark of the memory-slice hot path on one MI355X.

One step = one decode iteration over every layer of a synthetic paged KV cache
(Llama-3-8B-shaped by default: 32 layers, 32/8 heads, head dim 128, bf16,
block 16, batch 64, lengths U[1024, 4096], 30 % of each layer's blocks in the
slice). Per layer: the slice-resident blocks of layer l+1 are prefetched into a
double-buffered staging area on one stream while paged decode attention of
layer l runs on another (``--mode serial`` runs both on one stream: copy, then
attention). After the timed steps the lender reclaims part of the slice a few
times (compaction / write-back / preemption plus the device table rewrite).

Prints one JSON line. ``value`` is decode tokens/s of the whole step
(batch / step time; attention only, no projections or MLP). The roofline
object is for the attention entry point (its kernels' algorithmic HBM bytes
over their mean duration, from HIP events on the attention stream).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
for p in (ROOT, os.path.join(ROOT, "tests")):
    if p not in sys.path:
        sys.path.insert(0, p)

HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama3-8b-kv",
                    choices=["llama3-8b-kv", "llama-70b-tp8-share"])
    ap.add_argument("--mode", default="overlap", choices=["overlap", "serial"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--reclaim-reps", type=int, default=4)
    return ap.parse_args()


def attention_bytes(w, layer=0):
    """Algorithmic HBM bytes of one attention call: the K and V of every cached
    token, q in and fp32 out, the block-table entries in use and the lengths."""
    e = 2
    toks = int(w.lens.sum())
    nblk = int(((w.lens + w.bs - 1) // w.bs).sum())
    hq = w.cfg.q_heads
    return (toks * 2 * w.hkv * w.D * e + w.B * hq * w.D * (e + 4) + 4 * nblk + 4 * w.B)


def cpu_baseline(w, seconds):
    """The oracle timed on this host's cores on a bounded sample: float64
    attention of layer 0 for whole sequences, and block prefetch copies."""
    import oracle
    from harness import read_blocks
    from threadpoolctl import threadpool_limits

    rng = np.random.default_rng(0)
    order = rng.permutation(w.B)[:16]
    cache = {}
    for b in order:
        nb = (int(w.lens[b]) + w.bs - 1) // w.bs
        cache[int(b)] = read_blocks(w.local_view, w.attn_tables[0, b, :nb])
    with threadpool_limits(1):
        n_seq = 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            b = int(order[n_seq % len(order)])
            oracle.paged_decode_attention(w.q16[b:b + 1], w.attn_tables[0, b:b + 1],
                                          w.lens[b:b + 1], cache[b].__getitem__, w.hkv, w.D,
                                          w.bs, w.cfg.dtype)
            n_seq += 1
        t_attn = time.perf_counter() - t0
        # prefetch copies (slice layout -> local layout), one block at a time
        src = list(cache[int(order[0])].values())
        dst = np.empty((len(src), w.bb), dtype=np.uint8)
        n_cp = 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds / 4:
            i = n_cp % len(src)
            dst[i] = oracle.convert_block(src[i], w.slice_layout, oracle.LAYOUT_ATTN, w.hkv, w.D,
                                          w.bs)
            n_cp += 1
        t_cp = time.perf_counter() - t0
    tok_s = n_seq / t_attn / w.L      # one decode token needs every layer
    return {"value": tok_s, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": (f"float64 attention of {n_seq} whole sequences of layer 0 "
                       f"({t_attn:.1f} s, one thread), scaled to {w.L} layers per token; "
                       f"{n_cp} block prefetch copies ({t_cp:.1f} s)"),
            "prefetch_GBps": 2 * n_cp * w.bb / t_cp / 1e9,
            "host_cores_available": len(os.sched_getaffinity(0))}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build runs on one GPU; the slice stands in for the peer's share "
              "on the same device, so there is no multi-GPU configuration (use --gpus 1).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from harness import Workload
    from paper_2609_27040_amd import ema

    torch.cuda.set_device(0)
    cfg = synth.CONFIGS[args.workload]
    log(f"setting up {cfg.name}")
    w = Workload(cfg, fill="device")
    L, B = w.L, w.B
    log(f"{L} layers, batch {B}, {w.n_local} local + {w.slice_view.shape[0]} slice blocks")
    s1 = torch.cuda.Stream()
    s2 = torch.cuda.Stream() if args.mode == "overlap" else s1
    out = w.new_out()
    attn_b = attention_bytes(w)
    pf_b = [2 * len(w.pf_src[l]) * w.bb for l in range(L)]

    ev_pf = [torch.cuda.Event() for _ in range(L)]
    ev_at = [torch.cuda.Event() for _ in range(L)]

    def step(timers):
        for l in range(L):
            if l == 0:
                # staging slots 0/1 were last read by the previous step's last layers
                s2.wait_event(ev_at[L - 1])
                if L >= 2:
                    s2.wait_event(ev_at[L - 2])
                if timers:
                    timers["pf"][0][0].record(s2)
                w.prefetch(0, stream=s2)
                if timers:
                    timers["pf"][0][1].record(s2)
                ev_pf[0].record(s2)
            if l + 1 < L:
                if l >= 1:
                    s2.wait_event(ev_at[l - 1])   # slot (l+1) % 2 was read by layer l-1
                if timers:
                    timers["pf"][l + 1][0].record(s2)
                w.prefetch(l + 1, stream=s2)
                if timers:
                    timers["pf"][l + 1][1].record(s2)
                ev_pf[l + 1].record(s2)
            s1.wait_event(ev_pf[l])
            if timers:
                timers["at"][l][0].record(s1)
            w.attention(l, out, stream=s1)
            if timers:
                timers["at"][l][1].record(s1)
            ev_at[l].record(s1)

    def new_timers():
        mk = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        return {"pf": [mk() for _ in range(L)], "at": [mk() for _ in range(L)]}

    log(f"warmup {args.warmup}, timed {args.steps} steps ({args.mode})")
    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    timers = [new_timers() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(timers[k])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    errs = ema.slice_device_errors(w.h)
    if errs:
        raise RuntimeError(f"kernels skipped {errs} invalid ids")

    at_ms = np.array([[tm["at"][l][0].elapsed_time(tm["at"][l][1]) for l in range(L)]
                      for tm in timers])
    pf_ms = np.array([[tm["pf"][l][0].elapsed_time(tm["pf"][l][1]) for l in range(L)]
                      for tm in timers])
    at_mean_s = float(at_ms.mean()) / 1e3
    attn_gbps = attn_b / at_mean_s / 1e9
    pf_gbps = float(np.sum(pf_b) * args.steps / (pf_ms.sum() / 1e3) / 1e9)
    step_bytes = attn_b * L + float(np.sum(pf_b))

    log(f"{ms_step:.3f} ms/step; reclaim")
    # ---- reclaim: the lender takes part of the slice back, a few times ----------------
    reclaim = []
    for _ in range(args.reclaim_reps):
        lim = ema.slice_get_info(w.h)["lim"]
        n = max(1, lim // 20)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(s1)
        c0 = time.perf_counter()
        r = ema.slice_reclaim(w.h, n, w.tables_dev.view(-1), stream=s1)
        c1 = time.perf_counter()
        e1.record(s1)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        nbytes = 2 * r["moved"] * w.bb + 8 * w.tables_dev.numel()
        reclaim.append({"n": n, "moved": r["moved"], "written_back": r["written_back"],
                        "victims": len(r["victims"]), "ms": ms, "host_plan_ms": (c1 - c0) * 1e3,
                        "GBps": nbytes / (ms / 1e3) / 1e9})

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
                   "slice_frac": cfg.slice_frac, "mode": args.mode},
        "roofline": {"bound": "hbm", "achieved": attn_gbps, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": attn_gbps / HBM_PEAK_GBPS, "traffic": None},
        "attention": {"bytes_per_launch": attn_b, "mean_us": at_mean_s * 1e6,
                      "GBps": attn_gbps, "frac": attn_gbps / HBM_PEAK_GBPS},
        "prefetch": {"bytes_per_step": float(np.sum(pf_b)), "mean_us": float(pf_ms.mean()) * 1e3,
                     "GBps": pf_gbps, "frac": pf_gbps / HBM_PEAK_GBPS},
        "step": {"bytes": step_bytes, "GBps": step_bytes / (ms_step / 1e3) / 1e9,
                 "frac": step_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBPS},
        "reclaim": reclaim,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    w.close()
    print(json.dumps(res))


if __name__ == "__main__":
    main()

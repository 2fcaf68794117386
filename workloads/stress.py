"""Large-block copy stress: pure prefetch and reclaim throughput at large pools.

One layer of a cache with 8 KV heads, fp16, block size bs; N blocks in all,
N = min(2^20, 100 GiB / block bytes), spread over 1024 sequences, 60 % of them
slice-resident at random (seeded placement and allocation order). The local
pool holds the other 40 % plus a staging block for every slice block.

  prefetch   every slice block into its staging block, in one call;
  reclaim    after the staging blocks are freed, the lender takes back
             1 %, 5 %, 25 % and 100 % of its lent slots in turn; each reclaim
             writes the borrowed blocks of the returned range back to free
             local blocks and rewrites the tables; the slots are then lent
             again and the moved blocks migrated back to the slice, so every
             reclaim starts from the same placement.

Every copy is timed on the device (the reclaim behind a blocking copy, so its
host planning is excluded) and sampled blocks are compared bit for bit
(layout-independently when the slice pool is token-major).
"""
import numpy as np
import torch

import synth
from paper_2609_27040_amd.step import BlockedTimer
from workloads.synthetic import Workload
from paper_2609_27040_amd import ema

FRACTIONS = (0.01, 0.05, 0.25, 1.0)


def stress_blocks(cfg, bs):
    bb = 2 * bs * cfg.kv_heads * cfg.head_dim * 2
    return int(min(cfg.extra["max_blocks"], cfg.extra["max_kv_bytes"] // bb))


class StressRun:
    def __init__(self, bs, n_blocks=None, seqs=1024, slice_layout=ema.LAYOUT_ATTN,
                 cfg=synth.STRESS, samples=256, mirror=None):
        N = stress_blocks(cfg, bs) if n_blocks is None else int(n_blocks)
        per_seq = max(1, N // seqs)
        tok = per_seq * bs
        c = cfg.scaled(block_size=bs, batch=seqs, lens=("uniform", tok, tok))
        self.w = w = Workload(c, layers=1, staging_slots=1, fill="pattern",
                              slice_layout=slice_layout)
        self.cfg, self.bs, self.N = c, bs, per_seq * seqs
        self.layout = slice_layout
        self.rng = np.random.default_rng(c.seed + bs)
        self.samples = samples
        self.s = torch.cuda.Stream()
        self.timer = BlockedTimer()
        self.ns_per_mover = 50.0        # host planning estimate, refined as reclaims run
        # an observer (the tests pass an oracle without block data) replaying
        # every allocation, free, lend, migration and reclaim
        self.mirror = mirror(w) if mirror is not None else None
        if self.mirror is not None:
            self.mtables = w.tables.copy()

    # ---- helpers ---------------------------------------------------------------------
    def _rows(self, ids):
        """Host bytes of unified blocks (local or slice), in table order."""
        w = self.w
        ids = np.asarray(ids, np.int64)
        out = np.empty((len(ids), w.bb), dtype=np.uint8)
        loc = ids < w.n_local
        if loc.any():
            out[loc] = w.local_view[torch.as_tensor(ids[loc], device="cuda")].cpu().numpy()
        if (~loc).any():
            out[~loc] = w.slice_view[torch.as_tensor(ids[~loc] - w.n_local,
                                                     device="cuda")].cpu().numpy()
        return out

    def _logical(self, rows, ids):
        """Layout-independent K, V of each row (local blocks are ATTN)."""
        w = self.w
        res = []
        for r, u in zip(rows, ids):
            lay = synth.LAYOUT_ATTN if u < w.n_local else self.layout
            res.append(synth.unpack_block(r, lay, w.hkv, w.bs, w.D))
        return res

    def _same_content(self, src_rows, src_ids, dst_rows, dst_ids):
        if self.layout == synth.LAYOUT_ATTN:
            return np.array_equal(src_rows, dst_rows)
        a = self._logical(src_rows, src_ids)
        b = self._logical(dst_rows, dst_ids)
        return all(np.array_equal(x[0], y[0]) and np.array_equal(x[1], y[1])
                   for x, y in zip(a, b))

    def _sample(self, n):
        return self.rng.choice(n, size=min(n, self.samples), replace=False)

    # ---- phases ----------------------------------------------------------------------
    def prefetch_all(self, reps=3):
        w = self.w
        src, dst = w.pf_src[0], w.pf_dst[0]
        n = len(src)
        pick = self._sample(n)
        before = self._rows(src[pick])
        ms = []
        for _ in range(reps):
            _, t, _, _ = self.timer.time(self.s, lambda: w.prefetch(0, stream=self.s))
            ms.append(t)
        after = self._rows(dst[pick])
        ok = self._same_content(before, src[pick], after, dst[pick])
        t = float(np.median(ms))
        return {"blocks": n, "ms": t, "GBps": 2 * n * w.bb / (t / 1e3) / 1e9, "exact": ok}

    def free_staging(self):
        ema.slice_free_blocks(self.w.h, self.w.staging.ravel())
        if self.mirror is not None:
            self.mirror.free_blocks(self.w.staging.ravel())

    def reclaim_sweep(self, fractions=FRACTIONS):
        w = self.w
        res = []
        tables = w.tables
        for p in fractions:
            lim0 = ema.slice_get_info(w.h)["lim"]
            n = int(round(p * lim0))
            cut = lim0 - n
            # content of sampled borrowed blocks in the returned range, before
            rng_ids = tables[(tables >= w.n_local + cut) & (tables < w.n_local + lim0)]
            pick = rng_ids[self._sample(len(rng_ids))] if len(rng_ids) else rng_ids
            before = self._rows(pick)
            torch.cuda.synchronize()
            r, ms, host_ms, covered = self.timer.time(
                self.s, lambda: ema.slice_reclaim(w.h, n, w.tables_dev.view(-1), stream=self.s),
                host_ms=2.0 + n * self.ns_per_mover * 1e-6)
            self.ns_per_mover = max(self.ns_per_mover, host_ms * 1e6 / max(1, n))
            mv = np.asarray(r["moves"], dtype=np.int64).reshape(-1, 2)
            remap = np.arange(w.n_local + w.slice_view.shape[0], dtype=np.int64)
            remap[mv[:, 0]] = mv[:, 1]
            valid = tables >= 0
            tables[valid] = remap[tables[valid]]
            for v in r["victims"]:
                tables[:, v, :] = -1
            dev = w.tables_dev.cpu().numpy().reshape(tables.shape)
            tables_ok = np.array_equal(dev, tables.astype(np.int32))
            oracle_ok = None
            if self.mirror is not None:
                mr = self.mirror.reclaim(n, self.mtables)
                oracle_ok = (np.array_equal(mv, np.asarray(mr["moves"], np.int64).reshape(-1, 2))
                             and list(r["victims"]) == list(mr["victims"])
                             and r["lim"] == mr["lim"] and r["written_back"] == mr["written_back"]
                             and np.array_equal(tables, self.mtables))
            after_ids = remap[pick]
            exact = self._same_content(before, pick, self._rows(after_ids), after_ids)
            nbytes = 2 * r["moved"] * w.bb + 8 * w.tables_dev.numel()
            rec = {"frac": p, "n": n, "moved": r["moved"], "written_back": r["written_back"],
                   "victims": len(r["victims"]), "ms": ms, "host_plan_ms": host_ms,
                   "device_only": covered, "GBps": nbytes / (ms / 1e3) / 1e9,
                   "tables_ok": tables_ok, "exact": exact, "oracle_ok": oracle_ok}
            # lend the slots again and move the blocks back into the slice
            ema.slice_lend(w.h, n)
            if self.mirror is not None:
                self.mirror.lend(n)
            if len(mv):
                pos = np.argwhere(np.isin(tables, mv[:, 1]))
                cur = tables[pos[:, 0], pos[:, 1], pos[:, 2]]
                back = ema.slice_alloc_blocks(w.h, ema.POOL_SLICE, pos[:, 1]).astype(np.int64)
                if self.mirror is not None:
                    mback = self.mirror.alloc_blocks(ema.POOL_SLICE, pos[:, 1])
                    rec["oracle_ok"] = rec["oracle_ok"] and np.array_equal(back, mback)
                    self.mirror.migrate(cur, back)
                    self.mirror.free_blocks(cur)
                    self.mtables[pos[:, 0], pos[:, 1], pos[:, 2]] = back
                src_t = torch.as_tensor(cur.astype(np.int32), device="cuda")
                dst_t = torch.as_tensor(back.astype(np.int32), device="cuda")
                _, mms, _, _ = self.timer.time(
                    self.s, lambda: ema.slice_migrate(w.h, src_t, dst_t, stream=self.s))
                ema.slice_free_blocks(w.h, cur)
                tables[pos[:, 0], pos[:, 1], pos[:, 2]] = back
                w.tables_dev.copy_(torch.from_numpy(tables.astype(np.int32)))
                rec["migrate_back_GBps"] = 2 * len(cur) * w.bb / (mms / 1e3) / 1e9
            res.append(rec)
        return res

    def close(self):
        self.timer.close()
        self.w.close()


RUN_BLOCKS = (1, 4, 16, 64, 100, 200, 400)


def run_sweep(bs=16, n_blocks=1 << 17, run_blocks=RUN_BLOCKS, reps=3,
              engines=("kernel", "dma")):
    """Prefetch of every slice block as contiguous runs of R blocks (the slab x
    layer-group chunks of a layer-group-major slice), by the gather kernel and
    by the copy engines. Slice slots are taken in order (every slot is owned:
    the slice is exactly full) into the contiguous staging area. Returns, per
    R, device GB/s (events behind a blocking copy) and end-to-end GB/s (host
    submission included: one transfer per run for the copy engines)."""
    import time
    run = StressRun(bs, n_blocks=n_blocks)
    w = run.w
    try:
        n = len(w.pf_src[0])
        s0, d0 = w.n_local, int(w.staging[0, 0])
        out = []
        for R in run_blocks:
            k = n // R
            src_first = s0 + R * np.arange(k)
            dst_first = d0 + R * np.arange(k)
            runs = np.full(k, R)
            nbytes = 2 * k * R * w.bb
            rec = {"run_blocks": R, "run_bytes": R * w.bb, "runs": int(k)}
            for name, eng in (("kernel", ema.ENGINE_KERNEL), ("dma", ema.ENGINE_DMA)):
                if name not in engines:
                    continue
                call = lambda: ema.slice_prefetch_runs(w.h, src_first, dst_first, runs, eng,
                                                       stream=run.s)
                dev, wall = [], []
                for _ in range(reps):
                    _, ms, host_ms, covered = run.timer.time(run.s, call, host_ms=2.0 + k * 0.02)
                    dev.append(ms)
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    call()
                    torch.cuda.synchronize()
                    wall.append((time.perf_counter() - t0) * 1e3)
                rec[name] = {"GBps": nbytes / (np.median(dev) / 1e3) / 1e9,
                             "wall_GBps": nbytes / (np.median(wall) / 1e3) / 1e9,
                             "device_only": bool(covered)}
            pick = run._sample(k * R)
            ok = np.array_equal(run._rows(s0 + pick), run._rows(d0 + pick))
            rec["exact"] = bool(ok)
            out.append(rec)
        return out
    finally:
        run.close()

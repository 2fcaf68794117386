"""Bursty elastic trace over a paged KV cache, driven through the library.

Every step, in this order:
  1. the lender acts: with probability 1/2 it reclaims round(q * lim) slots,
     else it lends round(q * (n_slice - lim)) more, q ~ U[0.01, 0.25];
     sequences preempted by a reclaim are admitted again at once, all their
     blocks freshly allocated in the local pool with new values;
  2. the borrower's target slice fraction takes a step of a random walk,
     f <- clip(f + U(-0.1, 0.1), 0, fmax), and blocks migrate local <-> slice
     (allocate, copy, free) toward round(f * T), as far as free space allows;
  3. the staging lists and attention tables are rebuilt and one full decode
     step runs (prefetch per layer group, attention per layer, in the chosen
     schedule), timed with events.

Pools: the slice holds ceil((fmax + slack) * T) slots, the local pool
local_frac * T blocks plus two layer groups of staging (T = blocks of all
layers).
With local_frac = 1 the borrower can hold everything locally and a reclaim
never preempts; below 1, a large reclaim at a low slice fraction finds too
little room for write-back and preempts sequences.

After each step the caller can check the library's owners and tables: the
device-rewritten tables against the host's own application of the returned
moves and victims, the ownership invariants, and (with ``mirror``, a callable
that makes an observer of the workload -- the tests pass an oracle) a replay of
every operation compared after each.
"""
import math

import numpy as np
import torch

import synth
from paper_2609_27040_amd.kvcache import TORCH_DT
from paper_2609_27040_amd.step import StepRunner
from workloads.synthetic import Workload
from paper_2609_27040_amd import ema


def _round_half_up(x):
    return int(math.floor(x + 0.5))


class BurstyTrace:
    def __init__(self, cfg, layers=None, batch=None, seed=None, fill="device", mirror=None,
                 fmax=None, slack=0.02, f0=None, lens=None, slice_layout=ema.LAYOUT_ATTN,
                 local_frac=1.0, mode="serial", group=1):
        cfg = cfg if batch is None else cfg.scaled(batch=batch)
        fmax = cfg.extra.get("frac_max", 0.7) if fmax is None else fmax
        L = cfg.layers if layers is None else layers
        seed = cfg.seed if seed is None else seed
        f0 = cfg.slice_frac if f0 is None else f0
        lens_ = synth.seq_lens(cfg, np.random.default_rng(seed)) if lens is None else \
            np.asarray(lens, np.int64)
        n_l = int(((lens_ + cfg.block_size - 1) // cfg.block_size).sum())
        T = L * n_l
        slice0 = L * _round_half_up(f0 * n_l)
        n_slice = int(math.ceil((fmax + slack) * T))
        n_local = int(math.floor(local_frac * T))    # plus the staging area
        if n_local < T - slice0:
            raise ValueError("local pool smaller than the initial local share")
        self.w = w = Workload(cfg, layers=L, seed=seed, fill=fill, frac=f0, lens=lens,
                              stage_n=n_l, extra_local=n_local - (T - slice0),
                              extra_slice=n_slice - slice0,
                              slice_layout=slice_layout, group=group,
                              staging_slots=2 * group)
        self.cfg, self.L, self.B, self.T, self.fmax = cfg, L, w.B, T, fmax
        self.n_slice = n_slice
        self.rng = np.random.default_rng(seed + 1000)
        self.f = f0
        self.step_no = 0
        self.log = []
        self.runner = StepRunner(w, mode)
        self.out = w.new_out()
        self.fill = fill
        self.readmitted = set()
        self.waiting = set()
        self.len0 = w.lens.copy()
        # an observer (the tests pass an oracle) replaying every operation
        self.mirror = mirror(w) if mirror is not None else None
        if self.mirror is not None:
            self.mtables = w.tables.copy()

    # ---- library calls, mirrored ------------------------------------------------
    def _alloc(self, pool, owners):
        ids = ema.slice_alloc_blocks(self.w.h, pool, owners).astype(np.int64)
        if self.mirror is not None:
            mids = self.mirror.alloc_blocks(pool, owners)
            assert np.array_equal(ids, mids), "alloc: ids differ from the oracle's"
        return ids

    def _free(self, ids):
        ema.slice_free_blocks(self.w.h, ids)
        if self.mirror is not None:
            self.mirror.free_blocks(ids)

    def _migrate(self, src, dst):
        w = self.w
        ema.slice_migrate(w.h, torch.as_tensor(np.asarray(src, np.int32), device="cuda"),
                          torch.as_tensor(np.asarray(dst, np.int32), device="cuda"),
                          stream=self.runner.s1)
        if self.mirror is not None:
            self.mirror.migrate(src, dst)

    def _fill_new(self, ids):
        """New values for freshly allocated blocks (re-admitted sequences)."""
        w = self.w
        ids = np.asarray(ids, np.int64)
        for pool_ids, view, is_slice in ((ids[ids < w.n_local], w.local_view, False),
                                         (ids[ids >= w.n_local] - w.n_local, w.slice_view, True)):
            if not len(pool_ids):
                continue
            idx = torch.as_tensor(pool_ids, device="cuda")
            if self.fill == "host":
                data = synth.random_16bit(self.rng, (len(pool_ids), w.bb // 2), self.cfg.dtype)
                data = data.view(np.uint8).reshape(len(pool_ids), w.bb)
                view[idx] = torch.from_numpy(data).cuda()
                if self.mirror is not None and self.mirror.with_data:
                    (self.mirror.slice if is_slice else self.mirror.local)[pool_ids] = data
            else:
                g = torch.Generator(device="cuda")
                g.manual_seed(int(self.rng.integers(1 << 62)))
                vals = torch.randn((len(pool_ids), w.bb // 2), generator=g, device="cuda")
                view[idx] = vals.to(TORCH_DT[self.cfg.dtype]).view(torch.uint8)

    # ---- the trace ----------------------------------------------------------------
    def lender(self):
        w = self.w
        for b in sorted(self.waiting):
            self.readmit(b)
        info = ema.slice_get_info(w.h)
        lim = info["lim"]
        q = self.rng.uniform(*self.cfg.extra.get("step_frac", (0.01, 0.25)))
        if self.rng.integers(2) == 0:
            n = _round_half_up(q * lim)
            torch.cuda.synchronize()
            w.tables_dev.copy_(torch.from_numpy(w.tables.astype(np.int32)))
            r = ema.slice_reclaim(w.h, n, w.tables_dev.view(-1), stream=self.runner.s1)
            torch.cuda.synchronize()
            # the host applies the returned plan to its own tables; the device
            # rewrite must agree with it
            t = w.tables
            remap = np.arange(w.n_local + self.n_slice, dtype=np.int64)
            mv = np.asarray(r["moves"], dtype=np.int64).reshape(-1, 2)
            remap[mv[:, 0]] = mv[:, 1]
            valid = t >= 0
            t[valid] = remap[t[valid]]
            for v in r["victims"]:
                t[:, v, :] = -1
            self.check_device_tables()
            if self.mirror is not None:
                mr = self.mirror.reclaim(n, self.mtables)
                for k in ("reclaimed", "moved", "written_back", "lim"):
                    assert r[k] == mr[k], f"reclaim {k}: {r[k]} != oracle {mr[k]}"
                assert list(r["victims"]) == list(mr["victims"]), "reclaim victims differ"
                assert np.array_equal(mv, np.asarray(mr["moves"], np.int64).reshape(-1, 2)), \
                    "reclaim moves differ from the oracle's"
                assert np.array_equal(t, self.mtables), "reclaim: tables differ from the oracle's"
            self.log.append(("reclaim", n, r["moved"], r["written_back"], list(r["victims"])))
            for v in r["victims"]:
                self.readmit(int(v))
            return r
        n = _round_half_up(q * (self.n_slice - lim))
        added = ema.slice_lend(w.h, n)
        if self.mirror is not None:
            assert self.mirror.lend(n) == added
        self.log.append(("lend", n, added))
        return None

    def readmit(self, b):
        """A preempted sequence starts over with new values: as many of its
        blocks as fit in the local pool, the rest in free slice slots. Without
        room for all of them it waits, with length 0, for a later step."""
        w = self.w
        n0 = int(self.len0[b])
        nb = (n0 + w.bs - 1) // w.bs
        own_l, own_s, lim = ema.slice_owners(w.h)
        free_l = int((own_l == ema.FREE).sum())
        free_s = int((own_s[:lim] == ema.FREE).sum())
        need = self.L * nb
        if need > free_l + free_s:
            self.waiting.add(b)
            self._set_len(b, 0)
            return False
        self.waiting.discard(b)
        ids = self._alloc(ema.POOL_LOCAL, np.full(min(need, free_l), b))
        if need > free_l:
            ids = np.concatenate([ids, self._alloc(ema.POOL_SLICE, np.full(need - free_l, b))])
        w.tables[:, b, :nb] = ids.reshape(self.L, nb)
        if self.mirror is not None:
            self.mtables[:, b, :nb] = ids.reshape(self.L, nb)
        self._fill_new(ids)
        self._set_len(b, n0)
        self.readmitted.add(b)
        torch.cuda.synchronize()
        return True

    def _set_len(self, b, n):
        self.w.lens[b] = n
        self.w.lens_dev[b] = n

    def borrower(self):
        w = self.w
        self.f = float(np.clip(self.f + self.rng.uniform(-0.1, 0.1), 0.0, self.fmax))
        t = w.tables
        in_slice = t >= w.n_local
        cur = int(in_slice.sum())
        want = _round_half_up(self.f * self.T)
        own_l, own_s, lim = ema.slice_owners(w.h)
        if want > cur:
            free_s = int((own_s[:lim] == ema.FREE).sum())
            k = min(want - cur, free_s)
            cand = np.argwhere((t >= 0) & ~in_slice)
            to = ema.POOL_SLICE
        else:
            free_l = int((own_l == ema.FREE).sum())
            k = min(cur - want, free_l)
            cand = np.argwhere(in_slice)
            to = ema.POOL_LOCAL
        if k <= 0:
            self.log.append(("migrate", to, 0))
            return 0
        pick = cand[self.rng.choice(len(cand), size=k, replace=False)]
        src = t[pick[:, 0], pick[:, 1], pick[:, 2]]
        dst = self._alloc(to, pick[:, 1])
        self._migrate(src, dst)
        self._free(src)
        t[pick[:, 0], pick[:, 1], pick[:, 2]] = dst
        if self.mirror is not None:
            self.mtables[pick[:, 0], pick[:, 1], pick[:, 2]] = dst
        self.log.append(("migrate", to, k))
        return k

    def decode(self, timed=True):
        """Rebuild staging lists and attention tables, upload the canonical
        tables, run one overlapped decode step; returns its time in ms."""
        w = self.w
        torch.cuda.synchronize()
        w.tables_dev.copy_(torch.from_numpy(w.tables.astype(np.int32)))
        w.restage()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(self.runner.s1)
        self.runner.run(self.out)
        self.runner.s1.wait_stream(self.runner.s2)
        e1.record(self.runner.s1)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def step(self):
        r = self.lender()
        k = self.borrower()
        ms = self.decode()
        self.step_no += 1
        return {"step": self.step_no, "reclaim": r is not None, "migrated": k, "f": self.f,
                "slice_frac": float((self.w.tables >= self.w.n_local).sum()) / self.T,
                "lim": ema.slice_get_info(self.w.h)["lim"], "ms": ms}

    # ---- checks -------------------------------------------------------------------------
    def check_device_tables(self):
        dev = self.w.tables_dev.cpu().numpy().reshape(self.w.tables.shape)
        assert np.array_equal(dev, self.w.tables.astype(np.int32)), \
            "device-rewritten tables differ from the host's"

    def check_invariants(self):
        """Exactly-once ownership and tag conservation on the library's owner
        arrays, vectorised (the oracle's own checks loop over every block)."""
        w = self.w
        own_l, own_s, lim = ema.slice_owners(w.h)
        own = np.concatenate([own_l, own_s]).astype(np.int64)
        t = w.tables
        valid = t >= 0
        ids = t[valid]
        rows = np.nonzero(valid)[1]
        assert np.array_equal(own[ids], rows), "a table entry is not owned by its row"
        assert len(np.unique(ids)) == len(ids), "a block is referenced twice"
        assert np.array_equal(np.sort(ids), np.nonzero(own >= 0)[0]), \
            "an owned block is not referenced by any table"
        assert np.all((own_l >= 0) | (own_l == ema.FREE) | (own_l == ema.STAGING))
        assert np.all(own_s[lim:] == ema.LENDER), "non-lender tag at or above lim"
        assert np.all((own_s[:lim] >= 0) | (own_s[:lim] == ema.FREE)), "lender tag below lim"
        if self.mirror is not None:
            assert np.array_equal(own_l, self.mirror.own_local)
            assert np.array_equal(own_s, self.mirror.own_slice)
            assert lim == self.mirror.lim

    def fingerprints(self):
        """64-bit weighted checksum of every logical block (l, b, j) the
        canonical tables reference, in np.nonzero order; -1 where unused."""
        w = self.w
        t = w.tables
        pos = t >= 0
        ids = t[pos]
        words = w.bb // 4
        lv = w.local_view.view(torch.int32).view(-1, words)
        sv = w.slice_view.view(torch.int32).view(-1, words)
        weight = torch.arange(1, words + 1, device="cuda", dtype=torch.int64)
        fp = np.empty(len(ids), dtype=np.int64)
        for c0 in range(0, len(ids), 2048):
            chunk = torch.as_tensor(ids[c0:c0 + 2048], device="cuda")
            loc = chunk < w.n_local
            rows = torch.empty((len(chunk), words), dtype=torch.int32, device="cuda")
            if bool(loc.any()):
                rows[loc] = lv[chunk[loc]]
            if bool((~loc).any()):
                rows[~loc] = sv[chunk[~loc] - w.n_local]
            fp[c0:c0 + len(chunk)] = (rows.to(torch.int64) * weight).sum(dim=1).cpu().numpy()
        out = np.full(t.shape, -1, dtype=np.int64)
        out[pos] = fp
        return out

    def close(self):
        self.w.close()

"""Sets a synthetic KV-cache workload up in the library (GPU tests and bench).

A ``Workload`` owns one slice handle sized for the config: every logical
block of every layer allocated (local or slice per the seeded placement, in a
seeded random order so physical ids are scattered), ``staging_slots`` layers'
worth of STAGING local blocks that the prefetches fill, and device copies of
the canonical tables, the prefetch lists (per layer and per layer group) and
per-layer attention tables (canonical with each slice id replaced by the
staging block it is prefetched into).

Values: ``fill="host"`` draws every pool element on the host (iid N(0,1)
rounded to 16 bits) and writes NaN into unused tail token slots, keeping a host
image for the oracle; ``fill="device"`` draws them on the GPU with a seeded
torch generator (large configs) and the oracle reads back what it needs.
"""
import numpy as np
import torch

import synth
from paper_2609_27040_amd import ema

TORCH_DT = {"f16": torch.float16, "bf16": torch.bfloat16}


class Workload:
    def __init__(self, cfg, layers=None, batch=None, slice_layout=ema.LAYOUT_ATTN, seed=None,
                 staging_slots=2, extra_local=0, extra_slice=0, fill="host", checked=False,
                 lens=None, frac=None, shuffle=True, stage_n=None, group=1, attn_grid=False):
        self.cfg = cfg = cfg if batch is None else cfg.scaled(batch=batch)
        self.L = cfg.layers if layers is None else layers
        rng = np.random.default_rng(cfg.seed if seed is None else seed)
        self.lens = synth.seq_lens(cfg, rng) if lens is None else np.asarray(lens, np.int64)
        self.B = len(self.lens)
        self.pl = pl = synth.placement(cfg, self.lens, rng, frac=frac, layers=self.L,
                                       shuffle=shuffle)
        self.bs, self.hkv, self.D = cfg.block_size, cfg.kv_heads, cfg.head_dim
        self.bb = cfg.block_bytes
        self.maxblk = max(pl.maxblk, 1)
        self.slice_layout = slice_layout
        self.slice_per_layer = pl.in_slice.reshape(self.L, -1).sum(axis=1)
        self.stage_n = (int(self.slice_per_layer.max()) if self.L else 0) if stage_n is None \
            else int(stage_n)
        self.staging_slots = staging_slots
        self.group = max(1, int(group))
        n_local = len(pl.local_order) + staging_slots * self.stage_n + extra_local
        n_slice = len(pl.slice_order) + extra_slice
        self.h = ema.slice_create(self.hkv, self.D, self.bs, cfg.dtype, slice_layout,
                                  n_local * self.bb, n_slice * self.bb, checked=checked,
                                  attn_grid=attn_grid)
        self.alloc_log = []
        tables = np.full((self.L, self.B, self.maxblk), -1, dtype=np.int64)
        for pool, order in ((ema.POOL_LOCAL, pl.local_order), (ema.POOL_SLICE, pl.slice_order)):
            if len(order):
                owners = order[:, 1]
                ids = ema.slice_alloc_blocks(self.h, pool, owners)
                self.alloc_log.append((pool, owners.copy()))
                tables[order[:, 0], order[:, 1], order[:, 2]] = ids
        self.tables = tables
        st_owners = np.full(staging_slots * self.stage_n, ema.STAGING)
        self.staging = ema.slice_alloc_blocks(self.h, ema.POOL_LOCAL, st_owners).reshape(
            staging_slots, self.stage_n) if len(st_owners) else np.zeros((staging_slots, 0), np.int32)
        self.alloc_log.append((ema.POOL_LOCAL, st_owners))
        info = ema.slice_get_info(self.h)
        self.n_local = info["n_local"]
        self.q16 = synth.q_values(cfg, rng, self.B)
        dev = torch.device("cuda")
        self.q = torch.from_numpy(self.q16.view(np.int16)).to(dev).view(TORCH_DT[cfg.dtype])
        self.lens_dev = torch.from_numpy(self.lens.astype(np.int32)).to(dev)
        self.tables_dev = torch.from_numpy(tables.astype(np.int32)).to(dev)
        self.attn_dev = None
        self.restage()
        self.local_view = ema.pool_view(self.h, ema.POOL_LOCAL)
        self.slice_view = ema.pool_view(self.h, ema.POOL_SLICE)
        self.host_local = self.host_slice = None
        if fill == "host":
            self._fill_host(rng)
        elif fill == "device":
            self._fill_device(cfg.seed if seed is None else seed)
        elif fill == "pattern":
            self._fill_pattern()
        torch.cuda.synchronize()

    # ---- values -----------------------------------------------------------------
    def _tail_positions(self, layout):
        """(block-row index into tables, element indices) of unused tail slots."""
        out = []
        for b in range(self.B):
            n = int(self.lens[b])
            r = n % self.bs
            if n == 0 or r == 0:
                continue
            j = (n - 1) // self.bs
            t = np.arange(r, self.bs)
            h, tt, d = np.meshgrid(np.arange(self.hkv), t, np.arange(self.D), indexing="ij")
            idx = np.concatenate([synth.element_index(layout, half, h, tt, d, self.hkv, self.bs,
                                                      self.D).ravel() for half in (0, 1)])
            out.append((b, j, idx))
        return out

    def _fill_host(self, rng):
        n_l, n_s = self.local_view.shape[0], self.slice_view.shape[0]
        half = self.bb // 2
        loc = synth.random_16bit(rng, (n_l, half), self.cfg.dtype)
        sli = synth.random_16bit(rng, (n_s, half), self.cfg.dtype)
        nan = synth.NAN16[self.cfg.dtype]
        for pool_arr, layout, is_slice in ((loc, synth.LAYOUT_ATTN, False),
                                           (sli, self.slice_layout, True)):
            for b, j, idx in self._tail_positions(layout):
                for l in range(self.L):
                    u = int(self.tables[l, b, j])
                    if (u >= self.n_local) == is_slice:
                        pool_arr[u - self.n_local if is_slice else u, idx] = nan
        # staging blocks start as a recognisable sentinel
        stg = self.staging.ravel()
        loc[stg] = 0xA5A5
        self.host_local = loc.view(np.uint8).reshape(n_l, self.bb)
        self.host_slice = sli.view(np.uint8).reshape(n_s, self.bb)
        self.local_view.copy_(torch.from_numpy(self.host_local))
        if n_s:
            self.slice_view.copy_(torch.from_numpy(self.host_slice))

    def _fill_device(self, seed):
        g = torch.Generator(device="cuda")
        g.manual_seed(int(seed))
        dt = TORCH_DT[self.cfg.dtype]
        for view in (self.local_view, self.slice_view):
            flat = view.view(-1).view(dt)
            chunk = 1 << 28
            for s in range(0, flat.numel(), chunk):
                e = min(flat.numel(), s + chunk)
                flat[s:e].copy_(torch.randn(e - s, generator=g, device="cuda", dtype=torch.float32))

    def restage(self):
        """Per-layer prefetch lists and attention tables from the canonical
        tables ``self.tables``: layer l's slice-resident blocks are prefetched, in
        table order, into staging slot l % staging_slots, and its attention table
        is the canonical one with each slice id replaced by its staging block."""
        tables = self.tables
        self.pf_src, self.pf_dst = [], []
        attn = tables.copy()
        for l in range(self.L):
            mask = tables[l] >= self.n_local
            src = tables[l][mask]
            if len(src) > self.stage_n:
                raise ValueError(f"layer {l}: {len(src)} slice blocks, staging holds {self.stage_n}")
            dst = self.staging[l % self.staging_slots, :len(src)]
            attn[l][mask] = dst
            self.pf_src.append(src.astype(np.int32))
            self.pf_dst.append(dst.astype(np.int32))
        self.attn_tables = attn
        # blocks a decode-step append writes: each sequence's last block; those
        # in the slice are written through their staged copy and written back
        self.wb_src, self.wb_dst = [], []
        rows = np.arange(self.B)
        last = np.maximum(self.lens - 1, 0) // self.bs
        for l in range(self.L):
            canon = tables[l, rows, last] if self.B else np.zeros(0, np.int64)
            dirty = (canon >= self.n_local) & (self.lens > 0)
            self.wb_src.append(attn[l, rows, last][dirty].astype(np.int32))
            self.wb_dst.append(canon[dirty].astype(np.int32))
        dev = torch.device("cuda")
        a32 = torch.from_numpy(attn.astype(np.int32))
        if self.attn_dev is None or self.attn_dev.shape != a32.shape:
            self.attn_dev = a32.to(dev)
        else:
            self.attn_dev.copy_(a32)
        self.pf_src_dev = [torch.from_numpy(s).to(dev) for s in self.pf_src]
        self.pf_dst_dev = [torch.from_numpy(d).to(dev) for d in self.pf_dst]
        self.wb_src_dev = [torch.from_numpy(s).to(dev) for s in self.wb_src]
        self.wb_dst_dev = [torch.from_numpy(d).to(dev) for d in self.wb_dst]
        # one list per layer group (consecutive layers, swapped together)
        g = self.group
        self.groups = [list(range(k, min(self.L, k + g))) for k in range(0, self.L, g)]
        self.pf_src_grp, self.pf_dst_grp = [], []
        for ls in self.groups:
            src = np.concatenate([self.pf_src[l] for l in ls]) if ls else np.zeros(0, np.int32)
            dst = np.concatenate([self.pf_dst[l] for l in ls]) if ls else np.zeros(0, np.int32)
            self.pf_src_grp.append(src)
            self.pf_dst_grp.append(dst)
        self.wb_src_grp = [np.concatenate([self.wb_src[l] for l in ls]) for ls in self.groups]
        self.wb_dst_grp = [np.concatenate([self.wb_dst[l] for l in ls]) for ls in self.groups]
        if g == 1:
            self.pf_src_grp_dev, self.pf_dst_grp_dev = self.pf_src_dev, self.pf_dst_dev
            self.wb_src_grp_dev, self.wb_dst_grp_dev = self.wb_src_dev, self.wb_dst_dev
        else:
            self.pf_src_grp_dev = [torch.from_numpy(s).to(dev) for s in self.pf_src_grp]
            self.pf_dst_grp_dev = [torch.from_numpy(d).to(dev) for d in self.pf_dst_grp]
            self.wb_src_grp_dev = [torch.from_numpy(s).to(dev) for s in self.wb_src_grp]
            self.wb_dst_grp_dev = [torch.from_numpy(d).to(dev) for d in self.wb_dst_grp]

    def _fill_pattern(self):
        """Every 8-byte word of both pools gets a distinct value (its position,
        the slice pool offset past the local one): cheap at any size, and any
        misplaced copy shows. Not attention data (random bit patterns)."""
        base = 0
        for view in (self.local_view, self.slice_view):
            flat = view.view(-1).view(torch.int64)
            chunk = 1 << 28
            for s in range(0, flat.numel(), chunk):
                e = min(flat.numel(), s + chunk)
                torch.arange(base + s, base + e, dtype=torch.int64, device="cuda", out=flat[s:e])
            base += flat.numel()

    # ---- the hot path ---------------------------------------------------------------
    def prefetch(self, l, stream=None):
        ema.slice_prefetch(self.h, self.pf_src_dev[l], self.pf_dst_dev[l], len(self.pf_src[l]),
                           stream=stream)

    def prefetch_group(self, k, stream=None):
        """Every slice-resident block of layer group k in one call."""
        ema.slice_prefetch(self.h, self.pf_src_grp_dev[k], self.pf_dst_grp_dev[k],
                           len(self.pf_src_grp[k]), stream=stream)

    def append(self, l, k_new, v_new, stream=None):
        ema.kv_append(self.h, k_new, v_new, self.attn_dev[l], self.lens_dev, stream=stream)

    def writeback_group(self, k, stream=None):
        """The staged copies layer group k's appends modified, back to the slice."""
        ema.slice_writeback(self.h, self.wb_src_grp_dev[k], self.wb_dst_grp_dev[k],
                            len(self.wb_src_grp[k]), stream=stream)

    def new_token_kv(self, seed=0):
        """One new token's K and V per sequence (device, the cache dtype)."""
        g = torch.Generator(device="cuda")
        g.manual_seed(int(seed))
        shape = (self.B, self.hkv, self.D)
        dt = TORCH_DT[self.cfg.dtype]
        return (torch.randn(shape, generator=g, device="cuda").to(dt),
                torch.randn(shape, generator=g, device="cuda").to(dt))

    def attention(self, l, out, table=None, stream=None):
        ema.paged_decode_attention(self.h, self.q, self.attn_dev[l] if table is None else table,
                                   self.lens_dev, out, stream=stream)

    def new_out(self):
        return torch.empty((self.B, self.cfg.q_heads, self.D), dtype=torch.float32, device="cuda")

    def close(self):
        self.local_view = self.slice_view = None
        torch.cuda.synchronize()
        ema.slice_destroy(self.h)

    # ---- oracle side ------------------------------------------------------------------
    def oracle_mirror(self):
        """An oracle slice replaying the same allocations, holding the host image."""
        import oracle
        st = oracle.SliceOracle(self.hkv, self.D, self.bs, self.cfg.dtype, self.slice_layout,
                                self.local_view.shape[0] * self.bb,
                                self.slice_view.shape[0] * self.bb)
        for pool, owners in self.alloc_log:
            st.alloc_blocks(pool, owners)
        own_l, own_s, lim = ema.slice_owners(self.h)
        assert np.array_equal(own_l, st.own_local) and np.array_equal(own_s, st.own_slice)
        st.local[:] = self.host_local
        st.slice[:] = self.host_slice
        return st


class StepRunner:
    """One decode step of a workload, prefetching per layer group (the
    workload's ``group`` consecutive layers, swapped together in one call).
    Staging slot l % S holds layer l's staged blocks (S = ``w.staging_slots``,
    a multiple of the group size), so S / group groups are in flight at most;
    a group's slots are refilled only after the attention that last read them,
    and attention of a layer waits for its group's prefetch.

    ``mode="serial"``: one stream, each group's prefetch followed by its
    layers' attention (with S = 2·group the next group's prefetch is queued
    before the current group's attention, which is the same work in another
    order). ``mode="overlap"``: prefetches on a second stream, up to
    S / group − 1 groups ahead of the attention stream (needs S ≥ 2·group).

    With ``append``, each layer first stores the new token's K/V (into the
    staged copy where the block is in the slice) and, after the group's last
    attention, the group's modified staged copies are written back on the copy
    stream (one call per group), before its slots are refilled.

    ``timers`` (optional) maps group index (``"pf"``) or layer (``"at"``) to
    the event pair recorded around that call, and group index (``"atg"``) to
    one event pair around the group's consecutive attention calls (steps
    without append only); entries missing from a map are not timed (every
    timing event costs device time)."""

    def __init__(self, w, mode="overlap", append=False):
        self.w = w
        g, S = w.group, w.staging_slots
        if S % g or S < g or (mode == "overlap" and S < 2 * g):
            raise ValueError(f"{S} staging slots do not fit groups of {g} layers ({mode})")
        self.kv_new = w.new_token_kv() if append else None
        self.s1 = torch.cuda.Stream()
        self.s2 = torch.cuda.Stream() if mode == "overlap" else self.s1
        self.unit_slots = S // g
        self.ahead = self.unit_slots - 1
        self.ev_pf = [torch.cuda.Event() for _ in range(len(w.groups))]
        self.ev_at = [torch.cuda.Event() for _ in range(w.L)]

    def new_timers(self, layers=None, groups=None, attn_groups=()):
        mk = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        layers = range(self.w.L) if layers is None else layers
        if attn_groups and self.kv_new is not None:
            raise ValueError("group attention timers need steps without append")
        if groups is None:
            groups = sorted({l // self.w.group for l in layers} | set(attn_groups))
        return {"pf": {k: mk() for k in groups}, "at": {l: mk() for l in layers},
                "atg": {u: mk() for u in attn_groups}}

    def _attn_timer(self, l, timers):
        """(event pair, record before, record after) for layer l's attention."""
        if not timers:
            return None, False, False
        t = timers["at"].get(l)
        if t:
            return t, True, True
        grp = self.w.groups[l // self.w.group]
        t = timers.get("atg", {}).get(l // self.w.group)
        return t, bool(t) and l == grp[0], bool(t) and l == grp[-1]

    def _prefetch(self, k, timers):
        t = timers["pf"].get(k) if timers else None
        if t:
            t[0].record(self.s2)
        self.w.prefetch_group(k, stream=self.s2)
        if t:
            t[1].record(self.s2)
        self.ev_pf[k].record(self.s2)

    def ops(self, out):
        """One step in the one-stream schedule as an ordered list of
        (kind, index, call): "pf" (group prefetch), "ap" (append), "at"
        (attention of a layer), "wb" (group write-back). Stream order is the
        only dependency, so any contiguous run of them can be captured."""
        from functools import partial
        w, s = self.w, self.s1
        groups, ahead = w.groups, self.ahead
        NG = len(groups)
        ops = []
        for u in range(NG):
            first = range(min(ahead, NG)) if u == 0 else ()
            nxt = [u + ahead] if u + ahead < NG else []
            for k in list(first) + nxt:
                ops.append(("pf", k, partial(w.prefetch_group, k, stream=s)))
            for l in groups[u]:
                if self.kv_new is not None:
                    ops.append(("ap", l, partial(w.append, l, *self.kv_new, stream=s)))
                ops.append(("at", l, partial(w.attention, l, out, stream=s)))
            if self.kv_new is not None:
                ops.append(("wb", u, partial(w.writeback_group, u, stream=s)))
        return ops

    def run(self, out, timers=None):
        w, s1, s2 = self.w, self.s1, self.s2
        if s2 is s1:
            for kind, i, call in self.ops(out):
                if kind == "at":
                    t, before, after = self._attn_timer(i, timers)
                else:
                    t = timers.get(kind, {}).get(i) if timers else None
                    before = after = bool(t)
                if before:
                    t[0].record(s1)
                call()
                if after:
                    t[1].record(s1)
            return
        groups, US, ahead = w.groups, self.unit_slots, self.ahead
        NG = len(groups)
        for u in range(NG):
            if u == 0:
                # every slot was last read by the previous step's attention
                s2.wait_event(self.ev_at[w.L - 1])
                for k in range(min(ahead, NG)):
                    self._prefetch(k, timers)
            k = u + ahead
            if k < NG:
                if k - US >= 0:
                    # group k's slots were read by group k - US
                    s2.wait_event(self.ev_at[groups[k - US][-1]])
                self._prefetch(k, timers)
            s1.wait_event(self.ev_pf[u])
            for l in groups[u]:
                if self.kv_new is not None:
                    w.append(l, *self.kv_new, stream=s1)
                t, before, after = self._attn_timer(l, timers)
                if before:
                    t[0].record(s1)
                w.attention(l, out, stream=s1)
                if after:
                    t[1].record(s1)
                self.ev_at[l].record(s1)
            if self.kv_new is not None:
                # the group's modified staged copies go back before its slots are refilled
                s2.wait_event(self.ev_at[groups[u][-1]])
                w.writeback_group(u, stream=s2)


def capture_ops(runner, ops):
    """A contiguous run of a one-stream runner's step operations captured as a
    HIP graph (after warm-up steps, so every workspace already exists; nothing
    in the step allocates or clears memory, so the graph holds kernel and copy
    nodes only). None for an empty run."""
    if runner.s1 is not runner.s2:
        raise ValueError("only the one-stream schedule is captured")
    if not ops:
        return None
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=runner.s1):
        for _, _, call in ops:
            call()
    return g


def capture_step(runner, out):
    """One whole step of a one-stream runner as a HIP graph."""
    return capture_ops(runner, runner.ops(out))


class BlockedTimer:
    """Device time of one library call that also does host work (planning,
    uploads): the call is queued behind a device copy long enough to outlast
    its host part, so the events around it bracket device work only. The copy
    is sized from a host-time estimate (about 5 bytes per ns of copy traffic,
    three times the estimate, 2 to 32 GiB)."""

    def __init__(self):
        self.a = self.b = None

    def _blocker(self, host_ms):
        nbytes = int(min(32 << 30, max(2 << 30, 3 * host_ms * 1e-3 * 5e12 / 2)))
        if self.a is None or self.a.numel() * 2 < nbytes:
            self.a = self.b = None
            self.a = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
            self.b = torch.empty_like(self.a)
        return self.a[:nbytes // 2], self.b[:nbytes // 2]

    def time(self, stream, call, host_ms=0.0):
        """Returns (result, device ms, host ms, covered); covered is False when
        the blocking copy had already finished as the call returned."""
        import time as _time
        a, b = self._blocker(host_ms)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            b.copy_(a)
        e0.record(stream)
        c0 = _time.perf_counter()
        r = call()
        c1 = _time.perf_counter()
        covered = not e0.query()
        e1.record(stream)
        torch.cuda.synchronize()
        return r, e0.elapsed_time(e1), (c1 - c0) * 1e3, covered

    def close(self):
        self.a = self.b = None


def rel_err(out, ref):
    """max over (b, h) of ||o - ref||_inf / ||ref||_inf (rows with ref == 0: absolute)."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(out - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    den = np.where(den > 0, den, 1.0)
    return float((num / den).max()) if num.size else 0.0


def read_blocks(view, ids):
    """Host copies of the given blocks of a pool view (id -> bytes)."""
    ids = np.unique(np.asarray(ids, dtype=np.int64))
    ids = ids[ids >= 0]
    if not len(ids):
        return {}
    data = view[torch.from_numpy(ids).to(view.device)].cpu().numpy()
    return {int(u): data[i] for i, u in enumerate(ids)}

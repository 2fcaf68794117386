"""The decode step of a paged KV cache over a memory slice, and timers.

``StepRunner`` orders one decode step: per layer group, one prefetch call
swaps the group's slice-resident blocks into a staging area, then paged
decode attention runs for each of the group's layers (section 2.3: a layer is
not needed again until every other layer has run, which is the window the
swap of the next group overlaps; section 4.2.2: swaps are issued at layer
group boundaries into a swap buffer of one group). ``capture_ops`` and
``capture_step`` record a one-stream step as a HIP graph. ``BlockedTimer``
times a library call that also does host work.
"""
import torch


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

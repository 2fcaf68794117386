"""A seeded synthetic KV-cache workload on one slice handle.

``Workload`` takes a config from ``synth`` and builds a ``PagedKVCache``:
every logical block of every layer allocated (local or slice per the seeded
placement, in a seeded random order so physical ids are scattered, as in a
long-running cache), ``staging_slots`` layers' worth of STAGING local blocks
that the prefetches fill, the canonical and attention tables and the prefetch
lists, plus the decode queries.

Values: ``fill="host"`` draws every pool element on the host (iid N(0,1)
rounded to 16 bits) and writes NaN into unused tail token slots, keeping a host
image (``host_local`` / ``host_slice``) that an oracle can start from;
``fill="device"`` draws them on the GPU with a seeded torch generator (large
configs); ``fill="pattern"`` gives every 8-byte word a distinct value (copy
tests at any size).
"""
import numpy as np
import torch

import synth
from paper_2609_27040_amd import ema
from paper_2609_27040_amd.kvcache import TORCH_DT, PagedKVCache


class Workload(PagedKVCache):
    def __init__(self, cfg, layers=None, batch=None, slice_layout=ema.LAYOUT_ATTN, seed=None,
                 staging_slots=2, extra_local=0, extra_slice=0, fill="host", checked=False,
                 lens=None, frac=None, shuffle=True, stage_n=None, group=1, attn_grid=False):
        self.cfg = cfg = cfg if batch is None else cfg.scaled(batch=batch)
        L = cfg.layers if layers is None else layers
        rng = np.random.default_rng(cfg.seed if seed is None else seed)
        lens = synth.seq_lens(cfg, rng) if lens is None else np.asarray(lens, np.int64)
        self.pl = pl = synth.placement(cfg, lens, rng, frac=frac, layers=L, shuffle=shuffle)
        super().__init__(kv_heads=cfg.kv_heads, head_dim=cfg.head_dim,
                         block_size=cfg.block_size, dtype=cfg.dtype, slice_layout=slice_layout,
                         layers=L, lens=lens, maxblk=pl.maxblk, local_order=pl.local_order,
                         slice_order=pl.slice_order, q_heads=cfg.q_heads,
                         staging_slots=staging_slots, stage_n=stage_n, group=group,
                         extra_local=extra_local, extra_slice=extra_slice, checked=checked,
                         attn_grid=attn_grid)
        self.q16 = synth.q_values(cfg, rng, self.B)
        self.q = torch.from_numpy(self.q16.view(np.int16)).to("cuda").view(TORCH_DT[cfg.dtype])
        self.host_local = self.host_slice = None
        if fill == "host":
            self._fill_host(rng)
        elif fill == "device":
            self._fill_device(cfg.seed if seed is None else seed)
        elif fill == "pattern":
            self._fill_pattern()
        torch.cuda.synchronize()

    def _tail_positions(self, layout):
        """(sequence, last block index, element indices) of unused tail slots."""
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
        loc[self.staging.ravel()] = 0xA5A5
        self.host_local = loc.view(np.uint8).reshape(n_l, self.bb)
        self.host_slice = sli.view(np.uint8).reshape(n_s, self.bb)
        self.local_view.copy_(torch.from_numpy(self.host_local))
        if n_s:
            self.slice_view.copy_(torch.from_numpy(self.host_slice))

    def _fill_device(self, seed):
        fill_device(self, self.cfg.dtype, seed)

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


def fill_device(cache, dtype, seed):
    """Both pools of a cache: iid N(0,1) drawn on the GPU from a seeded torch
    generator, rounded to the 16-bit type."""
    g = torch.Generator(device="cuda")
    g.manual_seed(int(seed))
    dt = TORCH_DT[dtype]
    for view in (cache.local_view, cache.slice_view):
        flat = view.view(-1).view(dt)
        chunk = 1 << 28
        for s in range(0, flat.numel(), chunk):
            e = min(flat.numel(), s + chunk)
            flat[s:e].copy_(torch.randn(e - s, generator=g, device="cuda", dtype=torch.float32))

"""Paged KV caches over one memory slice: placement, tables and the calls of a
decode step (argument plumbing over the C ABI; every step runs in the
library's kernels).

``PagedKVCache`` places blocks one at a time (block-granular slice): each
layer's logical blocks go to the local pool or to slice slots in a caller-given
allocation order; before use, a layer group's slice-resident blocks are
prefetched into a staging area (section 5.1: the slice process prefetches
ahead of access; section 4.2.2: a swap buffer of one layer group per group in
flight), and attention reads an attention table -- the canonical table with
each slice id replaced by its staged copy -- so it only ever touches local
memory (section 3, local-remote symmetry).

``SlabKVCache`` manages the slice in slabs (section 4.2.1-4.2.3): a logical
block lives either locally in every layer or at one slab position (every
layer); the swap of a layer group copies whole slab runs into a staging image.

Both expose the same step interface (``groups``, ``group``, ``staging_slots``,
``prefetch_group``, ``attention``), which ``step.StepRunner`` drives.
"""
import numpy as np
import torch

from . import ema

TORCH_DT = {"f16": torch.float16, "bf16": torch.bfloat16}


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")


class PagedKVCache:
    """A block-granular paged KV cache on a new slice handle.

    ``local_order`` / ``slice_order``: int arrays [n][3] of (layer, sequence,
    logical block) giving each pool's allocation order (the owner of a block
    is its sequence). ``staging_slots`` layers' worth of STAGING local blocks,
    ``stage_n`` per layer, hold prefetched copies: layer l's in slot
    l % staging_slots. ``group`` consecutive layers are prefetched by one
    call. ``q`` (set by the caller) is the decode query [B][Hq][D]."""

    def __init__(self, *, kv_heads, head_dim, block_size, dtype, slice_layout, layers, lens,
                 maxblk, local_order, slice_order, q_heads, staging_slots=2, stage_n=None,
                 group=1, extra_local=0, extra_slice=0, checked=False, attn_grid=False):
        self.L, self.hkv, self.D, self.bs = int(layers), int(kv_heads), int(head_dim), int(block_size)
        self.dtype, self.slice_layout, self.q_heads = dtype, slice_layout, int(q_heads)
        self.bb = 2 * self.bs * self.hkv * self.D * 2
        self.lens = np.asarray(lens, dtype=np.int64)
        self.B = len(self.lens)
        self.maxblk = max(int(maxblk), 1)
        local_order = np.asarray(local_order, dtype=np.int64).reshape(-1, 3)
        slice_order = np.asarray(slice_order, dtype=np.int64).reshape(-1, 3)
        per_layer = np.bincount(slice_order[:, 0], minlength=self.L) if len(slice_order) \
            else np.zeros(self.L, np.int64)
        self.slice_per_layer = per_layer
        self.stage_n = (int(per_layer.max()) if self.L else 0) if stage_n is None else int(stage_n)
        self.staging_slots = int(staging_slots)
        self.group = max(1, int(group))
        n_local = len(local_order) + self.staging_slots * self.stage_n + int(extra_local)
        n_slice = len(slice_order) + int(extra_slice)
        self.h = ema.slice_create(self.hkv, self.D, self.bs, dtype, slice_layout,
                                  n_local * self.bb, n_slice * self.bb, checked=checked,
                                  attn_grid=attn_grid)
        self.alloc_log = []
        tables = np.full((self.L, self.B, self.maxblk), -1, dtype=np.int64)
        for pool, order in ((ema.POOL_LOCAL, local_order), (ema.POOL_SLICE, slice_order)):
            if len(order):
                owners = order[:, 1]
                ids = ema.slice_alloc_blocks(self.h, pool, owners)
                self.alloc_log.append((pool, owners.copy()))
                tables[order[:, 0], order[:, 1], order[:, 2]] = ids
        self.tables = tables
        st_owners = np.full(self.staging_slots * self.stage_n, ema.STAGING)
        self.staging = ema.slice_alloc_blocks(self.h, ema.POOL_LOCAL, st_owners).reshape(
            self.staging_slots, self.stage_n) if len(st_owners) else \
            np.zeros((self.staging_slots, 0), np.int32)
        self.alloc_log.append((ema.POOL_LOCAL, st_owners))
        self.n_local = ema.slice_get_info(self.h)["n_local"]
        self.q = None
        self.lens_dev = _dev(self.lens)
        self.tables_dev = _dev(tables)
        self.attn_dev = None
        self.restage()
        self.local_view = ema.pool_view(self.h, ema.POOL_LOCAL)
        self.slice_view = ema.pool_view(self.h, ema.POOL_SLICE)

    # ---- tables ---------------------------------------------------------------------
    def restage(self):
        """Per-layer prefetch lists and attention tables from the canonical
        tables ``self.tables``: layer l's slice-resident blocks are prefetched,
        in table order, into staging slot l % staging_slots, and its attention
        table is the canonical one with each slice id replaced by its staging
        block; plus, per layer, the write-back list of a decode-step append
        (each sequence's last block where it lives in the slice)."""
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
        self.wb_src, self.wb_dst = [], []
        rows = np.arange(self.B)
        last = np.maximum(self.lens - 1, 0) // self.bs
        for l in range(self.L):
            canon = tables[l, rows, last] if self.B else np.zeros(0, np.int64)
            dirty = (canon >= self.n_local) & (self.lens > 0)
            self.wb_src.append(attn[l, rows, last][dirty].astype(np.int32))
            self.wb_dst.append(canon[dirty].astype(np.int32))
        a32 = torch.from_numpy(attn.astype(np.int32))
        if self.attn_dev is None or self.attn_dev.shape != a32.shape:
            self.attn_dev = a32.to("cuda")
        else:
            self.attn_dev.copy_(a32)
        self.pf_src_dev = [_dev(s) for s in self.pf_src]
        self.pf_dst_dev = [_dev(d) for d in self.pf_dst]
        self.wb_src_dev = [_dev(s) for s in self.wb_src]
        self.wb_dst_dev = [_dev(d) for d in self.wb_dst]
        g = self.group
        self.groups = [list(range(k, min(self.L, k + g))) for k in range(0, self.L, g)]
        cat = lambda parts: np.concatenate(parts) if parts else np.zeros(0, np.int32)
        self.pf_src_grp = [cat([self.pf_src[l] for l in ls]) for ls in self.groups]
        self.pf_dst_grp = [cat([self.pf_dst[l] for l in ls]) for ls in self.groups]
        self.wb_src_grp = [cat([self.wb_src[l] for l in ls]) for ls in self.groups]
        self.wb_dst_grp = [cat([self.wb_dst[l] for l in ls]) for ls in self.groups]
        if g == 1:
            self.pf_src_grp_dev, self.pf_dst_grp_dev = self.pf_src_dev, self.pf_dst_dev
            self.wb_src_grp_dev, self.wb_dst_grp_dev = self.wb_src_dev, self.wb_dst_dev
        else:
            self.pf_src_grp_dev = [_dev(s) for s in self.pf_src_grp]
            self.pf_dst_grp_dev = [_dev(d) for d in self.pf_dst_grp]
            self.wb_src_grp_dev = [_dev(s) for s in self.wb_src_grp]
            self.wb_dst_grp_dev = [_dev(d) for d in self.wb_dst_grp]

    # ---- the calls of a decode step ------------------------------------------------------
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

    def attention(self, l, out, table=None, stream=None):
        ema.paged_decode_attention(self.h, self.q, self.attn_dev[l] if table is None else table,
                                   self.lens_dev, out, stream=stream)

    def new_token_kv(self, seed=0):
        """One new token's K and V per sequence (device, the cache dtype),
        drawn from a seeded generator: the values a decode step appends."""
        g = torch.Generator(device="cuda")
        g.manual_seed(int(seed))
        shape = (self.B, self.hkv, self.D)
        dt = TORCH_DT[self.dtype]
        return (torch.randn(shape, generator=g, device="cuda").to(dt),
                torch.randn(shape, generator=g, device="cuda").to(dt))

    def new_out(self, dtype=torch.float32):
        return torch.empty((self.B, self.q_heads, self.D), dtype=dtype, device="cuda")

    def close(self):
        self.local_view = self.slice_view = None
        torch.cuda.synchronize()
        ema.slice_destroy(self.h)


class SlabKVCache:
    """A paged KV cache whose slice is managed in slabs (section 4.2.1-4.2.3).

    ``in_slab``: bool [B][maxblk], the logical blocks that live at a slab
    position (all layers); the others get one local block per layer.
    ``order``: int array [n][2] of (sequence, logical block), the allocation
    order of all logical blocks. Slabs of ``slab_blocks`` positions, placed
    ``slab_layout``; ``group`` layers per layer group; ``images`` staging
    images of one group each, group u swapped into image u % images. The slice
    holds exactly the slabs needed plus ``extra_slabs``. ``gap_slabs``
    (optional bool per slab, in index order) marks slabs that another user
    holds while the borrower's blocks are placed: they are taken by a
    placeholder first and released at the end, so they sit free between the
    borrower's slabs."""

    def __init__(self, *, kv_heads, head_dim, block_size, dtype, slice_layout, layers, lens,
                 maxblk, in_slab, order, q_heads, slab_blocks, group, slab_layout,
                 images=2, extra_slabs=0, engine=ema.ENGINE_KERNEL, gap_slabs=None):
        self.L, self.hkv, self.D, self.bs = int(layers), int(kv_heads), int(head_dim), int(block_size)
        self.dtype, self.slice_layout, self.q_heads = dtype, slice_layout, int(q_heads)
        self.S, self.group, self.slab_layout = int(slab_blocks), int(group), slab_layout
        self.engine = engine
        self.bb = 2 * self.bs * self.hkv * self.D * 2
        self.lens = np.asarray(lens, dtype=np.int64)
        self.B = len(self.lens)
        self.maxblk = max(int(maxblk), 1)
        in_slab = np.asarray(in_slab, dtype=bool)
        order = np.asarray(order, dtype=np.int64).reshape(-1, 2)
        n_pos = int(in_slab.sum())
        n_slabs = -(-n_pos // self.S) + int(extra_slabs)
        n_loc_blocks = (len(order) - n_pos) * self.L
        self.images = int(images)
        stage = self.images * n_slabs * self.group * self.S
        self.h = ema.slice_create(self.hkv, self.D, self.bs, dtype, slice_layout,
                                  (n_loc_blocks + stage) * self.bb,
                                  n_slabs * self.L * self.S * self.bb)
        ema.slab_init(self.h, self.L, self.S, self.group, slab_layout)
        tables = np.full((self.L, self.B, self.maxblk), -1, dtype=np.int64)
        sl = in_slab[order[:, 0], order[:, 1]]
        slab_o, loc_o = order[sl], order[~sl]
        self.pos = np.full((self.B, self.maxblk), -1, dtype=np.int64)
        if len(slab_o):
            got = np.empty(len(slab_o), dtype=np.int64)
            held, t = [], 0
            gaps = np.zeros(0, bool) if gap_slabs is None else np.asarray(gap_slabs, bool)
            for gap in gaps:          # one slab per call, in slab order
                if t >= len(slab_o) or (t % self.S):
                    break
                if gap:
                    held.append(ema.slab_alloc(self.h, np.full(self.S, self.B)))
                else:
                    n = min(self.S, len(slab_o) - t)
                    got[t:t + n] = ema.slab_alloc(self.h, slab_o[t:t + n, 0])
                    t += n
            if t < len(slab_o):
                got[t:] = ema.slab_alloc(self.h, slab_o[t:, 0])
            if held:
                ema.slab_free(self.h, np.concatenate(held))
            self.pos[slab_o[:, 0], slab_o[:, 1]] = got
        if len(loc_o):
            ids = ema.slice_alloc_blocks(self.h, ema.POOL_LOCAL, np.repeat(loc_o[:, 0], self.L))
            ids = ids.reshape(len(loc_o), self.L)
            for l in range(self.L):
                tables[l, loc_o[:, 0], loc_o[:, 1]] = ids[:, l]
        used = self.pos >= 0
        for l in range(self.L):
            tables[l][used] = ema.slab_block_ids(self.h, self.pos[used], l)
        self.tables = tables
        self.n_local = ema.slice_get_info(self.h)["n_local"]
        info = ema.slab_get_info(self.h)
        self.m = info["borrowed"]
        per_image = self.m * self.group * self.S
        st = ema.slice_alloc_blocks(self.h, ema.POOL_LOCAL,
                                    np.full(self.images * per_image, ema.STAGING))
        if len(st) and not np.array_equal(st, st[0] + np.arange(len(st))):
            raise RuntimeError("staging images are not contiguous")
        self.image_first = [int(st[0]) + i * per_image if len(st) else 0
                            for i in range(self.images)]
        self.staging_slots = self.images * self.group     # step runner: images groups in flight
        self.groups = [list(range(k, k + self.group)) for k in range(0, self.L, self.group)]
        attn = tables.copy()
        for l in range(self.L):
            first = self.image_first[(l // self.group) % self.images]
            attn[l][used] = ema.slab_block_ids(self.h, self.pos[used], l, first)
        self.attn_tables = attn
        self.attn_dev = _dev(attn)
        self.tables_dev = _dev(tables)
        self.lens_dev = _dev(self.lens)
        self.q = None
        self.local_view = ema.pool_view(self.h, ema.POOL_LOCAL)
        self.slice_view = ema.pool_view(self.h, ema.POOL_SLICE)

    def group_runs(self, k):
        """(src_first, dst_first, run_blocks) of group k's swap."""
        return ema.slab_group_runs(self.h, k, self.image_first[k % self.images])

    def swap_blocks(self):
        """Blocks one group's swap moves (whole borrowed slabs)."""
        return self.m * self.group * self.S

    def prefetch_group(self, k, stream=None):
        ema.slab_prefetch_group(self.h, k, self.image_first[k % self.images], self.engine,
                                stream=stream)

    def attention(self, l, out, table=None, stream=None):
        ema.paged_decode_attention(self.h, self.q, self.attn_dev[l] if table is None else table,
                                   self.lens_dev, out, stream=stream)

    def new_out(self, dtype=torch.float32):
        return torch.empty((self.B, self.q_heads, self.D), dtype=dtype, device="cuda")

    def close(self):
        self.local_view = self.slice_view = None
        torch.cuda.synchronize()
        ema.slice_destroy(self.h)

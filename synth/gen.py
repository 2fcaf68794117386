"""Seeded generators: sequence lengths, block placement, 16-bit values.

Generation order for a workload is fixed: lengths, then placement, then values,
all from one ``numpy.random.default_rng(cfg.seed)`` stream.

The byte format helpers at the bottom (``element_index``, ``pack_block``)
state where each K/V element of a layer-block sits in the two block layouts, so
that tests can write values and NaN sentinels into exact token positions. They
are written independently of the oracle's own layout code on purpose: a parity
test through both catches a mistake in either.
"""
from dataclasses import dataclass
import numpy as np

LAYOUT_ATTN = 0   # local pool: K [Hkv][bs][D], then V transposed [Hkv][D][bs]
LAYOUT_NHD = 1    # token-major: K [bs][Hkv][D], then V [bs][Hkv][D]


def _round_half_up(x: float) -> int:
    return int(np.floor(x + 0.5))


def seq_lens(cfg, rng) -> np.ndarray:
    """Per-sequence token counts, int64 [batch].

    uniform: integers in [lo, hi] inclusive.
    lognormal: round(exp(N(ln median, sigma))) then clipped to [lo, hi].
    """
    kind = cfg.lens[0]
    if kind == "uniform":
        lo, hi = cfg.lens[1], cfg.lens[2]
        return rng.integers(lo, hi + 1, size=cfg.batch).astype(np.int64)
    if kind == "lognormal":
        median, sigma, lo, hi = cfg.lens[1:]
        x = rng.lognormal(mean=np.log(median), sigma=sigma, size=cfg.batch)
        return np.clip(np.rint(x), lo, hi).astype(np.int64)
    raise ValueError(kind)


@dataclass
class BlockPlacement:
    """Where each logical KV block of a batch goes.

    nblocks[b]       blocks of sequence b (same in every layer)
    maxblk           max(nblocks), the width of every block table
    in_slice         bool [L][B][maxblk]; True where the logical block is
                     slice-resident (False also on padding)
    local_order      int64 [n, 3] rows (layer, seq, j) of the local blocks, in
                     the order they are to be allocated (a seeded permutation,
                     so physical ids are scattered as in a long-running cache)
    slice_order      same for the slice-resident blocks
    """
    nblocks: np.ndarray
    maxblk: int
    in_slice: np.ndarray
    local_order: np.ndarray
    slice_order: np.ndarray


def placement(cfg, lens, rng, frac=None, layers=None, shuffle=True) -> BlockPlacement:
    """Pick, per layer, exactly round(frac * n_l) of the layer's n_l logical
    blocks (uniform, without replacement) to live in the slice, and a random
    allocation order for each pool (``shuffle=False``: layer-major order, as in
    a freshly filled cache)."""
    frac = cfg.slice_frac if frac is None else frac
    L = cfg.layers if layers is None else layers
    bs = cfg.block_size
    nblocks = (np.asarray(lens, dtype=np.int64) + bs - 1) // bs
    B = len(nblocks)
    maxblk = int(nblocks.max()) if B else 0
    valid = np.arange(maxblk)[None, :] < nblocks[:, None]          # [B][maxblk]
    flat_b, flat_j = np.nonzero(valid)                             # row-major (b, j)
    n_l = len(flat_b)
    in_slice = np.zeros((L, B, maxblk), dtype=bool)
    for l in range(L):
        k = _round_half_up(frac * n_l)
        pick = rng.choice(n_l, size=k, replace=False)
        in_slice[l, flat_b[pick], flat_j[pick]] = True
    all_l = np.repeat(np.arange(L), n_l)
    all_b = np.tile(flat_b, L)
    all_j = np.tile(flat_j, L)
    sl = in_slice[all_l, all_b, all_j]
    loc = np.stack([all_l[~sl], all_b[~sl], all_j[~sl]], axis=1)
    sli = np.stack([all_l[sl], all_b[sl], all_j[sl]], axis=1)
    if shuffle:
        loc = loc[rng.permutation(len(loc))]
        sli = sli[rng.permutation(len(sli))]
    return BlockPlacement(nblocks, maxblk, in_slice, loc, sli)


def round_to_16bit(x32: np.ndarray, dtype: str) -> np.ndarray:
    """float32 -> 16-bit pattern (uint16) with round-to-nearest-even."""
    x32 = np.asarray(x32, dtype=np.float32)
    if dtype == "f16":
        return x32.astype(np.float16).view(np.uint16)
    if dtype == "bf16":
        u = x32.view(np.uint32).astype(np.uint64)
        lsb = (u >> 16) & 1
        r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
        nan = np.isnan(x32)
        r[nan] = 0x7FC0
        return r
    raise ValueError(dtype)


def random_16bit(rng, shape, dtype: str) -> np.ndarray:
    """iid N(0,1) drawn in float32, stored as 16-bit patterns (uint16)."""
    return round_to_16bit(rng.standard_normal(size=shape, dtype=np.float32), dtype)


def q_values(cfg, rng, batch=None) -> np.ndarray:
    """Decode queries: 16-bit patterns, uint16 [B][Hq][D]."""
    B = cfg.batch if batch is None else batch
    return random_16bit(rng, (B, cfg.q_heads, cfg.head_dim), cfg.dtype)


NAN16 = {"f16": 0x7E00, "bf16": 0x7FC0}


def element_index(layout: int, half: int, h, t, d, kv_heads: int, block_size: int,
                  head_dim: int):
    """16-bit element index, inside one layer-block, of K (half=0) or V (half=1)
    of KV head h, token t of the block, channel d. Works on numpy arrays."""
    half_elems = block_size * kv_heads * head_dim
    if layout == LAYOUT_ATTN:
        if half == 0:
            return (h * block_size + t) * head_dim + d
        return half_elems + (h * head_dim + d) * block_size + t
    if layout == LAYOUT_NHD:
        return half * half_elems + (t * kv_heads + h) * head_dim + d
    raise ValueError(layout)


def _grid(kv_heads, block_size, head_dim):
    return np.meshgrid(np.arange(kv_heads), np.arange(block_size), np.arange(head_dim),
                       indexing="ij")


def pack_block(k16: np.ndarray, v16: np.ndarray, layout: int) -> np.ndarray:
    """Logical K, V (uint16 [Hkv][bs][D]) -> one layer-block as uint8 bytes."""
    hkv, bs, hd = k16.shape
    h, t, d = _grid(hkv, bs, hd)
    out = np.empty(2 * hkv * bs * hd, dtype=np.uint16)
    out[element_index(layout, 0, h, t, d, hkv, bs, hd)] = k16
    out[element_index(layout, 1, h, t, d, hkv, bs, hd)] = v16
    return out.view(np.uint8)


def unpack_block(block_u8: np.ndarray, layout: int, kv_heads: int, block_size: int,
                 head_dim: int):
    """One layer-block's bytes -> logical K, V (uint16 [Hkv][bs][D])."""
    e = np.ascontiguousarray(block_u8).view(np.uint16)
    h, t, d = _grid(kv_heads, block_size, head_dim)
    k = e[element_index(layout, 0, h, t, d, kv_heads, block_size, head_dim)]
    v = e[element_index(layout, 1, h, t, d, kv_heads, block_size, head_dim)]
    return k, v

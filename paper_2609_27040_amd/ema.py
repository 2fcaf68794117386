"""Thin ctypes binding of libema_slice.so -- argument marshalling only.

Each function has the C entry point's name without the ``ema_`` prefix and
passes its arguments straight through: torch tensors as their device address
(``data_ptr()``), numpy arrays as host pointers, streams as their hipStream_t.
Before a pointer goes to an entry point that launches kernels, the binding
checks that it is a contiguous GPU tensor of the expected type and at least
the size the call implies (a kernel would dereference a host address or read
past a short tensor); host-only slices take numpy arrays. Every step of the
hot path runs in the library's HIP kernels; there is no fallback. If the
library has not been built this module raises on import.
"""
import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libema_slice.so")

OK, ERR_INVAL, ERR_NOMEM, ERR_OWNER, ERR_HIP = 0, -1, -2, -3, -4
F16, BF16, F32 = 0, 1, 2
LAYOUT_ATTN, LAYOUT_NHD = 0, 1
ENGINE_KERNEL, ENGINE_DMA = 0, 1
SLAB_LAYER_MAJOR, SLAB_SLAB_MAJOR, SLAB_GROUP_MAJOR = 0, 1, 2
BORROWED = -4
POOL_LOCAL, POOL_SLICE = 0, 1
FREE, STAGING, LENDER = -1, -2, -3
CREATE_HOST_ONLY, CREATE_CHECKED, CREATE_ATTN_GRID = 1, 2, 4
DTYPES = {"f16": F16, "bf16": BF16}


class EmaError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"ema error {code}: {msg}")
        self.code = code


class KVShape(ctypes.Structure):
    _fields_ = [("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("slice_layout", ctypes.c_int32)]


class SliceInfo(ctypes.Structure):
    _fields_ = [("block_bytes", ctypes.c_int64), ("n_local", ctypes.c_int32),
                ("n_slice", ctypes.c_int32), ("lim", ctypes.c_int32),
                ("free_local", ctypes.c_int32), ("free_slice", ctypes.c_int32),
                ("device", ctypes.c_int32), ("local_base", ctypes.c_void_p),
                ("slice_base", ctypes.c_void_p)]


class ReclaimResult(ctypes.Structure):
    _fields_ = [("reclaimed", ctypes.c_int32), ("moved", ctypes.c_int32),
                ("written_back", ctypes.c_int32), ("n_victims", ctypes.c_int32),
                ("lim", ctypes.c_int32)]


class SlabCfg(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("slab_blocks", ctypes.c_int32),
                ("group", ctypes.c_int32), ("layout", ctypes.c_int32)]


class SlabInfo(ctypes.Structure):
    _fields_ = [("n_slabs", ctypes.c_int32), ("layers", ctypes.c_int32),
                ("slab_blocks", ctypes.c_int32), ("group", ctypes.c_int32),
                ("layout", ctypes.c_int32), ("borrowed", ctypes.c_int32)]


class SlabReclaimResult(ctypes.Structure):
    _fields_ = [("reclaimed", ctypes.c_int32), ("n_victims", ctypes.c_int32),
                ("released", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(python -m paper_2609_27040_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_uint32
    sig = {
        "ema_slice_create": [ctypes.POINTER(KVShape), SZ, SZ, U32, ctypes.POINTER(P)],
        "ema_slice_destroy": [P],
        "ema_slice_get_info": [P, ctypes.POINTER(SliceInfo)],
        "ema_slice_owners": [P, P, P],
        "ema_slice_alloc_blocks": [P, I32, I32, P, P],
        "ema_slice_free_blocks": [P, P, I32],
        "ema_slice_lend": [P, I32, ctypes.POINTER(I32)],
        "ema_slice_prefetch": [P, P, P, I32, P],
        "ema_slice_migrate": [P, P, P, I32, P],
        "ema_slice_writeback": [P, P, P, I32, P],
        "ema_slice_prefetch_runs": [P, P, P, P, I32, I32, P],
        "ema_kv_append": [P, P, P, P, P, I32, I32, P],
        "ema_slice_reclaim": [P, I32, P, I64, P, ctypes.POINTER(ReclaimResult), P, I32, P, P, I32],
        "ema_paged_decode_attention": [P, P, P, P, I32, I32, I32, ctypes.c_float, P, I32, P],
        "ema_paged_decode_attention_noalloc": [P, P, P, P, I32, I32, I32, ctypes.c_float, P, I32,
                                               P],
        "ema_slice_device_errors": [P, ctypes.POINTER(I32)],
        "ema_slab_init": [P, ctypes.POINTER(SlabCfg)],
        "ema_slab_get_info": [P, ctypes.POINTER(SlabInfo), P, P],
        "ema_slab_alloc": [P, I32, P, P],
        "ema_slab_free": [P, P, I32],
        "ema_slab_block_ids": [P, P, I32, I32, I32, P],
        "ema_slab_group_runs": [P, I32, I32, P, P, P, I32, ctypes.POINTER(I32)],
        "ema_slab_prefetch_group": [P, I32, I32, I32, P],
        "ema_slab_reclaim": [P, I32, P, I64, P, ctypes.POINTER(SlabReclaimResult), P, I32, P, I32],
        "ema_sched_create": [I32, I32, I64, ctypes.POINTER(P)],
        "ema_sched_destroy": [P],
        "ema_sched_place": [P, I32, I32, I32, I64, P, ctypes.POINTER(I32)],
        "ema_sched_release": [P, I32, I32, I32],
        "ema_sched_preempted": [P, I32, I32, I64],
        "ema_sched_usage": [P, I64, P, P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.ema_last_error.argtypes = []
    lib.ema_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def _check(rc):
    if rc != OK:
        raise EmaError(rc, _lib.ema_last_error().decode())


# Per handle: host-only flag, 16-bit dtype and KV heads, recorded at create,
# so that the checks below need no library call.
_HANDLES = {}


def _host_only(h):
    rec = _HANDLES.get(h)
    if rec is None:
        return slice_get_info(h)["device"] < 0
    return rec[0]


def _bad(msg):
    raise EmaError(ERR_INVAL, msg)


def _dev(t, name, dtypes, numel=0):
    """A device-array argument: a contiguous torch tensor on the GPU of one of
    ``dtypes`` with at least ``numel`` elements. The kernels read whatever the
    pointer addresses, so a host array or a short tensor is refused here."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        _bad(f"{name}: expected a GPU tensor, got {type(t).__name__}")
    if t.dtype not in dtypes:
        _bad(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        _bad(f"{name}: not contiguous")
    if t.numel() < numel:
        _bad(f"{name}: {t.numel()} elements, {numel} needed")
    return t


def _i32_dev(t, name, numel=0):
    import torch
    return _dev(t, name, (torch.int32,), numel)


def _kv16_dev(h, t, name, numel):
    """16-bit K/V/query data; when the handle's dtype is known, it must match."""
    import torch
    rec = _HANDLES.get(h)
    want = {F16: (torch.float16,), BF16: (torch.bfloat16,)}.get(rec[1]) if rec else None
    return _dev(t, name, want or (torch.float16, torch.bfloat16, torch.int16), numel)


def _ids(h, a, n, name):
    """Id list: host int32 array for a host-only slice, else a GPU int32 tensor."""
    if _host_only(h):
        a = _i32_host(a)
        if len(a) < n:
            _bad(f"{name}: {len(a)} ids, {n} needed")
        return a
    return _i32_dev(a, name, n)


def _ptr(x):
    """Device address of a torch tensor, host address of a numpy array."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _i32_host(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---- entry points ---------------------------------------------------------------

def slice_create(num_kv_heads, head_dim, block_size, dtype, slice_layout, local_bytes,
                 lent_bytes, host_only=False, checked=False, attn_grid=False):
    shape = KVShape(num_kv_heads, head_dim, block_size, DTYPES.get(dtype, dtype), slice_layout)
    h = ctypes.c_void_p()
    flags = ((CREATE_HOST_ONLY if host_only else 0) | (CREATE_CHECKED if checked else 0)
             | (CREATE_ATTN_GRID if attn_grid else 0))
    _check(_lib.ema_slice_create(ctypes.byref(shape), int(local_bytes), int(lent_bytes), flags,
                                 ctypes.byref(h)))
    _HANDLES[h.value] = (bool(host_only), shape.dtype, int(num_kv_heads))
    return h.value


def slice_destroy(h):
    _check(_lib.ema_slice_destroy(h))
    _HANDLES.pop(h, None)


def slice_get_info(h):
    info = SliceInfo()
    _check(_lib.ema_slice_get_info(h, ctypes.byref(info)))
    return {k: getattr(info, k) for k, _ in SliceInfo._fields_}


def slice_owners(h):
    info = slice_get_info(h)
    own_l = np.empty(info["n_local"], dtype=np.int32)
    own_s = np.empty(info["n_slice"], dtype=np.int32)
    _check(_lib.ema_slice_owners(h, own_l.ctypes.data, own_s.ctypes.data))
    return own_l, own_s, info["lim"]


def slice_alloc_blocks(h, pool, owners):
    owners = _i32_host(owners)
    out = np.empty(len(owners), dtype=np.int32)
    _check(_lib.ema_slice_alloc_blocks(h, pool, len(owners), owners.ctypes.data, out.ctypes.data))
    return out


def slice_free_blocks(h, ids):
    ids = _i32_host(ids)
    _check(_lib.ema_slice_free_blocks(h, ids.ctypes.data, len(ids)))


def slice_lend(h, n_blocks):
    added = ctypes.c_int32()
    _check(_lib.ema_slice_lend(h, int(n_blocks), ctypes.byref(added)))
    return added.value


def _copy_call(fn, h, src, dst, n, stream):
    n = len(src) if n is None else int(n)
    src, dst = _ids(h, src, n, "source ids"), _ids(h, dst, n, "destination ids")
    _check(fn(h, _ptr(src), _ptr(dst), n, None if _host_only(h) else _stream(stream)))


def slice_prefetch(h, block_ids, dst_block_table, n=None, stream=None):
    """block_ids, dst_block_table: int32 device tensors (numpy arrays for a
    host-only slice)."""
    _copy_call(_lib.ema_slice_prefetch, h, block_ids, dst_block_table, n, stream)


def slice_migrate(h, src_ids, dst_ids, n=None, stream=None):
    _copy_call(_lib.ema_slice_migrate, h, src_ids, dst_ids, n, stream)


def slice_prefetch_runs(h, src_first, dst_first, run_blocks, engine=0, stream=None):
    """Contiguous runs (host int arrays); engine ENGINE_KERNEL or ENGINE_DMA."""
    src_first, dst_first, run_blocks = (_i32_host(a) for a in (src_first, dst_first, run_blocks))
    info_host = slice_get_info(h)["device"] < 0
    _check(_lib.ema_slice_prefetch_runs(h, src_first.ctypes.data, dst_first.ctypes.data,
                                        run_blocks.ctypes.data, len(run_blocks), int(engine),
                                        None if info_host else _stream(stream)))


def slice_writeback(h, staging_ids, slice_ids, n=None, stream=None):
    """staging_ids, slice_ids: int32 device tensors (numpy arrays for a
    host-only slice)."""
    _copy_call(_lib.ema_slice_writeback, h, staging_ids, slice_ids, n, stream)


def kv_append(h, k_new, v_new, block_table, seq_lens, stream=None):
    """k_new, v_new [B][Hkv][D] (16-bit), block_table int32 [B][max_blocks],
    seq_lens int32 [B] counting the new token: device tensors (numpy arrays
    for a host-only slice)."""
    B = int(block_table.shape[0])
    max_blocks = int(block_table.shape[1]) if block_table.ndim == 2 else 0
    host = _host_only(h)
    if host:
        block_table, seq_lens = _i32_host(block_table), _i32_host(seq_lens)
    else:
        rec = _HANDLES.get(h)
        row = rec[2] * 128 if rec else 0          # K/V elements per sequence
        block_table = _i32_dev(block_table, "block_table", B * max_blocks)
        seq_lens = _i32_dev(seq_lens, "seq_lens", B)
        k_new = _kv16_dev(h, k_new, "k_new", B * row)
        v_new = _kv16_dev(h, v_new, "v_new", B * row)
    _check(_lib.ema_kv_append(h, _ptr(k_new), _ptr(v_new), _ptr(block_table), _ptr(seq_lens), B,
                              max_blocks, None if host else _stream(stream)))


def slice_reclaim(h, n_blocks, canon_tables=None, stream=None, caps=None):
    """canon_tables: int32 device tensor rewritten in place (None for none).
    Returns the result counts, the victims (list) and the copies made
    ("moves": int64 array [moved][2] of (source, destination) unified ids)."""
    info = slice_get_info(h)
    cap = int(caps) if caps is not None else info["n_local"] + info["n_slice"]
    res = ReclaimResult()
    victims = np.empty(max(cap, 1), dtype=np.int32)
    msrc = np.empty(max(cap, 1), dtype=np.int32)
    mdst = np.empty(max(cap, 1), dtype=np.int32)
    host_only = info["device"] < 0
    if canon_tables is not None and not host_only:
        canon_tables = _i32_dev(canon_tables, "canon_tables")
    n_entries = 0 if canon_tables is None else canon_tables.numel()
    _check(_lib.ema_slice_reclaim(h, int(n_blocks), _ptr(canon_tables), n_entries,
                                  None if host_only else _stream(stream), ctypes.byref(res),
                                  victims.ctypes.data, cap, msrc.ctypes.data, mdst.ctypes.data,
                                  cap))
    m = min(res.moved, cap)
    return {"reclaimed": res.reclaimed, "moved": res.moved, "written_back": res.written_back,
            "victims": victims[:min(res.n_victims, cap)].tolist(), "lim": res.lim,
            "moves": np.stack([msrc[:m], mdst[:m]], axis=1).astype(np.int64)}


def _attention_call(fn, h, q, block_table, seq_lens, out, scale, stream):
    import torch
    B, Hq = int(q.shape[0]), int(q.shape[1])
    max_blocks = int(block_table.shape[1]) if block_table.dim() == 2 else 0
    out_types = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
    if out.dtype not in out_types:
        _bad(f"out: dtype {out.dtype} not in {tuple(out_types)}")
    if not _host_only(h):
        q = _kv16_dev(h, q, "q", B * Hq * 128)
        block_table = _i32_dev(block_table, "block_table", B * max_blocks)
        seq_lens = _i32_dev(seq_lens, "seq_lens", B)
        out = _dev(out, "out", tuple(out_types), B * Hq * 128)
    _check(fn(h, _ptr(q), _ptr(block_table), _ptr(seq_lens), B, Hq, max_blocks, float(scale),
              _ptr(out), out_types[out.dtype], _stream(stream)))


def paged_decode_attention(h, q, block_table, seq_lens, out, scale=0.0, stream=None):
    """q [B][Hq][D] (16-bit), block_table int32 [B][max_blocks], seq_lens int32
    [B], out [B][Hq][D] of float32, float16 or bfloat16 (the output type is
    the tensor's): device tensors."""
    _attention_call(_lib.ema_paged_decode_attention, h, q, block_table, seq_lens, out, scale,
                    stream)


def paged_decode_attention_noalloc(h, q, block_table, seq_lens, out, scale=0.0, stream=None):
    """The same as paged_decode_attention, in the library's fixed per-GPU
    workspace: for callers that cannot allocate (see the C header)."""
    _attention_call(_lib.ema_paged_decode_attention_noalloc, h, q, block_table, seq_lens, out,
                    scale, stream)


def slice_device_errors(h):
    c = ctypes.c_int32()
    _check(_lib.ema_slice_device_errors(h, ctypes.byref(c)))
    return c.value


# ---- slab management of the slice --------------------------------------------------

def slab_init(h, layers, slab_blocks, group, layout=SLAB_GROUP_MAJOR):
    cfg = SlabCfg(int(layers), int(slab_blocks), int(group), int(layout))
    _check(_lib.ema_slab_init(h, ctypes.byref(cfg)))


def slab_get_info(h):
    """Shape and state: dict with n_slabs, layers, slab_blocks, group, layout,
    borrowed, slab_tag (int32 [n_slabs]) and pos_owner (int32 [n_slabs * S])."""
    info = SlabInfo()
    _check(_lib.ema_slab_get_info(h, ctypes.byref(info), None, None))
    tag = np.empty(info.n_slabs, dtype=np.int32)
    own = np.empty(info.n_slabs * info.slab_blocks, dtype=np.int32)
    _check(_lib.ema_slab_get_info(h, ctypes.byref(info), tag.ctypes.data, own.ctypes.data))
    d = {k: getattr(info, k) for k, _ in SlabInfo._fields_}
    d["slab_tag"], d["pos_owner"] = tag, own
    return d


def slab_alloc(h, owners):
    owners = _i32_host(owners)
    out = np.empty(len(owners), dtype=np.int32)
    _check(_lib.ema_slab_alloc(h, len(owners), owners.ctypes.data, out.ctypes.data))
    return out


def slab_free(h, positions):
    positions = _i32_host(positions)
    _check(_lib.ema_slab_free(h, positions.ctypes.data, len(positions)))


def slab_block_ids(h, positions, layer, staging_first=-1):
    """Unified ids of `layer`'s blocks at the positions (slice blocks, or
    their staged copies when staging_first >= 0)."""
    positions = _i32_host(positions)
    out = np.empty(len(positions), dtype=np.int32)
    _check(_lib.ema_slab_block_ids(h, positions.ctypes.data, len(positions), int(layer),
                                   int(staging_first), out.ctypes.data))
    return out


def slab_group_runs(h, group, staging_first):
    """(src_first, dst_first, run_blocks) int32 arrays of the group's swap."""
    n = ctypes.c_int32()
    _check(_lib.ema_slab_group_runs(h, int(group), int(staging_first), None, None, None, 0,
                                    ctypes.byref(n)))
    a, b, c = (np.empty(max(n.value, 1), dtype=np.int32) for _ in range(3))
    _check(_lib.ema_slab_group_runs(h, int(group), int(staging_first), a.ctypes.data,
                                    b.ctypes.data, c.ctypes.data, n.value, ctypes.byref(n)))
    return a[:n.value], b[:n.value], c[:n.value]


def slab_prefetch_group(h, group, staging_first, engine=ENGINE_KERNEL, stream=None):
    _check(_lib.ema_slab_prefetch_group(h, int(group), int(staging_first), int(engine),
                                        None if _host_only(h) else _stream(stream)))


def slab_reclaim(h, n_slabs, canon_tables=None, stream=None):
    """Returns reclaimed, n_victims, released counts plus the slabs taken and
    the victims (lists)."""
    info = slab_get_info(h)
    res = SlabReclaimResult()
    slabs = np.empty(max(info["n_slabs"], 1), dtype=np.int32)
    cap = int(info["n_slabs"] * info["slab_blocks"] + 1)
    victims = np.empty(cap, dtype=np.int32)
    host_only = _host_only(h)
    if canon_tables is not None and not host_only:
        canon_tables = _i32_dev(canon_tables, "canon_tables")
    n_entries = 0 if canon_tables is None else canon_tables.numel()
    _check(_lib.ema_slab_reclaim(h, int(n_slabs), _ptr(canon_tables), n_entries,
                                 None if host_only else _stream(stream), ctypes.byref(res),
                                 slabs.ctypes.data, len(slabs), victims.ctypes.data, cap))
    return {"reclaimed": res.reclaimed, "released": res.released,
            "slabs": slabs[:res.reclaimed].tolist(),
            "victims": victims[:min(res.n_victims, cap)].tolist()}


# ---- slice scheduling across GPUs (host policy) -------------------------------------

def sched_create(n_gpus, slice_units, cap_window=0):
    h = ctypes.c_void_p()
    _check(_lib.ema_sched_create(int(n_gpus), int(slice_units), int(cap_window), ctypes.byref(h)))
    return h.value


def sched_destroy(s):
    _check(_lib.ema_sched_destroy(s))


def sched_place(s, gpu, req, n, t=0):
    """Peers of the slices the n units went to (-1: refused)."""
    peers = np.empty(max(int(n), 1), dtype=np.int32)
    placed = ctypes.c_int32()
    _check(_lib.ema_sched_place(s, int(gpu), int(req), int(n), int(t), peers.ctypes.data,
                                ctypes.byref(placed)))
    return peers[:int(n)].tolist()


def sched_release(s, gpu, req, n):
    _check(_lib.ema_sched_release(s, int(gpu), int(req), int(n)))


def sched_preempted(s, gpu, peer, t):
    _check(_lib.ema_sched_preempted(s, int(gpu), int(peer), int(t)))


def sched_usage(s, m, t=0):
    """(use, cap) as int arrays [m][m]; cap -1 where none is active."""
    use = np.empty(m * m, dtype=np.int32)
    cap = np.empty(m * m, dtype=np.int32)
    _check(_lib.ema_sched_usage(s, int(t), use.ctypes.data, cap.ctypes.data))
    return use.reshape(m, m), cap.reshape(m, m)


class Scheduler:
    """Greedy-Least-Loaded placement over the slices of n_gpus GPUs, with
    bursty preemption caps (the sched_* calls on one handle)."""

    def __init__(self, n_gpus, slice_units, cap_window=0):
        self.m = int(n_gpus)
        self.h = sched_create(n_gpus, slice_units, cap_window)

    def place(self, gpu, req, n, t=0):
        return sched_place(self.h, gpu, req, n, t)

    def release(self, gpu, req, n):
        sched_release(self.h, gpu, req, n)

    def preempted(self, gpu, peer, t):
        sched_preempted(self.h, gpu, peer, t)

    def usage(self, t=0):
        return sched_usage(self.h, self.m, t)

    def close(self):
        if self.h:
            sched_destroy(self.h)
            self.h = None


# ---- plumbing: library-owned pools as torch tensors ---------------------------------

class _DeviceBuffer:
    def __init__(self, ptr, nbytes):
        self.__cuda_array_interface__ = {"shape": (int(nbytes),), "typestr": "|u1",
                                         "data": (int(ptr), False), "version": 3,
                                         "strides": None}


def pool_view(h, pool):
    """uint8 torch tensor [n_blocks][block_bytes] aliasing a library pool.
    Valid until slice_destroy(h)."""
    import torch
    info = slice_get_info(h)
    n = info["n_local"] if pool == POOL_LOCAL else info["n_slice"]
    base = info["local_base"] if pool == POOL_LOCAL else info["slice_base"]
    if n == 0 or not base:
        return torch.empty((0, info["block_bytes"]), dtype=torch.uint8, device="cuda")
    t = torch.as_tensor(_DeviceBuffer(base, n * info["block_bytes"]), device="cuda")
    return t.view(n, info["block_bytes"])


def last_error():
    return _lib.ema_last_error().decode()

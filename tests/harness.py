"""Test helpers: the workloads and step machinery the GPU tests share with the
bench (re-exported from ``workloads`` and the package), an oracle mirror of a
workload, the error metric and block read-back."""
import numpy as np
import torch

from paper_2609_27040_amd.kvcache import TORCH_DT            # noqa: F401
from paper_2609_27040_amd.step import (BlockedTimer, StepRunner, capture_ops,  # noqa: F401
                                       capture_step)
from workloads.synthetic import Workload                      # noqa: F401


def oracle_mirror(w):
    """An oracle slice replaying a host-filled workload's allocations, holding
    its host image."""
    import oracle
    from paper_2609_27040_amd import ema
    st = oracle.SliceOracle(w.hkv, w.D, w.bs, w.cfg.dtype, w.slice_layout,
                            w.local_view.shape[0] * w.bb, w.slice_view.shape[0] * w.bb)
    for pool, owners in w.alloc_log:
        st.alloc_blocks(pool, owners)
    own_l, own_s, lim = ema.slice_owners(w.h)
    assert np.array_equal(own_l, st.own_local) and np.array_equal(own_s, st.own_slice)
    st.local[:] = w.host_local
    st.slice[:] = w.host_slice
    return st


def owners_mirror(w):
    """An oracle slice without block data replaying a workload's allocations
    (bookkeeping only: owners, plans, tables)."""
    import oracle
    st = oracle.SliceOracle(w.hkv, w.D, w.bs, w.dtype, w.slice_layout,
                            w.local_view.shape[0] * w.bb, w.slice_view.shape[0] * w.bb,
                            with_data=False)
    for pool, owners in w.alloc_log:
        st.alloc_blocks(pool, owners)
    return st


def rel_err(out, ref):
    """max over (b, h) of ||o - ref||_inf / ||ref||_inf (rows with ref == 0: absolute)."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(out - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    den = np.where(den > 0, den, 1.0)
    return float((num / den).max()) if num.size else 0.0


def elem_err(out, ref, floor=1e-3):
    """max over elements of |o - ref| / max(|ref|, floor * row max |ref|): the
    elementwise error with a floor, reported beside the normwise gate."""
    out = np.asarray(out, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rowmax = np.abs(ref).max(axis=-1, keepdims=True)
    den = np.maximum(np.abs(ref), floor * rowmax)
    den = np.where(den > 0, den, 1.0)
    return float((np.abs(out - ref) / den).max()) if out.size else 0.0


def read_blocks(view, ids):
    """Host copies of the given blocks of a pool view (id -> bytes)."""
    ids = np.unique(np.asarray(ids, dtype=np.int64))
    ids = ids[ids >= 0]
    if not len(ids):
        return {}
    data = view[torch.from_numpy(ids).to(view.device)].cpu().numpy()
    return {int(u): data[i] for i, u in enumerate(ids)}

"""The C-ABI library loads and exports every entry point its header declares
(no compute calls: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ema_slice.h")
LIB = os.path.join(ROOT, "paper_2609_27040_amd", "lib", "libema_slice.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ema_[a-z_]+)\s*\(", text)))


def test_header_declares_the_hot_path_calls():
    names = declared_functions()
    for required in ["ema_slice_create", "ema_slice_alloc_blocks", "ema_slice_prefetch",
                     "ema_slice_reclaim", "ema_paged_decode_attention", "ema_last_error"]:
        assert required in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_binding_exposes_the_same_names():
    from paper_2609_27040_amd import ema
    for n in declared_functions():
        assert hasattr(ema, n[len("ema_"):]), n


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_every_entry_point_rejects_a_null_handle():
    """The header's error contract at the boundary itself: a NULL handle (or
    NULL out-pointer) returns EMA_ERR_INVAL with a message, before anything
    else is read -- no GPU needed."""
    from paper_2609_27040_amd import ema
    lib = ema._lib
    z = None
    calls = {
        "ema_slice_create": (z, 0, 0, 0, z),
        "ema_slice_destroy": (z,),
        "ema_slice_get_info": (z, z),
        "ema_slice_owners": (z, z, z),
        "ema_slice_alloc_blocks": (z, 0, 0, z, z),
        "ema_slice_free_blocks": (z, z, 0),
        "ema_slice_lend": (z, 0, z),
        "ema_slice_prefetch": (z, z, z, 0, z),
        "ema_slice_migrate": (z, z, z, 0, z),
        "ema_slice_writeback": (z, z, z, 0, z),
        "ema_slice_prefetch_runs": (z, z, z, z, 0, 0, z),
        "ema_kv_append": (z, z, z, z, z, 0, 0, z),
        "ema_slice_reclaim": (z, 0, z, 0, z, z, z, 0, z, z, 0),
        "ema_paged_decode_attention": (z, z, z, z, 0, 0, 0, 0.0, z, 2, z),
        "ema_paged_decode_attention_noalloc": (z, z, z, z, 0, 0, 0, 0.0, z, 2, z),
        "ema_slice_device_errors": (z, z),
        "ema_slab_init": (z, z),
        "ema_slab_get_info": (z, z, z, z),
        "ema_slab_alloc": (z, 0, z, z),
        "ema_slab_free": (z, z, 0),
        "ema_slab_block_ids": (z, z, 0, 0, 0, z),
        "ema_slab_group_runs": (z, 0, 0, z, z, z, 0, z),
        "ema_slab_prefetch_group": (z, 0, 0, 0, z),
        "ema_slab_reclaim": (z, 0, z, 0, z, z, z, 0, z, 0),
        "ema_sched_destroy": (z,),
        "ema_sched_create": (2, 1, 0, z),
        "ema_sched_place": (z, 0, 0, 0, 0, z, z),
        "ema_sched_release": (z, 0, 0, 0),
        "ema_sched_preempted": (z, 0, 1, 0),
        "ema_sched_usage": (z, 0, z, z),
    }
    declared = set(declared_functions()) - {"ema_last_error"}
    assert declared == set(calls), declared ^ set(calls)
    for name, args in calls.items():
        rc = getattr(lib, name)(*args)
        assert rc == ema.ERR_INVAL, (name, rc)
        assert lib.ema_last_error().decode(), name

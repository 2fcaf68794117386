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

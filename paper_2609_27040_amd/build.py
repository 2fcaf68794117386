"""Builds libema_slice.so (the C-ABI library) in-tree for gfx950, and
libema_calib.so beside it (HBM calibration kernels that only the benchmark
loads).

Every source is compiled with hipcc for gfx950 only, with the packed-fp32
instructions switched off in device code, then linked into
paper_2609_27040_amd/lib/. Run as ``python -m paper_2609_27040_amd.build`` or
through ``__graft_entry__.build()``.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libema_slice.so")

SOURCES = ["slice_book.cpp", "slab_book.cpp", "ema_slice.cpp", "slice_sched.cpp", "block_copy.hip",
           "paged_attention_mfma.hip", "attn_combine.hip"]
CALIB_LIB = os.path.join(LIBDIR, "libema_calib.so")
CALIB_SOURCES = ["hbm_calib.hip"]

ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-command-line-argument",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def _hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found: the ROCm toolchain is required to build")
    return exe


# Host code checked with AddressSanitizer and UBSan (device code untouched):
# `python -m paper_2609_27040_amd.build --sanitize-host` writes
# lib/host-sanitized/libema_slice.so, for host-only runs with clang's ASan
# runtime preloaded.
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-fno-omit-frame-pointer", "-g"]


def _compile(src, obj, hipcc, extra=()):
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [hipcc, *FLAGS, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r.stderr


def _link(objs, lib, hipcc, extra=()):
    tmp = lib + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)


def build(verbose=False) -> str:
    hipcc = _hipcc()
    objdir = os.path.join(LIBDIR, "obj")
    os.makedirs(objdir, exist_ok=True)
    srcs = SOURCES + CALIB_SOURCES
    objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in srcs]
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        logs = list(ex.map(lambda so: _compile(so[0], so[1], hipcc), zip(srcs, objs)))
    if verbose:
        for s, log in zip(srcs, logs):
            if log.strip():
                print(f"[{s}]\n{log}", file=sys.stderr)
    _link(objs[:len(SOURCES)], LIB, hipcc)
    _link(objs[len(SOURCES):], CALIB_LIB, hipcc)
    return LIB


def build_host_sanitized() -> str:
    """The library with its host code built under AddressSanitizer and UBSan."""
    hipcc = _hipcc()
    out_dir = os.path.join(LIBDIR, "host-sanitized")
    objdir = os.path.join(out_dir, "obj")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        list(ex.map(lambda so: _compile(so[0], so[1], hipcc, SAN_FLAGS), zip(SOURCES, objs)))
    lib = os.path.join(out_dir, "libema_slice.so")
    _link(objs, lib, hipcc, SAN_FLAGS[:4])
    return lib


if __name__ == "__main__":
    if "--sanitize-host" in sys.argv:
        print(build_host_sanitized())
    else:
        print(build(verbose="-v" in sys.argv))

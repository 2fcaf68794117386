"""Runs the host-only tests against the library built with its host code under
AddressSanitizer and UBSan (CPU only; no device code runs).

    python -m paper_2609_27040_amd.check_host_sanitized

Builds lib/host-sanitized/libema_slice.so, copies the packages and tests into
a temporary directory with that library in place of the ordinary one, and
runs the bookkeeping, slab, scheduling and ABI tests there with clang's ASan
runtime preloaded; any report stops the run. Exits with pytest's status.
"""
import glob
import os
import shutil
import subprocess
import sys
import tempfile

from paper_2609_27040_amd.build import ROOT, build_host_sanitized

TESTS = ["tests/test_host_logic.py", "tests/test_host_slab.py", "tests/test_sched.py",
         "tests/test_abi.py"]


def asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang's ASan runtime (libclang_rt.asan-x86_64.so) not found")
    return hits[-1]


def main() -> int:
    lib = build_host_sanitized()
    with tempfile.TemporaryDirectory() as tmp:
        for d in ("oracle", "synth", "workloads", "tests", "include"):
            shutil.copytree(os.path.join(ROOT, d), os.path.join(tmp, d),
                            ignore=shutil.ignore_patterns("__pycache__"))
        pkg = os.path.join(tmp, "paper_2609_27040_amd")
        shutil.copytree(os.path.join(ROOT, "paper_2609_27040_amd"), pkg,
                        ignore=shutil.ignore_patterns("__pycache__", "lib"))
        os.makedirs(os.path.join(pkg, "lib"))
        shutil.copy(lib, os.path.join(pkg, "lib", "libema_slice.so"))
        env = dict(os.environ,
                   LD_PRELOAD=asan_runtime(),
                   ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:detect_odr_violation=0",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        cmd = [sys.executable, "-m", "pytest", *TESTS, "-q", "-p", "no:cacheprovider"]
        return subprocess.run(cmd, cwd=tmp, env=env).returncode


if __name__ == "__main__":
    sys.exit(main())

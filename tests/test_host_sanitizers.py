"""libleap's host layer under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).

The library is built into a temporary directory with the sanitizers applied
to its host code only (-Xarch_host before each flag; the gfx950 device code
is compiled as in the product), and the C-ABI tests -- argument checks,
status codes, workspace sizes, symbol exports, none of which launches a
kernel -- run against that build in a child process with clang's ASan
runtime preloaded.  The run must be clean."""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

import pytest

from paper_2608_01804_amd import _build

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

_CHILD = """
import sys
sys.path.insert(0, {root!r})
import paper_2608_01804_amd.leap as L
L.LIB_PATH = {lib!r}
import pytest
sys.exit(pytest.main(["-x", "-q", "-s", "-p", "no:cacheprovider", {tests!r}]))
"""


def _asan_runtime() -> str | None:
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return found[-1] if found else None


def test_abi_clean_under_host_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None or shutil.which("nm") is None:
        pytest.skip("clang's ASan runtime or nm is not available")
    lib = str(tmp_path / "libleap.so")
    flags = [f for f in _build.HIPCC_FLAGS if f != "-O3"] + [
        "-O1", "-g",
        "-Xarch_host", "-fsanitize=address",
        "-Xarch_host", "-fsanitize=undefined",
        "-Xarch_host", "-fno-omit-frame-pointer"]
    subprocess.run([_build.hipcc_path(), *flags, "-I" + _build.INCLUDE_DIR, "-o", lib,
                    *_build.sources()], check=True, capture_output=True, text=True)
    # the build really carries the instrumentation
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_" in syms and "__ubsan_" in syms
    env = dict(os.environ, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:detect_odr_violation=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = _CHILD.format(root=ROOT, lib=lib, tests=os.path.join(HERE, "test_abi.py"))
    r = subprocess.run([sys.executable, "-c", code], cwd=str(tmp_path), env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "passed" in r.stdout

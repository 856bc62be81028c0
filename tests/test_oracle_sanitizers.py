"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only, host code built with gcc).

A copy of the oracle is built with both sanitizers in a temporary directory
and the pin files that exercise its C entry points run against it in a child
process (Python is not instrumented, so the child preloads gcc's ASan
runtime).  Any out-of-bounds access, use after free or undefined operation
in the oracle halts the child with a sanitizer report; the test requires a
clean run."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
# the pin files whose oracle calls go through the C library
PIN_FILES = [os.path.join(HERE, f) for f in (
    "test_oracle_rank.py", "test_oracle_gate_discount.py", "test_oracle_grpo.py",
    "test_oracle_rollout_stats.py", "test_oracle_properties.py")]


def _gcc_runtime(name: str) -> str | None:
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def _sanitized_copy(dest: str, plant=None) -> str:
    """The oracle copied into dest and built with both sanitizers; plant,
    if given, is one (original, replacement) edit of the C source."""
    pkg = os.path.join(dest, "oracle")
    os.makedirs(pkg)
    for f in ("leap_oracle.c", "__init__.py"):
        text = open(os.path.join(ROOT, "oracle", f)).read()
        if plant and f == "leap_oracle.c":
            assert text.count(plant[0]) == 1
            text = text.replace(*plant)
        open(os.path.join(pkg, f), "w").write(text)
    cmd = ["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
           "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-o", os.path.join(pkg, "liboracle.so"),
           os.path.join(pkg, "leap_oracle.c"), "-lm"]
    subprocess.run(cmd, check=True)
    return dest


def _run(dest: str, files) -> subprocess.CompletedProcess:
    env = dict(os.environ, PYTHONPATH=dest, OMP_NUM_THREADS="2",
               LD_PRELOAD=_gcc_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:detect_odr_violation=0:"
                            "alloc_dealloc_mismatch=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # -s: a sanitizer report goes to fd 2 and the child exits at once, so
    # pytest must not be capturing that descriptor
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider",
                           "--import-mode=append", "-m", "not gpu", *files],
                          cwd=dest, env=env, capture_output=True, text=True, timeout=900)


@pytest.fixture(scope="module", autouse=True)
def _need_asan():
    if shutil.which("gcc") is None or _gcc_runtime("libasan.so") is None:
        pytest.skip("gcc with the ASan runtime is not available")


def test_oracle_pins_clean_under_asan_and_ubsan(tmp_path):
    r = _run(_sanitized_copy(str(tmp_path)), PIN_FILES)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "passed" in r.stdout


def test_planted_overread_is_caught(tmp_path):
    # Control: the gate reading one byte past each group (past the array for
    # the last group) must halt the child with an ASan report, which shows
    # that the sanitized copy is the one the pins load.
    plant = ("if (first_turn_pass[g * (int64_t)G + i] == 0) nf += 1;",
             "if (first_turn_pass[g * (int64_t)G + i + 1] == 0) nf += 1;")
    r = _run(_sanitized_copy(str(tmp_path), plant),
             [os.path.join(HERE, "test_oracle_gate_discount.py")])
    out = r.stdout + r.stderr
    assert r.returncode != 0
    assert "AddressSanitizer" in out and "heap-buffer-overflow" in out, out[-3000:]

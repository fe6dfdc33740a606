"""The oracle's C under AddressSanitizer and UndefinedBehaviorSanitizer, on
the CPU.  A sanitized build of oracle/gva_oracle.c runs every oracle pin in
a child process (the ASan runtime preloaded, leak checks off: the Python
interpreter itself is not instrumented), and a copy with a planted heap
overflow must be caught, so the sanitizers are known to be live."""

import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
GCC_SAN = ["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _asan_runtime():
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.fixture(scope="module")
def runtime():
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("a preload is already set in this environment; the ASan runtime must come first")
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("gcc's ASan runtime is not installed")
    return rt


def _build(src: str, lib: str):
    subprocess.run(GCC_SAN + ["-o", lib, src, "-lm"], check=True)


def _run_pins(lib: str, rt: str):
    env = dict(os.environ, GVA_ORACLE_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    cmd = [sys.executable, "-m", "pytest", os.path.join(HERE, "test_oracle_pins.py"), "-x", "-q", "-s",
           "-p", "no:cacheprovider"]
    return subprocess.run(cmd, env=env, capture_output=True, text=True, timeout=900, cwd=ROOT)


def test_oracle_pins_pass_under_sanitizers(tmp_path, runtime):
    lib = str(tmp_path / "libgva_oracle_san.so")
    _build(oracle._SRC, lib)
    res = _run_pins(lib, runtime)
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert "passed" in res.stdout and "runtime error" not in res.stderr


def test_sanitizers_catch_a_planted_overflow(tmp_path, runtime):
    # the decode's score buffer one element short: its last store overflows
    src = open(oracle._SRC).read()
    good = "double* s = (double*)malloc(sizeof(double) * (size_t)n);"
    assert src.count(good) == 1
    bad = tmp_path / "gva_oracle_overflow.c"
    bad.write_text(src.replace(good, "double* s = (double*)malloc(sizeof(double) * (size_t)(n - 1));"))
    lib = str(tmp_path / "libgva_oracle_overflow.so")
    _build(str(bad), lib)
    res = _run_pins(lib, runtime)
    assert res.returncode != 0
    assert "AddressSanitizer" in res.stderr

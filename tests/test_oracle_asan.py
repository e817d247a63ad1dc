"""The oracle's C code under AddressSanitizer (host code only): a private build of
oracle/kmq_oracle.c with -fsanitize=address runs every oracle pin in a child
process, so that an out-of-bounds access or a use after free in the checker, or a
caller that hands it a buffer too small for the sizes it passes, stops the run
instead of corrupting memory silently."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    try:
        path = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                              check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_under_asan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    so = tmp_path / "libkmq_oracle_asan.so"
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-omit-frame-pointer",
                           "-fsanitize=address", "-fPIC", "-shared", "-I", os.path.join(ROOT, "oracle"),
                           "-o", str(so), os.path.join(ROOT, "oracle", "kmq_oracle.c"), "-lm"])
    env = dict(os.environ, LD_PRELOAD=rt, KMQ_ORACLE_LIB=str(so), OMP_NUM_THREADS="2",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"), "-x", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr, tail
    assert " passed" in r.stdout, tail

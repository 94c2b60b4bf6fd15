"""The oracle's pins once more, with tco.c built under the address and
undefined-behaviour sanitizers (any report is fatal): out-of-bounds reads or
writes, use after free, signed overflow, shifts out of range and the like in
the oracle would fail here even where its results happen to come out right.
Runs the oracle test files in a child process that preloads the sanitizer
runtime (the interpreter itself is not instrumented)."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime():
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    p = r.stdout.strip()
    return p if r.returncode == 0 and os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.skipif(bool(os.environ.get("LD_PRELOAD")), reason="another library is already preloaded")
def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan = _runtime()
    if asan is None:
        pytest.skip("gcc's address sanitizer runtime is not installed")
    sys.path.insert(0, ROOT)
    try:
        from oracle import build as ob
    finally:
        sys.path.pop(0)
    lib = ob.build(sanitize=True, out=str(tmp_path / "liboracle_san.so"))
    files = sorted(glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py")))
    assert len(files) >= 7
    env = dict(os.environ, TCO_LIB=lib, LD_PRELOAD=asan, OMP_NUM_THREADS="2",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *files],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " passed" in out

"""The oracle's pins once more with the oracle built under AddressSanitizer and
UndefinedBehaviorSanitizer: any out-of-bounds access, use after free, signed
overflow or misaligned access in its C code aborts the run (CPU only)."""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _runtime(name):
    out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(_runtime("libasan.so") is None, reason="gcc's AddressSanitizer runtime is not installed")
def test_oracle_pins_under_sanitizers(tmp_path):
    so = oracle.build_sanitized(str(tmp_path / "liboracle_asan.so"))
    env = dict(os.environ, ORACLE_LIB=so, LD_PRELOAD=_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1",
               OMP_NUM_THREADS="4")
    tests = [os.path.join(HERE, f) for f in
             ("test_oracle_pins.py", "test_oracle_adaptive_pins.py", "test_oracle_conv_pins.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
                        *tests], cwd=os.path.dirname(HERE), env=env, capture_output=True, text=True,
                       timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error:" not in r.stderr, tail

"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

oracle/spot_oracle.c is built with -fsanitize=address,undefined (any
undefined-behaviour report aborts) and the oracle's pin tests and the input
generator tests run against that build in a child Python process with the
sanitizer runtimes preloaded.  An out-of-bounds access, use after free,
signed overflow or misaligned load in the oracle fails this test.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "spot_oracle.c")


def runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(runtime("libasan.so") is None or runtime("libubsan.so") is None,
                    reason="gcc sanitizer runtimes not installed")
def test_oracle_pins_under_sanitizers(tmp_path):
    so = str(tmp_path / "liboracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-std=c11",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-shared", "-fPIC", "-o", so, SRC, "-lm"], check=True)
    env = dict(os.environ)
    env.update({
        "SPOT_ORACLE_SO": so,
        "LD_PRELOAD": runtime("libasan.so") + ":" + runtime("libubsan.so"),
        # the interpreter's own allocations are not the oracle's leaks
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "OMP_NUM_THREADS": "2",
    })
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_synth.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail

"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

oracle.c is rebuilt in a temporary directory with -fsanitize=address,undefined
(any finding aborts), and the oracle's pin suites run against that build in a
child process with the sanitizer runtimes preloaded.  The pins exercise every
oracle routine, including empty pools, padding and the capacity branches."""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = ["test_oracle.py", "test_oracle_verify.py", "test_oracle_lexical.py", "test_oracle_recycle.py",
        "test_oracle_fp8.py"]


def _runtime(name):
    out = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(_runtime("libasan.so") is None, reason="gcc's AddressSanitizer runtime is not installed")
def test_oracle_pins_clean_under_asan_ubsan():
    with tempfile.TemporaryDirectory() as td:
        so = os.path.join(td, "liboracle_san.so")
        subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fno-fast-math", "-ffp-contract=off",
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fPIC", "-shared",
                        "-std=c11", "-o", so, SRC, "-lm"], check=True)
        env = dict(os.environ, OILBIRD_ORACLE_LIB=so,
                   LD_PRELOAD=" ".join(x for x in (_runtime("libasan.so"), _runtime("libubsan.so")) if x),
                   ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider"] +
                           [os.path.join(ROOT, "tests", f) for f in PINS],
                           env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
        tail = (r.stdout + r.stderr)[-3000:]
        assert r.returncode == 0, tail
        assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail

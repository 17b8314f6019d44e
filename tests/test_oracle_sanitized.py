"""The oracle's pins under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle's C is built a second time with ``-fsanitize=address,undefined``
(gcc, host code) and the whole pin suite runs against that build in a child
process with the sanitizer runtimes preloaded: an out-of-bounds access, a
use of freed memory, a signed overflow, a misaligned access or an invalid
shift anywhere the pins drive the oracle aborts the child and fails this
test."""
import os
import subprocess
import sys

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_pins_pass_under_sanitizers():
    env = oracle.sanitizer_env()
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
           os.path.join(ROOT, "tests", "test_oracle_pins.py")]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr, tail
    assert "runtime error" not in r.stderr, tail


def test_the_sanitized_harness_catches_a_planted_error(tmp_path):
    """The same flags and environment turn a heap read one past the end into
    an abort (so a passing run above means the pins really ran checked)."""
    src = tmp_path / "oob.c"
    src.write_text("#include <stdlib.h>\n"
                   "int oob(int n) { int *a = malloc(n * sizeof(int)); for (int i = 0; i < n; ++i) a[i] = i;\n"
                   "  int s = a[n]; free(a); return s; }\n")
    lib = tmp_path / "liboob.so"
    subprocess.run(["gcc", *oracle.SANITIZE_FLAGS, "-shared", "-fPIC", "-o", str(lib), str(src)], check=True)
    code = f"import ctypes; ctypes.CDLL({str(lib)!r}).oob(8)"
    r = subprocess.run([sys.executable, "-c", code], env=oracle.sanitizer_env(), capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, r.stderr[-2000:]

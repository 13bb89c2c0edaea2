"""The oracle's pins under AddressSanitizer and UndefinedBehaviorSanitizer:
the oracle is rebuilt with -fsanitize=address,undefined and its pin tests run
in a child process that preloads the gcc runtimes (any report aborts it)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_pins_under_asan_ubsan():
    import oracle
    try:
        oracle.build(force=True, sanitize=True)
        env = oracle.sanitize_env()
    except (OSError, subprocess.CalledProcessError) as e:  # no gcc sanitizer runtime here
        pytest.skip(f"sanitizer build unavailable: {e}")
    # the runtime must really be active in the child
    probe = "import ctypes; ctypes.CDLL(None).__asan_init; import oracle; print(oracle.lib()._name)"
    out = subprocess.check_output([sys.executable, "-c", probe], env=env, cwd=ROOT, text=True)
    assert out.strip().endswith("libsparsepr_oracle_san.so")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_pins.py", "tests/test_oracle_diagnostics.py"],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]

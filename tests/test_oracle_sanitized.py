"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer runs
every pin cleanly (CPU only; a separate process preloads the sanitizer
runtime, since the Python interpreter itself is not instrumented)."""
import os
import subprocess
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SCRIPT = r"""
import sys
sys.path.insert(0, %(repo)r)
sys.path.insert(0, %(tests)r)
import oracle, oracle_pins
o = oracle.variant(["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                    "-fno-omit-frame-pointer", "-O1"], "sanitized")
for pin in oracle_pins.ALL_PINS:
    pin(o)
print("sanitized oracle: %%d pins passed" %% len(oracle_pins.ALL_PINS))
"""


def _libasan():
    try:
        out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_oracle_pins_under_sanitizers():
    asan = _libasan()
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "4"
    code = SCRIPT % {"repo": REPO, "tests": os.path.join(REPO, "tests")}
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "pins passed" in r.stdout

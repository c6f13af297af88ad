"""The host side of librfq (the C-ABI argument validation and size
arithmetic in front of every kernel launch) built with AddressSanitizer and
UndefinedBehaviorSanitizer runs the ABI tests cleanly.  CPU only: a separate
process preloads the sanitizer runtime (the Python interpreter itself is not
instrumented), and only host code is instrumented."""
import glob
import os
import subprocess
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(REPO, "paper_2608_26581_amd", "librfq_sanitized.so")

HOST_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-sanitize-recover=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-shared-libasan"]

SCRIPT = r"""
import sys
sys.path.insert(0, %(repo)r)
sys.path.insert(0, %(tests)r)
import paper_2608_26581_amd as pkg
from paper_2608_26581_amd import rfq as binding
binding.LIB_PATH = pkg.LIB_PATH = %(lib)r
import pytest
sys.exit(pytest.main([%(abi)r, "-q", "-p", "no:cacheprovider", "-m", "not gpu"]))
"""


def _runtime():
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return hits[0] if hits else None


def test_abi_tests_under_sanitizers():
    import torch
    if torch.cuda.is_available():
        pytest.skip("host-side check: runs where no GPU is present")
    rt = _runtime()
    if rt is None:
        pytest.skip("no clang AddressSanitizer runtime here")
    from paper_2608_26581_amd import build as rfq_build
    rfq_build.build(extra_flags=HOST_FLAGS, out=LIB)
    env = dict(os.environ)
    env["LD_PRELOAD"] = rt + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    code = SCRIPT % {"repo": REPO, "tests": os.path.join(REPO, "tests"), "lib": LIB,
                     "abi": os.path.join(REPO, "tests", "test_abi.py")}
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=900, cwd=REPO)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-4000:])
    assert " passed" in r.stdout and "failed" not in r.stdout

"""Host-side logic checked on the CPU: the product path never reaches the
oracle, bench.py's traffic record is honoured only while the kernel sources
it was measured on are unchanged, and bench.py refuses step counts it
cannot time."""
import json
import os
import re
import shutil

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(REPO, "paper_2608_26581_amd")


def test_product_path_does_not_use_the_oracle():
    for root, _, files in os.walk(PKG):
        for f in files:
            if f.endswith((".py", ".hip", ".h")):
                text = open(os.path.join(root, f)).read()
                # No import, load or call of the oracle (prose may name it).
                assert not re.search(r"import\s+oracle|from\s+oracle|oracle\.[A-Za-z_]|rfq_oracle|"
                                     r"oracle_[a-z]", text), os.path.join(root, f)


def test_binding_has_no_cpu_fallback():
    text = open(os.path.join(PKG, "rfq.py")).read()
    # Every public entry point ends in a library call; none computes with torch.
    assert "torch.matmul" not in text and "numpy" not in text


def _copy_repo_subset(tmp_path, rec):
    root = tmp_path / "r"
    (root / "profiles").mkdir(parents=True)
    for rel in rec["sources"]:
        dst = root / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(REPO, rel), dst)
    shutil.copy(os.path.join(REPO, "profiles", "rfq_gemm_large_qwen_hbm_counters.md"),
                root / "profiles" / "rfq_gemm_large_qwen_hbm_counters.md")
    return root


def test_traffic_record_follows_the_sources(tmp_path, monkeypatch):
    import bench
    rec = bench.recorded_traffic()
    if rec is None:
        pytest.skip("the committed record does not match the current sources")
    assert rec["read_bytes"] > 0 and rec["write_bytes"] > 0
    root = _copy_repo_subset(tmp_path, rec)
    monkeypatch.setattr(bench, "REPO", str(root))
    path = str(root / "profiles" / "rfq_gemm_large_qwen_hbm_counters.md")
    assert bench.recorded_traffic(path) == rec
    # Any change to a listed source voids the record.
    first = sorted(rec["sources"])[0]
    with open(root / first, "a") as f:
        f.write("\n// changed\n")
    assert bench.recorded_traffic(path) is None


@pytest.mark.parametrize("args", [["--steps", "0"], ["--steps", "-3"], ["--warmup", "-1"]])
def test_bench_rejects_step_counts_it_cannot_time(args):
    """bench.py times at least one step (its product events bracket every
    fourth timed step, starting with the first) and needs a warm-up count of
    zero or more; it says so and exits before touching a GPU."""
    import subprocess
    import sys
    res = subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), *args],
                         capture_output=True, text=True, timeout=60)
    assert res.returncode == 2
    assert "--steps must be at least 1" in res.stderr

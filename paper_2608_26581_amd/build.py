"""Builds librfq.so (the HIP kernels and the C ABI) in-tree for gfx950."""
import glob
import os
import subprocess

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
REPO_DIR = os.path.dirname(PKG_DIR)
LIB_PATH = os.path.join(PKG_DIR, "librfq.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# -packed-fp32-ops: no packed fp32 VALU instructions are generated.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG_DIR, "csrc", "*.hip")))


def build(verbose=False, extra_flags=(), out=LIB_PATH):
    """Compile every source under csrc/ into librfq.so, or into `out` with
    extra compiler flags (always recompiles)."""
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra_flags,
           "-I", os.path.join(REPO_DIR, "include"),
           "-I", os.path.join(PKG_DIR, "csrc"),
           *sources(), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError("librfq build failed:\n" + err)
    if verbose and err.strip():
        print(err)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))

"""Build libhsap.so for gfx950 in-tree with hipcc.

Every translation unit under ``csrc/`` is compiled (``.hip`` as HIP device +
host code, ``.cpp`` as host C++), then linked into ``libhsap.so`` next to this
file.  Always rebuilds (a stale library is never reused); object files go to
``_build/`` at the repository root.

    python -m paper_2606_30460_amd.build
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG_DIR, "libhsap.so")
ARCH = "gfx950"

# Device-code flags: packed fp32 VALU instructions are disabled on purpose
# (hipcc's host pass warns that it does not know the feature; harmless).
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
    "-munsafe-fp-atomics",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]
# Per-source additions.  The forward kernels never see a NaN (finite bf16 inputs; masked scores are
# -inf, which stays honoured): without NaN semantics the compiler drops the canonicalising maxes
# around the row maximum (5 VALU instructions per 64-key step; c4 forward +0.6-0.8 % on one box).
EXTRA_FLAGS = {"attn_fwd.hip": ["-fno-honor-nans"]}


def _hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    if src.endswith(".hip"):
        cmd = [_hipcc(), *HIP_FLAGS, *EXTRA_FLAGS.get(os.path.basename(src), []), "-c", src, "-o", obj]
    else:
        cmd = [shutil.which("g++") or "g++", *CXX_FLAGS, "-I/opt/rocm/include", "-c", src, "-o", obj]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s\n%s" % (" ".join(cmd), proc.stdout, proc.stderr))
    return obj


def build(verbose: bool = False) -> str:
    """Compile and link libhsap.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    sources = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))
    jobs = min(len(sources), int(os.environ.get("MAX_JOBS", "8")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile, sources))
    tmp = LIB_PATH + ".tmp"
    cmd = [_hipcc(), "-shared", "-fPIC", "--offload-arch=" + ARCH, *objs, "-o", tmp]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("link failed: %s\n%s\n%s" % (" ".join(cmd), proc.stdout, proc.stderr))
    os.replace(tmp, LIB_PATH)
    if verbose:
        print("built", LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

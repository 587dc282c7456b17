"""Build librk.so (the HIP library behind include/rk.h) for gfx950, in-tree.

    python -m paper_2608_08684_amd.build        # or __graft_entry__.build()

Device code is compiled with packed-fp32 instructions disabled; host files are
plain C++17.  The shared object lands next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "librk.so")
BUILD_DIR = os.path.join(ROOT, "_build")

SOURCES = ["api.cpp", "budgets.cpp", "elementwise.hip", "gemm.hip", "attention.hip", "lm_kl.hip", "snapkv.hip",
           "scratch.hip"]
ARCH = "gfx950"
# Per-file code-generation options.  Attention keeps its MFMA accumulators in
# ordinary VGPRs: its softmax reads and rescales them every tile, and the AGPR
# form would copy them across register files around every MFMA.  Its scores are
# never NaN (masked keys are -inf), so max reductions need no NaN canonicalising.
EXTRA = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"]}


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found")
    return p


def _flags(src: str):
    common = ["-O3", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function",
              "-Wno-unused-variable", "-Wno-unused-but-set-variable"]
    if src.endswith(".hip"):
        return common + [f"--offload-arch={ARCH}", "-x", "hip", "-Xclang", "-target-feature", "-Xclang",
                         "-packed-fp32-ops", "-ffp-contract=fast"] + EXTRA.get(src, [])
    return common + ["-x", "c++", "-D__HIP_PLATFORM_AMD__"]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, src + ".o")
    cmd = [hipcc(), "-c", os.path.join(CSRC, src), "-o", obj] + _flags(src)
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("linking librk.so failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

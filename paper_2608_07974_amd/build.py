"""Build libzl.so (HIP kernels for gfx950 + the C-ABI host code) in-tree.

Usage: python -m paper_2608_07974_amd.build [--jobs N]
Each source compiles to an object under _build/ in parallel, then links.
"""
import argparse
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libzl.so")
BUILD = os.path.join(ROOT, "_build")
SOURCES = ["gemm.hip", "attention.hip", "attention_mfma.hip", "rowops.hip",
           "objective.hip", "optim.hip", "zl.cpp", "runtime.cpp", "noalloc.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-Wno-unused-command-line-argument",
         # a requested unroll that fails leaves register arrays indexed at run
         # time (scratch memory): make it an error
         "-Werror=pass-failed"]


# Hot kernels must not use scratch memory: a spill or an argument block
# copied to scratch costs far more than any schedule gains (checked from the
# compiler's resource-usage remarks).
NO_SCRATCH = {"gemm.hip": "gemm_dma_kernel", "attention_mfma.hip": "attn_"}


def _scratch_users(stderr, pattern):
    bad, name = [], None
    for line in stderr.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "ScratchSize [bytes/lane]:" in line and name and pattern in name:
            size = int(line.split("ScratchSize [bytes/lane]:")[1].split()[0])
            if size:
                bad.append((name, size))
    return bad


def _compile(src):
    obj = os.path.join(BUILD, src + ".o")
    extra = ["-Rpass-analysis=kernel-resource-usage"] if src in NO_SCRATCH else []
    cmd = [HIPCC] + FLAGS + extra + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{r.stderr}")
    if src in NO_SCRATCH:
        bad = _scratch_users(r.stderr, NO_SCRATCH[src])
        if bad:
            raise RuntimeError(f"{src}: hot kernels use scratch memory: {bad}")
    return obj


def build(jobs=None, verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(OUT_DIR, exist_ok=True)
    jobs = jobs or min(len(SOURCES), max(1, (os.cpu_count() or 4)))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    a = ap.parse_args()
    build(a.jobs, verbose=True)
    sys.exit(0)

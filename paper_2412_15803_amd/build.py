"""Build the HIP library in-tree for gfx950.

    python -m paper_2412_15803_amd.build

compiles every csrc/*.hip with hipcc (one process per file, in parallel) and
links paper_2412_15803_amd/lib/libwq.so.  The output is replaced atomically.
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_DIR = os.path.join(PKG, "lib")
LIB_PATH = os.path.join(LIB_DIR, "libwq.so")
ARCH = "gfx950"

COMPILE_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-command-line-argument",
    # Keep the compiler from forming packed-fp32 instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # The ticket claims are issued by one lane on purpose and their results
    # read much later; the wave-level atomic rewrite would wait right away.
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-I", INCLUDE,
    "-I", CSRC,
]


# Sources the batch-1 decode-step kernel and its launch plan are built from.
STEP_KERNEL_SOURCES = ("wq_api.hip", "wq_decode.hip", "wq_device.h", "wq_internal.h", "wq_limits.h", "wq_plan.h",
                       "wq_plan.hip")


def source_hash(names=STEP_KERNEL_SOURCES) -> str:
    """Short hash of the named HIP sources under csrc/; profile summaries
    record it so that figures taken from an older kernel are recognised as
    stale."""
    import hashlib

    h = hashlib.sha256()
    files = sorted(os.path.join(CSRC, n) for n in names)
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def _run(cmd, verbose):
    if verbose:
        print("+", " ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{res.stdout}")
    if verbose and res.stdout.strip():
        print(res.stdout, flush=True)


def build(verbose: bool = True) -> str:
    """Compile and link the library; returns the path of the built .so."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    os.makedirs(LIB_DIR, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not sources:
        raise RuntimeError(f"no HIP sources under {CSRC}")
    objects = [os.path.join(BUILD_DIR, os.path.basename(s)[:-4] + ".o") for s in sources]
    jobs = [[hipcc, *COMPILE_FLAGS, "-c", s, "-o", o] for s, o in zip(sources, objects)]
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), 8)) as ex:
        for fut in [ex.submit(_run, j, verbose) for j in jobs]:
            fut.result()
    tmp = LIB_PATH + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objects], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)

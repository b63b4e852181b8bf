"""Build of libwq.so with AddressSanitizer on its host code only (the device
code is compiled as usual), for the host-sanitizer test.

The host passes of every csrc/*.hip get the sanitizer through -Xarch_host;
the library links the shared ASan runtime, which the test preloads into a
child Python process."""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess

from paper_2412_15803_amd import build as B

HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """Path of clang's shared ASan runtime next to hipcc's compiler."""
    out = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True).stdout.strip()
    if not os.path.isabs(out) or not os.path.exists(out):
        cands = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        if not cands:
            raise RuntimeError("clang's shared ASan runtime not found")
        out = cands[0]
    return out


def build_asan(out_dir: str) -> str:
    """Compile every csrc/*.hip with host-side ASan into out_dir; return the
    path of the linked library."""
    hipcc = B._hipcc()
    os.makedirs(out_dir, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(B.CSRC, "*.hip")))
    objects = [os.path.join(out_dir, os.path.basename(s)[:-4] + ".o") for s in sources]
    flags = [f for f in B.COMPILE_FLAGS if f != "-O3"] + ["-O1", "-g"] + HOST_SANITIZE
    jobs = [[hipcc, *flags, "-c", s, "-o", o] for s, o in zip(sources, objects)]
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), 8)) as ex:
        for fut in [ex.submit(B._run, j, False) for j in jobs]:
            fut.result()
    lib = os.path.join(out_dir, "libwq_asan.so")
    B._run([hipcc, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address",
            "-shared-libsan", "-o", lib, *objects], False)
    return lib

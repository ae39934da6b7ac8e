"""Build libm2c.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2410_14740_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libm2c.so")
BUILD_DIR = os.path.join(ROOT, "_build", "m2c")
ARCH = os.environ.get("M2C_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the first kernel arguments arrive in SGPRs at wave launch (gfx950), which
    # saves a dependent scalar load at the start of every workgroup; the code
    # keeps a loading prologue for runtimes that do not preload
    "-mllvm", "-amdgpu-kernarg-preload-count=16",
    "-Wall", "-Wno-unused-result", f"-I{os.path.join(ROOT, 'include')}",
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def source_id() -> str:
    """SHA-256 (first 16 hex digits) over every file the library is built
    from: the kernels, their headers and the public header. The build bakes
    it into the library (m2c_build_id), so a loader can tell a library built
    from other sources."""
    files = sorted(glob.glob(os.path.join(CSRC, "*")) +
                   glob.glob(os.path.join(ROOT, "include", "*.h")))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(BUILD_DIR, os.path.basename(s) + ".o") for s in srcs]

    sid = source_id()

    def compile_one(pair):
        src, obj = pair
        cmd = [HIPCC, *FLAGS, f'-DM2C_SOURCE_ID="{sid}"', "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {os.path.basename(src)}:\n{r.stdout}{r.stderr}")
        noise = "is not a recognized feature for this target"
        msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
        if verbose and msgs.strip():
            print(msgs, file=sys.stderr)
        return obj

    workers = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")), 16)
    with cf.ThreadPoolExecutor(max_workers=max(1, workers)) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    tmp = OUT + f".tmp{os.getpid()}"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))

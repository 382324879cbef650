"""Builds the gfx950 HIP library libpbg.so in-tree with hipcc.

Every source under csrc/ (HIP kernels and the host runtime behind the C ABI
of include/pbg.h) is compiled for gfx950 and linked into lib/libpbg.so.  The
library depends on the HIP runtime only (no PyTorch symbols).
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_DIR = os.path.join(HERE, "lib")
LIB = os.path.join(LIB_DIR, "libpbg.so")
OBJ_DIR = os.path.join(HERE, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
    "-I", INCLUDE, "-I", CSRC,
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-instruction accumulators in ordinary VGPRs: the loss epilogues
    # then read them in place instead of copying 64 AGPRs out first
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wno-unused-result",
]


def sources():
    out = []
    for name in sorted(os.listdir(CSRC)):
        if name.endswith(".hip") or name.endswith(".cpp"):
            out.append(os.path.join(CSRC, name))
    return out


def _compile(src: str) -> str:
    obj = os.path.join(OBJ_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-6000:]}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    os.makedirs(LIB_DIR, exist_ok=True)
    srcs = sources()
    jobs = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    # every symbol must resolve at link time (a missing definition fails the build, not the load)
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,--no-undefined", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-6000:]}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_asan(verbose: bool = False) -> str:
    """A copy of the library whose host code (the *.cpp runtime) is built with
    AddressSanitizer, for host-side tests of the ABI's error paths; the
    kernels are the regular objects (device code is never instrumented).  The
    AddressSanitizer runtime comes from the executable that loads it.
    Returns the path of _build/asan/libpbg_asan.so."""
    if not all(os.path.exists(os.path.join(OBJ_DIR, os.path.basename(f) + ".o"))
               for f in sources() if f.endswith(".hip")):
        build(verbose=False)
    out_dir = os.path.join(OBJ_DIR, "asan")
    os.makedirs(out_dir, exist_ok=True)
    host = [f for f in sources() if f.endswith(".cpp")]
    # host code only: each sanitizer flag applies to the host pass
    asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]

    def compile_host(src):
        obj = os.path.join(out_dir, os.path.basename(src) + ".o")
        r = subprocess.run([HIPCC, *COMMON, *asan, "-x", "hip", "-c", src, "-o", obj], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr[-6000:]}")
        return obj

    jobs = min(len(host), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_host, host))
    kern = [os.path.join(OBJ_DIR, os.path.basename(f) + ".o") for f in sources() if f.endswith(".hip")]
    lib = os.path.join(out_dir, "libpbg_asan.so")
    r = subprocess.run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", lib, *objs, *kern],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-6000:]}")
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build()
    sys.exit(0)

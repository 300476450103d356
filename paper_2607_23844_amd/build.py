"""Build the OmniCache HIP library (liboc.so) for gfx950, in-tree.

    python -m paper_2607_23844_amd.build          # liboc.so
    python -m paper_2607_23844_amd.build asan     # liboc_asan.so

Every source is compiled with hipcc for gfx950 only; packed fp32 vector
instructions are disabled for device code.  Objects go to _build/, the
shared library next to this file.  The asan variant instruments the host
code only (argument checks, planning, the schedule, the timer) with
AddressSanitizer; device code is built as usual.  It is for CPU-side tests:
load it with the sanitizer runtime preloaded (OC_LIBRARY names it).
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
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liboc.so")
BUILD_ASAN = os.path.join(ROOT, "_build_asan")
LIB_ASAN = os.path.join(PKG, "liboc_asan.so")
ARCH = "gfx950"

# no packed fp32 vector instructions; MFMA accumulators in ordinary VGPRs
# (the softmax and epilogues then read them without AGPR<->VGPR copies)
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-mllvm", "-amdgpu-mfma-vgpr-form=1"]
COMMON = ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wno-unused-result"]
# host-side AddressSanitizer (each flag for the host pass only)
ASAN_FLAGS = "-Xarch_host -fsanitize=address -Xarch_host -fno-omit-frame-pointer -Xarch_host -g".split()


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the OmniCache library needs ROCm's hipcc")


def _compile(src: str, obj: str, extra=()) -> None:
    cmd = [_hipcc(), *COMMON, *DEVICE_FLAGS, *extra, "-c", src, "-o", obj]
    if src.endswith(".cpp"):
        cmd = [_hipcc(), *COMMON, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")


def build(verbose: bool = False, jobs: int = 8, asan: bool = False) -> str:
    bdir, lib = (BUILD_ASAN, LIB_ASAN) if asan else (BUILD, LIB)
    extra = ASAN_FLAGS if asan else ()
    os.makedirs(bdir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = [os.path.join(bdir, os.path.basename(s) + ".o") for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_compile, s, o, extra) for s, o in zip(srcs, objs)]
        for f in futs:
            f.result()
    tmp = lib + ".tmp"
    cmd = [_hipcc(), "-shared", f"--offload-arch={ARCH}", "-fPIC", *extra, "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


def asan_runtime() -> str:
    """The AddressSanitizer runtime of ROCm's clang (to preload)."""
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("AddressSanitizer runtime of ROCm's clang not found")
    return hits[-1]


if __name__ == "__main__":
    args = sys.argv[1:]
    asan = "asan" in args
    nums = [a for a in args if a.isdigit()]
    build(verbose=True, jobs=int(nums[0]) if nums else 8, asan=asan)

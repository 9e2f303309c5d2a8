"""Build libffmlp.so (the HIP kernels and the C ABI) for gfx950, in-tree.

    python -m paper_2403_17607_amd.build [--incremental]

Each translation unit under csrc/ is compiled with hipcc in parallel into
_build/, then linked into paper_2403_17607_amd/libffmlp.so.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libffmlp.so")
SOURCES = ["api.hip", "fwd.hip", "fwd16.hip", "fwd32.hip", "fwd64.hip", "fwd128.hip",
           "bwd.hip", "bwd16.hip", "bwd32.hip", "bwd64.hip", "bwd128.hip",
           "bwdg.hip", "bwdg16.hip", "bwdg32.hip", "bwdg64.hip", "bwdg128.hip",
           "trainf.hip", "trainf16.hip", "trainf32.hip", "trainf64.hip", "wgrad.hip", "optim.hip"]
ARCH = "gfx950"

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in VGPRs: otherwise the compiler gives some kernels' accumulators
    # to AGPRs, from which every conversion must first copy them (width-64
    # inference at 2^20 rows 43.8 -> 38.7 us, 3 -> 4 waves per SIMD)
    "-mllvm", "--amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _stale(src: str, obj: str) -> bool:
    """True unless obj is newer than src and every header it may include."""
    if not os.path.exists(obj):
        return True
    deps = [os.path.join(CSRC, src)]
    deps += [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    deps += [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))]
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(d) >= t for d in deps)


def _compile(src: str, incremental: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    if incremental and not _stale(src, obj):
        return obj
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, incremental: bool = False) -> str:
    """Compile every HIP source and link libffmlp.so; returns its path.
    With incremental=True, sources whose object is newer than the source and
    every header are not recompiled."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1, 16)) as ex:
        objs = list(ex.map(lambda src: _compile(src, incremental), SOURCES))
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True, incremental="--incremental" in sys.argv[1:])
    sys.exit(0)

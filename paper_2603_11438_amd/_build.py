"""Compile libar.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libar.so")

SOURCES = ["ar_kernels.hip", "ar_runtime.cpp", "ar_tuner.cpp", "ar_profile.cpp", "ar_noalloc.hip"]

# -packed-fp32-ops: no packed fp32 instructions in device code.
# -ffp-contract=off / no fast-math: every fp32 add is one IEEE RNE operation.
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wno-unused-variable",
    "-Wno-unused-but-set-variable",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libar)")


def build(verbose: bool = False) -> str:
    """Compile every HIP/C++ source of libar into _lib/libar.so (always rebuilds)."""
    os.makedirs(LIBDIR, exist_ok=True)
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    env = dict(os.environ)
    r = subprocess.run(cmd, cwd=PKG, env=env, capture_output=True, text=True)
    out = (r.stdout or "") + (r.stderr or "")
    # hipcc's host pass does not know the packed-fp32 target feature; that
    # warning is expected and harmless.
    lines = [l for l in out.splitlines() if "packed-fp32-ops" not in l]
    if r.returncode != 0:
        raise RuntimeError("libar build failed:\n" + "\n".join(lines))
    if verbose and lines:
        print("\n".join(lines))
    os.replace(tmp, LIB)
    return LIB


ABI_CHECK_SRC = os.path.join(ROOT, "tests", "native", "abi_gpu_check.cpp")
ABI_CHECK = os.path.join(ROOT, "tests", "native", "abi_gpu_check")


def build_abi_check() -> str:
    """Compile the host program that drives libar through its C ABI alone
    (a GPU test runs it); it links the in-tree libar.so by a relative rpath."""
    rpath = "$ORIGIN/" + os.path.relpath(LIBDIR, os.path.dirname(ABI_CHECK))
    tmp = ABI_CHECK + ".tmp"
    cmd = [hipcc(), "-O2", "-std=c++17", "-Wall", "-I", INCLUDE, ABI_CHECK_SRC, "-L", LIBDIR, "-lar",
           f"-Wl,-rpath,{rpath}", "-o", tmp]
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("abi_gpu_check build failed:\n" + (r.stdout or "") + (r.stderr or ""))
    os.replace(tmp, ABI_CHECK)
    return ABI_CHECK


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_abi_check())

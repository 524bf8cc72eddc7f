"""Build libaal.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2609_24150_amd.build              # compile every source, link
    python -m paper_2609_24150_amd.build --sanitize   # also the C-ABI layer's host code with
                                                      # AddressSanitizer + UBSan (_build/aal_api_asan.o)

Each .hip source compiles to an object in parallel, then one shared library
is linked next to this file.  Device code is built with packed-fp32
instructions disabled, FP contraction off (explicit fmaf only) and no-NaN
assumptions on device (inputs must be finite or -inf).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libaal.so")
ARCH = os.environ.get("AAL_OFFLOAD_ARCH", "gfx950")

COMMON_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-ffp-contract=off",
    "-Xarch_device", "-fno-honor-nans",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
] + os.environ.get("AAL_EXTRA_HIPCC_FLAGS", "").split()


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    cmd = [hipcc(), *COMMON_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


# Host-side sanitizers for the C-ABI layer (argument validation, workspace
# carve-up, dispatch).  Each -fsanitize= applies to the host compilation only:
# device code is never built with them.
SANITIZE_FLAGS = ["-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                  "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def compile_api_sanitized(obj: str | None = None) -> str:
    """Compile csrc/aal_api.hip with the host sanitizers into an object that a
    driver links with host-side stand-ins for the kernel launchers."""
    os.makedirs(BUILD, exist_ok=True)
    obj = obj or os.path.join(BUILD, "aal_api_asan.o")
    flags = [f for f in COMMON_FLAGS if f != "-O3"] + SANITIZE_FLAGS
    cmd = [hipcc(), *flags, "-c", os.path.join(CSRC, "aal_api.hip"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
    if "--sanitize" in sys.argv[1:]:
        print(f"built {compile_api_sanitized()}")
    sys.exit(0)

"""Builds libsn.so (the codec's C-ABI library) for gfx950 with hipcc.

    python -m paper_2506_01260_amd.build        # or: from ... import build; build.build()

Objects go to ``_build/`` at the repository root; the library is written
next to this file.  Every call recompiles.
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
LIB = os.path.join(PKG, "libsn.so")

ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-FP32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc(), *FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # hipcc's host pass does not know the device-only feature flag: drop that note
    noise = "not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if msg.strip():
        print(msg, file=sys.stderr)
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


# ---------------------------------------------------------------------------
# Host sanitizers: the C ABI's validation code (sn_api.cpp) built with g++
# under AddressSanitizer and UndefinedBehaviorSanitizer, linked with the
# regular (uninstrumented) kernel objects.  Only host code is instrumented;
# the library it makes is for the CPU tests of the argument checks
# (LD_PRELOAD the ASan runtime and point SN_LIBRARY at it).
SAN_LIB = os.path.join(BUILD, "libsn_hostsan.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-fno-omit-frame-pointer", "-g", "-O1"]


def build_host_sanitized() -> str:
    """Build _build/libsn_hostsan.so: sn_api.cpp under ASan + UBSan (g++),
    the kernel objects from the regular build (compiled first if missing or
    older than their sources)."""
    gxx = shutil.which("g++")
    if not gxx:
        raise RuntimeError("g++ not found")
    hips = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    objs = [os.path.join(BUILD, os.path.basename(h) + ".o") for h in hips]
    headers = glob.glob(os.path.join(CSRC, "*.h")) + [os.path.join(INCLUDE, "sn.h")]
    newest_h = max(os.path.getmtime(h) for h in headers)
    stale = [o for h, o in zip(hips, objs)
             if not os.path.exists(o) or os.path.getmtime(o) < max(os.path.getmtime(h), newest_h)]
    if stale:
        build()
    os.makedirs(BUILD, exist_ok=True)
    api_obj = os.path.join(BUILD, "sn_api.hostsan.o")
    cmd = [gxx, "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           f"-I{INCLUDE}", f"-I{CSRC}", *SAN_FLAGS, "-c", os.path.join(CSRC, "sn_api.cpp"),
           "-o", api_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stderr}")
    cmd = [gxx, "-shared", "-fPIC", *SAN_FLAGS, api_obj, *objs, "-L/opt/rocm/lib",
           "-Wl,-rpath,/opt/rocm/lib", "-lamdhip64", "-o", SAN_LIB]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stderr}")
    return SAN_LIB


if __name__ == "__main__":
    print(build())

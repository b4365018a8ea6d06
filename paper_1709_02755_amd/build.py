"""Build libsru.so (HIP for gfx950) in-tree with hipcc.

Each source compiles to an object in parallel, then one link.  Cross-compiles
without a GPU.  Usage: python -m paper_1709_02755_amd.build
"""

from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libsru.so")
OBJDIR = os.path.join(PKG, "_build")

ARCH = "gfx950"
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-fvisibility=hidden",
    # keep the compiler from forming packed fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libsru.so)")


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [hipcc(), "-x", "hip", "-c", src, "-o", obj] + HIP_FLAGS
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    # -z defs: an unresolved symbol (e.g. a kernel stub the host pass did not
    # emit) fails the build instead of the first load
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


# Host-side AddressSanitizer + UndefinedBehaviorSanitizer build of the C ABI
# layer (argument checks, workspace planning, dispatch), linked with the
# normal kernel objects: a CPU test runs the ABI checks against it.  The
# sanitizers apply to host code only; the device code is unchanged.
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
SAN_LIB = os.path.join(OBJDIR, "libsru_sanitized.so")


def sanitizer_runtime() -> str:
    """The clang ASan runtime the sanitized library needs preloaded."""
    llvm = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm")
    hits = sorted(glob.glob(os.path.join(llvm, "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    if not hits:
        raise RuntimeError("clang ASan runtime not found")
    return os.path.realpath(hits[-1])


def build_sanitized(verbose: bool = False) -> str:
    if not all(os.path.exists(os.path.join(OBJDIR, os.path.basename(p) + ".o"))
               for p in glob.glob(os.path.join(CSRC, "*.hip"))):
        build()
    api = os.path.join(CSRC, "sru_api.hip")
    obj = os.path.join(OBJDIR, "sru_api.sanitized.o")
    flags = [f if f != "-O3" else "-O1" for f in HIP_FLAGS] + ["-g"]
    cmd = [hipcc(), "-x", "hip", "-c", api, "-o", obj] + flags + SAN_FLAGS
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized compile failed:\n{r.stdout}\n{r.stderr}")
    others = [os.path.join(OBJDIR, os.path.basename(p) + ".o")
              for p in sorted(glob.glob(os.path.join(CSRC, "*.hip"))) if p != api]
    cmd = ([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-shared-libsan", "-o",
            SAN_LIB, obj] + others + SAN_FLAGS)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {SAN_LIB}")
    return SAN_LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

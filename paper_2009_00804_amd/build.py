"""Build libsaga.so (the HIP kernels + C ABI) for gfx950 with hipcc.

Usage: python -m paper_2009_00804_amd.build   (or build() from Python)
Objects go to <package>/_build/, the library to <package>/libsaga.so.
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
LIB = os.path.join(PKG, "libsaga.so")
SOURCES = ["abi.hip", "plan.hip", "gather.hip", "gemm.hip", "lstm.hip", "rel.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libsaga.so)")


FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# roctx: the stage ranges saga_layer opens when stage markers are on
LIBS = ["-lrocprofiler-sdk-roctx"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *FLAGS, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs, *LIBS]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


# Host sanitizers for the C-ABI layer: abi.hip (argument validation, shape
# and overlap checks, error messages) rebuilt with AddressSanitizer and
# UndefinedBehaviorSanitizer on its host code only (device code is built as
# usual), linked with the package's other objects from build().  The result
# is for host-side tests on a machine without a GPU: load it with the ASan
# runtime preloaded (asan_runtime()) and drive the validation paths.
SANITIZED = os.path.join(BUILD, "sanitize", "libsaga_sanitized.so")
SAN_FLAGS = [
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined",
    "-Xarch_host", "-fno-omit-frame-pointer",
    "-g",
]


def clangxx() -> str:
    return os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang++")


def asan_runtime() -> str:
    r = subprocess.run([clangxx(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True, check=True)
    return r.stdout.strip()


def build_sanitized(verbose: bool = False) -> str:
    """libsaga with abi.hip's host code under ASan + UBSan (see above).
    Needs the objects of build(); rebuilt only when abi.hip or a header is
    newer than the library."""
    out_dir = os.path.dirname(SANITIZED)
    os.makedirs(out_dir, exist_ok=True)
    others = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "abi.hip"]
    if not all(os.path.exists(o) for o in others):
        build()
    deps = [os.path.join(CSRC, "abi.hip"), os.path.join(INCLUDE, "saga.h"),
            os.path.join(CSRC, "saga_internal.h"), os.path.join(CSRC, "saga_device.h"), *others]
    if os.path.exists(SANITIZED) and os.path.getmtime(SANITIZED) >= max(map(os.path.getmtime, deps)):
        return SANITIZED
    obj = os.path.join(out_dir, "abi_sanitized.o")
    flags = [f for f in FLAGS if f != "-O3"] + ["-O1"] + SAN_FLAGS
    cmd = [hipcc(), *flags, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "abi.hip"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on abi.hip (sanitized):\n{r.stderr}")
    rocm_lib = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "lib")
    tmp = SANITIZED + ".tmp"
    cmd = [clangxx(), "-shared", "-fPIC", "-fsanitize=address,undefined", "-shared-libsan", "-o", tmp,
           obj, *others, "-L", rocm_lib, "-lamdhip64", *LIBS, f"-Wl,-rpath,{rocm_lib}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stderr}")
    os.replace(tmp, SANITIZED)
    if verbose:
        print("built", SANITIZED)
    return SANITIZED


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

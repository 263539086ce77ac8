"""Builds libkashin.so (the C-ABI library) in-tree with hipcc for gfx950.

    python -m paper_2609_11687_amd.build [-v] [--host-sanitized]

Each kernel translation unit (one per supported vector length) compiles in
parallel; objects go to ``_build/`` next to this file and the library to
``libkashin.so`` in this package directory.  The C consumer of the ABI that the
tests run (tests/c_abi/kashin_abi_check.c) is built into ``_build/`` after it.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libkashin.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # no packed-fp32 instructions: plain fp32 VALU only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-I", CSRC,
]


# the Cholesky factorisation and triangular inverse of the compensation factor (kashin_optq_factor)
LINK_LIBS = ["-L/opt/rocm/lib", "-lrocsolver", "-lrocblas", "-Wl,-rpath,/opt/rocm/lib"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list[str]:
    srcs = [os.path.join(CSRC, "kashin_api.cpp"), os.path.join(CSRC, "kashin_dispatch.hip"),
            os.path.join(CSRC, "kashin_rotate.hip"), os.path.join(CSRC, "kashin_optq.hip")]
    srcs += sorted(glob.glob(os.path.join(CSRC, "kashin_n*.hip")))
    return srcs


def source_digest() -> str:
    """SHA-256 over every kernel and interface source (csrc/ and include/): a profile taken on
    other sources no longer describes the built kernels."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(CSRC, "*")) + glob.glob(os.path.join(ROOT, "include", "*.h")))
    for f in files:
        if os.path.isfile(f):
            h.update(os.path.relpath(f, ROOT).encode())
            with open(f, "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [_hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source and link libkashin.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4)))
    # biggest translation units first
    order = sorted(srcs, key=lambda p: ("11008" not in p, "13824" not in p, "14336" not in p, "16384" not in p, p))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), order))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, *LINK_LIBS]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


# A C program that uses the library through include/kashin.h and the HIP runtime alone (the tests
# run it): the boundary exercised without the Python binding.
ABI_CHECK_SRC = os.path.join(ROOT, "tests", "c_abi", "kashin_abi_check.c")
ABI_CHECK = os.path.join(BUILD, "kashin_abi_check")


def build_abi_check(verbose: bool = False) -> str:
    """Compile tests/c_abi/kashin_abi_check.c with the host C compiler against libkashin.so."""
    os.makedirs(BUILD, exist_ok=True)
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise RuntimeError("no C compiler")
    cmd = [cc, "-O1", "-std=c11", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", "/opt/rocm/include", ABI_CHECK_SRC, "-o", ABI_CHECK, "-L", HERE, "-lkashin", "-L/opt/rocm/lib",
           "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath,/opt/rocm/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"C ABI check failed to build:\n{res.stderr}")
    return ABI_CHECK


# Host-code sanitizers for the C-ABI layer (device code is built without them: the GPU runs no
# sanitizer).  Each -fsanitize= follows -Xarch_host, so only the host pass sees it.
HOST_SANITIZE = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split()
SANITIZED_LIB = os.path.join(BUILD, "libkashin_host_sanitized.so")


def asan_runtime() -> str:
    """Path of the compiler's AddressSanitizer runtime (preloaded into a process that loads the
    sanitized library, since the Python interpreter itself is not instrumented)."""
    res = subprocess.run([_hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return res.stdout.strip()


def build_host_sanitized(verbose: bool = False) -> str:
    """libkashin with the host layer (kashin_api.cpp: validation, plan tables, dispatch) compiled
    under AddressSanitizer and UndefinedBehaviorSanitizer, linked with the kernel objects of the
    regular build (built first if missing).  Written to _build/, never next to libkashin.so."""
    if not all(os.path.exists(os.path.join(BUILD, os.path.basename(s_) + ".o")) for s_ in sources()):
        build(verbose)
    api = os.path.join(CSRC, "kashin_api.cpp")
    obj = os.path.join(BUILD, "kashin_api.host_sanitized.o")
    flags = [a for a in HIPCC_FLAGS if a != "-O3"] + ["-O1", "-g", "-Xarch_host", "-fno-omit-frame-pointer",
                                                      "-Xarch_host", "-fno-sanitize-recover=undefined"]
    cmd = [_hipcc(), *flags, *HOST_SANITIZE, "-c", api, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for the sanitized host layer:\n{res.stderr}")
    objs = [obj] + [os.path.join(BUILD, os.path.basename(s_) + ".o") for s_ in sources() if s_ != api]
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *HOST_SANITIZE, "-shared-libasan",
           "-o", SANITIZED_LIB, *objs, *LINK_LIBS]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link of the sanitized library failed:\n{res.stderr}")
    return SANITIZED_LIB


if __name__ == "__main__":
    if "--host-sanitized" in sys.argv:
        print(build_host_sanitized(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
        print(build_abi_check(verbose="-v" in sys.argv))

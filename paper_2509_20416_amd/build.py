"""Build libfe.so (gfx950) in-tree with hipcc.

    python -m paper_2509_20416_amd.build [--asan]

Object files go to paper_2509_20416_amd/_build/, the library to
paper_2509_20416_amd/libfe.so.  With --asan, a second library,
libfe_asan.so, whose host code (the runtime: argument checks, layouts,
chunking, graph cache) is built with AddressSanitizer; the device code is
the same.  Its __asan_* symbols come from the sanitizer runtime preloaded
into the process (LD_PRELOAD=ASAN_RUNTIME); it is for host-only test runs
and is never loaded on a GPU.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libfe.so")
LIB_ASAN = os.path.join(HERE, "libfe_asan.so")
SOURCES = ["fe_gemm.hip", "fe_attn.hip", "fe_misc.hip", "fe_pass.hip", "fe_runtime.hip"]
ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result", "-I", os.path.join(ROOT, "include")]
# host code only: every sanitizer flag goes through -Xarch_host
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
# roctx ranges (rocprofiler-sdk) around the entry points
LINK_LIBS = ["-L", os.path.join(ROCM, "lib"), "-lrocprofiler-sdk-roctx",
             "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def asan_runtime() -> str:
    """Path of the AddressSanitizer runtime that libfe_asan.so expects preloaded."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True, check=True)
    return r.stdout.strip()


def _compile(src: str, verbose: bool, asan: bool = False) -> str:
    out = os.path.join(OUT, "asan") if asan else OUT
    obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *(ASAN_FLAGS if asan else []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
    if msg.strip() and verbose:
        print(msg)
    return obj


def build(verbose: bool = False, asan: bool = False) -> str:
    lib = LIB_ASAN if asan else LIB
    os.makedirs(os.path.join(OUT, "asan") if asan else OUT, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, asan), SOURCES))
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, *LINK_LIBS]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    build(verbose=True, asan="--asan" in sys.argv[1:])
    sys.exit(0)

"""Build libkvpool.so in-tree for gfx950.

HIP device code (``csrc/*.hip``) is compiled by hipcc for gfx950 only; host
C++ (``csrc/*.cpp``) by g++ against the HIP runtime headers.  The shared
library is linked by hipcc.  Run ``python -m paper_2606_14779_amd.build``.
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
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libkvpool.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Wno-unused-parameter",
    "--offload-arch=" + ARCH,
    # no packed fp32 instructions in any device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Wno-unused-parameter",
             "-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include")]


def _hipcc() -> str:
    p = os.path.join(ROCM, "bin", "hipcc")
    return p if os.path.exists(p) else (shutil.which("hipcc") or "hipcc")


def _compile(src: str, extra: list[str]) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    if src.endswith(".hip"):
        cmd = [_hipcc()] + HIPCC_FLAGS + extra + ["-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
    else:
        cmd = ["g++"] + CXX_FLAGS + extra + ["-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    return obj


def build(verbose: bool = False, extra: list[str] | None = None) -> str:
    """Compile every source and link libkvpool.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, extra or []), srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs + [
        "-L" + os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, LIB)
    # a plain C++ client of the ABI (used by the tests): links the library, no Python
    client_src = os.path.join(ROOT, "tests", "abi_client", "abi_client.cpp")
    if os.path.exists(client_src):
        exe = os.path.join(ROOT, "tests", "abi_client", "abi_client")
        cmd = ["g++"] + CXX_FLAGS + ["-I", INCLUDE, client_src, "-o", exe + ".tmp", "-L" + PKG, "-lkvpool",
                                     "-Wl,-rpath,$ORIGIN/../../paper_2606_14779_amd", "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
                                     "-Wl,--export-dynamic-symbol=hipHostMalloc",
                                     "-Wl,-rpath," + os.path.join(ROCM, "lib")]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("abi client build failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
        os.replace(exe + ".tmp", exe)
        # the same client over a host-sanitized build of the library (its own file: g++ only)
        from . import build_asan
        build_asan.build(os.path.join(BUILD, "kernels.hip.o"))
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True, extra=sys.argv[1:])

"""Host-side AddressSanitizer / UndefinedBehaviorSanitizer build of the library
and of the plain C++ ABI client, for a GPU test of the library's host code.

Only host C++ is instrumented, with g++ (GPU code cannot run under a sanitizer
here): the library's .cpp sources are compiled with the sanitizers and linked
with the already built, uninstrumented kernels object.  The results sit under
tests/abi_client/ and are used by tests/test_abi_client.py only.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
OUT = os.path.join(ROOT, "tests", "abi_client", "asan")
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("sanitizer build failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))


def build(kernels_obj: str) -> str:
    """Instrumented libkvpool.so and abi_client_asan; returns the client's path."""
    import concurrent.futures as cf
    os.makedirs(OUT, exist_ok=True)
    names = sorted(n for n in os.listdir(CSRC) if n.endswith(".cpp"))
    objs = [os.path.join(OUT, n + ".o") for n in names]

    def one(name, obj):
        _run(["g++", "-O1", "-g", "-std=c++17", "-fPIC"] + SAN + ["-D__HIP_PLATFORM_AMD__", "-isystem",
             os.path.join(ROCM, "include"), "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, name), "-o", obj])
    with cf.ThreadPoolExecutor(max_workers=min(8, len(names))) as ex:
        list(ex.map(one, names, objs))
    lib = os.path.join(OUT, "libkvpool.so")
    _run(["g++", "-shared", "-fPIC"] + SAN + ["-o", lib + ".tmp"] + objs + [kernels_obj, "-L" + os.path.join(ROCM, "lib"),
         "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    os.replace(lib + ".tmp", lib)
    exe = os.path.join(ROOT, "tests", "abi_client", "abi_client_asan")
    _run(["g++", "-O1", "-g", "-std=c++17"] + SAN + ["-D__HIP_PLATFORM_AMD__", "-isystem", os.path.join(ROCM, "include"),
         "-I", INCLUDE, os.path.join(ROOT, "tests", "abi_client", "abi_client.cpp"), "-o", exe + ".tmp", "-L" + OUT,
         "-lkvpool", "-Wl,-rpath,$ORIGIN/asan", "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
         "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-Wl,--export-dynamic-symbol=hipHostMalloc"])
    os.replace(exe + ".tmp", exe)
    for o in objs:
        os.remove(o)
    return exe

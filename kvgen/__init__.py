"""Seeded synthetic inputs shared by the tests, the bench and the oracle side.

This package defines inputs only: bf16 KV values (``kvgen.c``) and the
structure of the five workloads (``workloads.py``: shapes, pool regions and
their bandwidth weights, destination block tables, context lengths, present
prefixes).  It contains none of the method's arithmetic -- no placement, no
store and no gather -- so that the GPU path and the oracle can both consume
the same bytes without sharing any method code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvgen.c")
_LIB = os.path.join(_HERE, "libkvgen.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile kvgen.c into libkvgen.so next to it (gcc, host code only)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=False)
            lib = ctypes.CDLL(_LIB)
            u64, u32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p
            lib.kvgen_block_key.restype = u64
            lib.kvgen_block_key.argtypes = [u64, u64, u64]
            lib.kvgen_sm64.restype = u64
            lib.kvgen_sm64.argtypes = [u64]
            lib.kvgen_fill_elems.restype = None
            lib.kvgen_fill_elems.argtypes = [u64, u64, u64, u64, u64, vp]
            lib.kvgen_fill_cache.restype = ctypes.c_int
            lib.kvgen_fill_cache.argtypes = [u64, u64, u32, vp, vp, u32, u32, u32, u32,
                                             vp, vp, u32]
            lib.kvgen_normal_table.restype = None
            lib.kvgen_normal_table.argtypes = [vp]
            lib.kvgen_ppnd16.restype = ctypes.c_double
            lib.kvgen_ppnd16.argtypes = [ctypes.c_double]
            lib.kvgen_fill_u16.restype = None
            lib.kvgen_fill_u16.argtypes = [vp, u64, ctypes.c_uint16, u32]
            _lib = lib
    return _lib


def default_threads() -> int:
    """Threads for host-side generation: the CPUs this process may run on, at most 16."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def sm64(x: int) -> int:
    """splitmix64 output function of a 64-bit integer."""
    return int(_load().kvgen_sm64(x & 0xFFFFFFFFFFFFFFFF))


def subseed(seed: int, tag: str) -> int:
    """A 64-bit sub-seed for a named stream of structural randomness."""
    h = seed & 0xFFFFFFFFFFFFFFFF
    for ch in tag.encode():
        h = sm64(h ^ ch)
    return h


def normal_table() -> np.ndarray:
    """The 65536-entry bf16 table Q[i] = bf16(Phi^-1((i + 0.5) / 65536)) the values come from."""
    out = np.empty(65536, dtype=np.uint16)
    _load().kvgen_normal_table(out.ctypes.data)
    return out


def ppnd16(p: float) -> float:
    """Standard normal quantile (Wichura AS 241) as used to build the table."""
    return float(_load().kvgen_ppnd16(p))


def block_values(seed: int, request: int, block: int, L: int, H: int, bs: int, D: int) -> np.ndarray:
    """Logical contents of one block: uint16 (bf16 bits) array [L][2][H][bs][D]."""
    n = L * 2 * H * bs * D
    out = np.empty(n, dtype=np.uint16)
    _load().kvgen_fill_elems(seed, request, block, 0, n, out.ctypes.data)
    return out.reshape(L, 2, H, bs, D)


def elems(seed: int, request: int, block: int, e0: int, count: int) -> np.ndarray:
    """Elements [e0, e0+count) of one block in canonical [L][2][H][bs][D] order."""
    out = np.empty(count, dtype=np.uint16)
    _load().kvgen_fill_elems(seed, request, block, e0, count, out.ctypes.data)
    return out


def fill_cache(seed: int, request: int, block_ids, slots, L: int, H: int, bs: int, D: int,
               k_ptrs, v_ptrs, threads: int | None = None) -> None:
    """Write the values of blocks ``block_ids`` into an engine-layout cache on the host.

    ``k_ptrs[l]`` / ``v_ptrs[l]`` are host addresses of per-layer caches laid out
    ``[num_slots][H][bs][D]`` (bf16); block ``block_ids[i]`` lands in slot ``slots[i]``.
    """
    ids = np.ascontiguousarray(block_ids, dtype=np.uint64)
    sl = np.ascontiguousarray(slots, dtype=np.int32)
    assert ids.shape == sl.shape and ids.ndim == 1
    kp = (ctypes.c_void_p * L)(*[int(p) for p in k_ptrs])
    vp_ = (ctypes.c_void_p * L)(*[int(p) for p in v_ptrs])
    _load().kvgen_fill_cache(seed, request, len(ids), ids.ctypes.data, sl.ctypes.data,
                             L, H, bs, D, ctypes.cast(kp, ctypes.c_void_p),
                             ctypes.cast(vp_, ctypes.c_void_p),
                             threads or default_threads())


def fill_u16(addr: int, count: int, value: int, threads: int | None = None) -> None:
    """Fill ``count`` uint16 words at host address ``addr`` with ``value``."""
    _load().kvgen_fill_u16(addr, count, value & 0xFFFF, threads or default_threads())

"""CPU oracle for the KV-pool retrieval path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it.  The arithmetic lives in ``oracle.c`` (plain C); this
module compiles it with gcc and wraps it with ctypes and numpy.

Functions and the passage each follows (Unified KV Pooling):
  counts(bw, n)        Eq. (1) and Eq. (2); Algorithm 1 counting part.
  Pool.place(req, n)   Algorithm 1 partition part; Sec. 4.2 contiguous range;
                       GLT record (Table "Fields of the GLT").
  Pool.release(req)    returns the ranges (free list, first fit).
  store(...)           Algorithm 1 store part (MemStore): block chunks into
                       the pool layout.
  gather(...)          Sec. 4.3 KV retrieval: pool chunks back into the
                       engine's per-layer paged cache.
Every function is pinned by tests under ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

ABSENT = 0xFFFFFFFF
SECTOR = 4096
LOC_DTYPE = np.dtype([("region", "<u4"), ("gen", "<u4"), ("offset", "<u8")])


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB):
                build(force=False)
            lib = ctypes.CDLL(_LIB)
            u64, u32, vp, i32 = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_int
            lib.oracle_counts.restype = i32
            lib.oracle_counts.argtypes = [vp, u32, u64, vp]
            lib.oracle_pool_new.restype = vp
            lib.oracle_pool_new.argtypes = [u32, vp, vp, u64]
            lib.oracle_pool_free.restype = None
            lib.oracle_pool_free.argtypes = [vp]
            lib.oracle_place.restype = i32
            lib.oracle_place.argtypes = [vp, u64, u32, vp]
            lib.oracle_extend.restype = i32
            lib.oracle_extend.argtypes = [vp, u64, u32, vp]
            lib.oracle_lookup.restype = i32
            lib.oracle_lookup.argtypes = [vp, u64, u32, vp]
            lib.oracle_release.restype = i32
            lib.oracle_release.argtypes = [vp, u64]
            lib.oracle_largest_free.restype = u64
            lib.oracle_largest_free.argtypes = [vp, u32]
            copy_args = [u32, vp, vp, vp, vp, vp, u32, u32, u32, u32, u32, u32]
            lib.oracle_store.restype = None
            lib.oracle_store.argtypes = copy_args
            lib.oracle_gather.restype = None
            lib.oracle_gather.argtypes = copy_args
            _lib = lib
    return _lib


def counts(bandwidths, n: int) -> np.ndarray:
    """Target counts per device for n KV blocks (Eq. 2 with the remainder rule)."""
    bw = np.ascontiguousarray(bandwidths, dtype=np.uint64)
    out = np.zeros(len(bw), dtype=np.uint64)
    rc = _load().oracle_counts(bw.ctypes.data, len(bw), n, out.ctypes.data)
    if rc:
        raise ValueError("oracle_counts rejected the input")
    return out


class Pool:
    """Placement bookkeeping of one pool: per-device free lists and GLT records."""

    def __init__(self, bandwidths, capacities, block_bytes: int):
        self._bw = np.ascontiguousarray(bandwidths, dtype=np.uint64)
        cap = np.ascontiguousarray(capacities, dtype=np.uint64)
        assert len(cap) == len(self._bw)
        self.n_dev = len(self._bw)
        self.block_bytes = block_bytes
        self._p = _load().oracle_pool_new(self.n_dev, self._bw.ctypes.data, cap.ctypes.data,
                                          block_bytes)
        if not self._p:
            raise ValueError("oracle_pool_new rejected the input")

    def close(self):
        if self._p:
            _load().oracle_pool_free(self._p)
            self._p = None

    __del__ = close

    @staticmethod
    def _count(n) -> int:
        # the C side takes uint32_t; ctypes would wrap a negative count into a huge one
        n = int(n)
        if not 0 <= n < 1 << 32:
            raise ValueError("block count %d outside [0, 2^32)" % n)
        return n

    def place(self, request: int, n_blocks: int) -> np.ndarray:
        n_blocks = self._count(n_blocks)
        out = np.zeros(n_blocks, dtype=LOC_DTYPE)
        rc = _load().oracle_place(self._p, request, n_blocks, out.ctypes.data)
        if rc:
            raise PlacementError(rc)
        return out

    def try_place(self, request: int, n_blocks: int):
        n_blocks = self._count(n_blocks)
        out = np.zeros(max(n_blocks, 1), dtype=LOC_DTYPE)
        rc = _load().oracle_place(self._p, request, n_blocks, out.ctypes.data)
        return rc, out[:n_blocks]

    def extend(self, request: int, n_new: int) -> np.ndarray:
        """The next offload set of a placed request: entries of its blocks n_old .. n_old+n_new-1."""
        n_new = self._count(n_new)
        out = np.zeros(n_new, dtype=LOC_DTYPE)
        rc = _load().oracle_extend(self._p, request, n_new, out.ctypes.data)
        if rc:
            raise PlacementError(rc)
        return out

    def try_extend(self, request: int, n_new: int):
        n_new = self._count(n_new)
        out = np.zeros(max(n_new, 1), dtype=LOC_DTYPE)
        rc = _load().oracle_extend(self._p, request, n_new, out.ctypes.data)
        return rc, out[:n_new]

    def lookup(self, request: int, n_blocks: int) -> np.ndarray:
        n_blocks = self._count(n_blocks)
        out = np.zeros(n_blocks, dtype=LOC_DTYPE)
        rc = _load().oracle_lookup(self._p, request, n_blocks, out.ctypes.data)
        if rc:
            raise PlacementError(rc)
        return out

    def release(self, request: int) -> int:
        return _load().oracle_release(self._p, request)

    def largest_free(self, dev: int) -> int:
        return int(_load().oracle_largest_free(self._p, dev))


class PlacementError(RuntimeError):
    def __init__(self, rc):
        super().__init__("oracle placement failed with code %d" % rc)
        self.rc = rc


def _ptr_array(ptrs):
    arr = (ctypes.c_void_p * len(ptrs))(*[int(p) for p in ptrs])
    return arr


def _addr(a) -> int:
    if isinstance(a, np.ndarray):
        assert a.flags.c_contiguous
        return a.ctypes.data
    return int(a)


def _copy(fn, loc_map, slots, region_mem, k_layers, v_layers, shape, layout):
    """Shared argument marshalling of store/gather (all host memory)."""
    L, H, bs, D, eb = shape
    m = np.ascontiguousarray(loc_map, dtype=LOC_DTYPE)
    s = np.ascontiguousarray(slots, dtype=np.int32)
    assert len(m) == len(s)
    assert len(k_layers) == L and len(v_layers) == L
    regs = _ptr_array([_addr(r) for r in region_mem])
    ks = _ptr_array([_addr(k) for k in k_layers])
    vs = _ptr_array([_addr(v) for v in v_layers])
    fn(len(m), m.ctypes.data, s.ctypes.data, ctypes.addressof(regs), ctypes.addressof(ks),
       ctypes.addressof(vs), L, H, bs, D, eb, layout)


def store(loc_map, src_slots, region_mem, k_layers, v_layers, shape, layout=0):
    """Offload copy into the pool (host buffers; ``shape`` = (L, H, bs, D, elem_bytes))."""
    _copy(_load().oracle_store, loc_map, src_slots, region_mem, k_layers, v_layers, shape, layout)


def gather(loc_map, dst_slots, region_mem, k_layers, v_layers, shape, layout=0):
    """Retrieval copy from the pool into the engine cache (host buffers)."""
    _copy(_load().oracle_gather, loc_map, dst_slots, region_mem, k_layers, v_layers, shape, layout)

"""ctypes binding of libkvpool.so (argument marshalling only).

Every function maps one-to-one onto an ``extern "C"`` entry point declared in
``include/kvpool.h``; all computation, validation and GPU work happens in the
library.  Device memory and streams are passed as integers (``tensor.data_ptr()``,
``torch.cuda.Stream.cuda_stream``).  If the library has not been built this
module raises on import: there is no fallback path.
"""
from __future__ import annotations

import atexit
import ctypes
import operator
import os
import weakref
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvpool.so")

KVP_OK = 0
ERRORS = {-1: "INVALID", -2: "NOMEM", -3: "NOSPACE", -4: "NOTFOUND", -5: "STALE", -6: "HIP", -7: "IO"}
REGION_HOST, REGION_STAGING, REGION_FILE = 0, 1, 2
HOST_DEFAULT, HOST_COHERENT, HOST_NONCOHERENT = 0, 1, 2
FILE_BUFFERED = 1            # file regions: through the page cache instead of O_DIRECT
ABSENT = 0xFFFFFFFF
CLASS_HOST, CLASS_STAGING = 0, 1
OP_RETRIEVE, OP_STORE = 0, 1
LAUNCH_NT_LOAD, LAUNCH_NT_STORE, LAUNCH_LDS, LAUNCH_SPLIT2, LAUNCH_XCD, LAUNCH_SDMA = 1, 2, 4, 8, 16, 32
LAUNCH_CHUNK_MAJOR = 64
LAUNCH_UPLOAD = 128          # no small-call launch: upload the work list, one launch per class
LAUNCH_TILE = 256            # workgroup-owned tiles of 8 work items x 1 chunk
MEASURE_SHARED_LINK = 1
MEASURE_SHARED_HBM = 4       # staging regions share the one GPU's HBM: their rate divided by their count
MEASURE_FILES_TOGETHER = 2   # file regions read all at once, as a retrieve reads them

LOC_DTYPE = np.dtype([("region", "<u4"), ("gen", "<u4"), ("offset", "<u8")])


class _RegionDesc(ctypes.Structure):
    _fields_ = [("type", ctypes.c_uint32), ("numa_node", ctypes.c_int32),
                ("capacity_bytes", ctypes.c_uint64), ("flags", ctypes.c_uint32),
                ("reserved", ctypes.c_uint32)]


class _KVSpec(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_uint32), ("num_kv_heads", ctypes.c_uint32),
                ("head_dim", ctypes.c_uint32), ("block_size", ctypes.c_uint32),
                ("elem_bytes", ctypes.c_uint32), ("pool_layout", ctypes.c_uint32)]


class _RegionInfo(ctypes.Structure):
    _fields_ = [("type", ctypes.c_uint32), ("numa_node", ctypes.c_int32),
                ("numa_node_actual", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("capacity_bytes", ctypes.c_uint64), ("bandwidth", ctypes.c_uint64),
                ("host_ptr", ctypes.c_void_p), ("device_ptr", ctypes.c_void_p)]


class _Timing(ctypes.Structure):
    _fields_ = [("host_ms", ctypes.c_float), ("staging_ms", ctypes.c_float),
                ("host_blocks", ctypes.c_uint32), ("staging_blocks", ctypes.c_uint32)]


class _TimingSummary(ctypes.Structure):
    _fields_ = [("calls", ctypes.c_uint32), ("host_calls", ctypes.c_uint32),
                ("staging_calls", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("host_ms_sum", ctypes.c_float), ("host_ms_min", ctypes.c_float), ("host_ms_max", ctypes.c_float),
                ("staging_ms_sum", ctypes.c_float), ("staging_ms_min", ctypes.c_float),
                ("staging_ms_max", ctypes.c_float)]


assert ctypes.sizeof(_RegionDesc) == 24 and ctypes.sizeof(_KVSpec) == 24
assert LOC_DTYPE.itemsize == 16

# A process must hold one HIP runtime.  PyTorch-ROCm ships its own
# libamdhip64 and asks for it by an unversioned name, which would not match a
# runtime loaded earlier under its soname; loading torch first makes this
# library bind to torch's runtime instead of mapping a second one.
try:
    import torch  # noqa: F401
except ImportError:
    pass

if not os.path.exists(LIB_PATH):
    raise ImportError("libkvpool.so is not built (%s); run `python -m paper_2606_14779_amd.build`"
                      % LIB_PATH)
_cdll = ctypes.CDLL(LIB_PATH)

# Pools still open when the interpreter exits are closed by an exit hook, so
# that kv_pool_destroy (which waits for the pool's streams and frees its HIP
# memory) runs while the HIP runtime is whole, not from a finaliser after the
# runtime's own exit-time teardown.  The hook is registered after torch's
# import above, and exit hooks run last-registered first, so it runs before
# any that torch registered.
_live_pools = weakref.WeakSet()


def _close_live_pools():
    for p in list(_live_pools):
        try:
            p.close()
        except Exception:
            pass


atexit.register(_close_live_pools)

_u32, _u64, _i32, _vp = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p
_SIGS = {
    "kv_pool_create": (_i32, [_vp, _vp, _u32, _vp, _i32, _vp]),
    "kv_pool_create_files": (_i32, [_vp, _vp, _u32, _vp, _i32, _vp, _vp]),
    "kv_pool_place": (_i32, [_vp, _u64, _u32, _vp]),
    "kv_pool_extend": (_i32, [_vp, _u64, _u32, _vp]),
    "kv_pool_lookup": (_i32, [_vp, _u64, _u32, _vp]),
    "kv_pool_store": (_i32, [_vp, _vp, _u32, _vp, _u32, _vp, _vp, _vp]),
    "kv_pool_retrieve": (_i32, [_vp, _vp, _u32, _vp, _u32, _vp, _vp, _vp]),
    "kv_pool_retrieve_request": (_i32, [_vp, _u64, _u32, _vp, _u32, _vp, _vp, _vp]),
    "kv_pool_retrieve_noalloc": (_i32, [_vp, _vp, _u32, _vp, _u32, _vp, _vp, _vp]),
    "kv_pool_retrieve_layers": (_i32, [_vp, _vp, _u32, _vp, _u32, _u32, _u32, _vp, _vp, _vp]),
    "kv_pool_store_layers": (_i32, [_vp, _vp, _u32, _vp, _u32, _u32, _u32, _vp, _vp, _vp]),
    "kv_pool_release": (_i32, [_vp, _u64]),
    "kv_pool_destroy": (None, [_vp]),
    "kv_pool_last_error": (ctypes.c_char_p, []),
    "kv_pool_region_info": (_i32, [_vp, _u32, _vp]),
    "kv_pool_region_read": (_i32, [_vp, _u32, _u64, _u64, _vp]),
    "kv_pool_counts": (_i32, [_vp, _u32, _u64, _vp]),
    "kv_pool_measure_bandwidth": (_i32, [_vp, _u64, _u32, _vp]),
    "kv_pool_set_bandwidths": (_i32, [_vp, _vp]),
    "kv_pool_set_launch": (_i32, [_vp, _u32, _u32, _u32, _u32]),
    "kv_pool_set_copy_ring": (_i32, [_vp, _u64]),
    "kv_pool_set_file_ring": (_i32, [_vp, _u64]),
    "kv_pool_set_timing": (_i32, [_vp, _i32]),
    "kv_pool_last_timing": (_i32, [_vp, _vp]),
    "kv_pool_timing_summary": (_i32, [_vp, _vp]),
    "kv_probe_copy_kernel": (_i32, [_vp, _vp, _u64, _u32, _u32, _vp]),
    "kv_probe_memcpy": (_i32, [_vp, _vp, _u64, _vp]),
}
# ctypes wraps an integer outside its C type's range silently (-1 becomes
# 2^32-1 for a uint32_t: a slot count that every table entry passes), so every
# integer argument is checked against its type's range first.
_RANGES = {_u32: (0, 1 << 32), _u64: (0, 1 << 64), _i32: (-(1 << 31), 1 << 31)}


def _range_checked(name, f, argtypes):
    checks = [(i, _RANGES[t]) for i, t in enumerate(argtypes) if t in _RANGES]

    def call(*args):
        for i, (lo, hi) in checks:
            v = operator.index(args[i])
            if not lo <= v < hi:
                raise ValueError("%s: argument %d = %d is outside [%d, %d)" % (name, i, v, lo, hi))
        return f(*args)
    call.__name__ = name
    return call


class _Lib:
    """The library's entry points, with their integer arguments range-checked."""


_lib = _Lib()
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_cdll, _name)
    _f.restype = _res
    _f.argtypes = _args
    setattr(_lib, _name, _range_checked(_name, _f, _args))

EXPORTED = tuple(_SIGS)


class KVPoolError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (%d): %s" % (ERRORS.get(code, "?"), code, msg))
        self.code = code
        self.name = ERRORS.get(code, "?")


def _check(rc: int) -> None:
    if rc != KVP_OK:
        raise KVPoolError(rc, (_lib.kv_pool_last_error() or b"").decode())


def _ptrs(ptrs) -> ctypes.Array:
    return (ctypes.c_void_p * len(ptrs))(*[int(p) for p in ptrs])


def _block_count(n) -> int:
    """A block count as the ABI's uint32_t, checked before an output array of that size is made."""
    n = operator.index(n)
    if not 0 <= n < 1 << 32:
        raise ValueError("block count %d is outside [0, 2^32)" % n)
    return n


def _struct(cls, *vals):
    """A ctypes structure of the ABI, each integer field checked against its type's range first."""
    for (name, t), v in zip(cls._fields_, vals):
        lo, hi = _RANGES[t]
        if not lo <= operator.index(v) < hi:
            raise ValueError("%s.%s = %d is outside [%d, %d)" % (cls.__name__, name, v, lo, hi))
    return cls(*vals)


def _int_array(t, dtype, what) -> np.ndarray:
    """An integer array as the ABI's element type; entries of another integer type are checked
    against that type's range, not wrapped."""
    a = np.asarray(t)
    dt = np.dtype(dtype)
    if a.dtype != dt and a.size:
        if a.dtype.kind not in "iu":
            raise ValueError("%s must hold integers" % what)
        info = np.iinfo(dt)
        if int(a.min()) < info.min or int(a.max()) > info.max:
            raise ValueError("%s entry outside the range of %s" % (what, dt.name))
    return np.ascontiguousarray(a, dtype=dt)


def _loc_array(m) -> np.ndarray:
    a = np.ascontiguousarray(m, dtype=LOC_DTYPE)
    return a


@dataclass
class Region:
    kind: str                 # "host", "staging" or "file"
    capacity_bytes: int
    numa_node: int = -1
    coherence: int = HOST_DEFAULT   # the region's flags: host KVP_HOST_*, file 0 or FILE_BUFFERED
    path: str | None = None         # file regions: the file to create, or a block device


@dataclass
class KVSpec:
    num_layers: int
    num_kv_heads: int
    head_dim: int
    block_size: int = 16
    elem_bytes: int = 2
    pool_layout: int = 0

    @property
    def chunk_bytes(self) -> int:
        return self.num_kv_heads * self.block_size * self.head_dim * self.elem_bytes

    @property
    def block_bytes(self) -> int:
        return 2 * self.num_layers * self.chunk_bytes


def counts(bandwidths, n: int) -> np.ndarray:
    """The library's per-region target counts for n blocks (kv_pool_counts)."""
    bw = _int_array(bandwidths, np.uint64, "bandwidths")
    out = np.zeros(len(bw), dtype=np.uint64)
    _check(_lib.kv_pool_counts(bw.ctypes.data if len(bw) else None, len(bw), n, out.ctypes.data))
    return out


def probe_copy_kernel(dst: int, src: int, nbytes: int, grid: int = 0, flags: int = 0, stream: int = 0):
    _check(_lib.kv_probe_copy_kernel(dst, src, nbytes, grid, flags, stream or None))


def probe_memcpy(dst: int, src: int, nbytes: int, stream: int = 0):
    _check(_lib.kv_probe_memcpy(dst, src, nbytes, stream or None))


class KVPool:
    """A pool of regions with bandwidth weights (kv_pool_create ... kv_pool_destroy).

    Every method is one entry point of include/kvpool.h, which documents its
    arguments and errors; failures raise KVPoolError with the library's code
    and message.  A minimal round trip::

        import torch
        from paper_2606_14779_amd import kvpool as K
        spec = K.KVSpec(num_layers=32, num_kv_heads=8, head_dim=128)          # 2 MiB blocks
        pool = K.KVPool([K.Region("host", 8 << 30), K.Region("staging", 2 << 30)], [4, 1], spec, device=0)
        cache = torch.randn(32, 2, 1024, 8, 16, 128, device="cuda").to(torch.bfloat16)
        k = [cache[l, 0].data_ptr() for l in range(32)]
        v = [cache[l, 1].data_ptr() for l in range(32)]
        m = pool.place(7, 100)                                  # Eq. 2 counts, striped map
        s = torch.cuda.current_stream().cuda_stream
        pool.store(m, list(range(100)), 1024, k, v, s)          # offload slots 0..99
        pool.retrieve_request(7, list(range(200, 300)), 1024, k, v, s)   # back into slots 200..299
        torch.cuda.synchronize()
        assert torch.equal(cache[:, :, 200:300], cache[:, :, :100])
        pool.release(7)
        pool.close()

    Options: set_launch(K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA) moves the
    host-link bytes by the copy engines; retrieve_layers / store_layers move a
    layer range; a map may concatenate several requests (one call per batch).
    """

    def __init__(self, regions, bandwidths, spec: KVSpec, device: int = 0):
        n = len(regions)
        descs = (_RegionDesc * n)()
        paths = (ctypes.c_char_p * n)()
        for i, r in enumerate(regions):
            kind = {"host": REGION_HOST, "staging": REGION_STAGING, "file": REGION_FILE}[r.kind]
            descs[i] = _struct(_RegionDesc, kind, r.numa_node, r.capacity_bytes, r.coherence, 0)
            paths[i] = os.fsencode(r.path) if r.path is not None else None
        bw = None if bandwidths is None else _int_array(bandwidths, np.uint64, "bandwidths")
        if bw is not None and len(bw) != n:
            raise ValueError("one bandwidth per region")
        self.spec = spec
        self.n_regions = n
        cs = _struct(_KVSpec, spec.num_layers, spec.num_kv_heads, spec.head_dim, spec.block_size,
                     spec.elem_bytes, spec.pool_layout)
        h = ctypes.c_void_p()
        _check(_lib.kv_pool_create_files(ctypes.addressof(descs), None if bw is None else bw.ctypes.data, n,
                                         ctypes.addressof(cs), device, ctypes.addressof(paths), ctypes.byref(h)))
        self._h = h
        _live_pools.add(self)

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            _lib.kv_pool_destroy(self._h)
            self._h = ctypes.c_void_p()
        _live_pools.discard(self)

    def __del__(self):
        try:
            self.close()
        except Exception:   # interpreter shutdown: module globals may already be gone
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # ---- placement / GLT
    def place(self, request: int, n_blocks: int) -> np.ndarray:
        n_blocks = _block_count(n_blocks)
        out = np.zeros(max(n_blocks, 1), dtype=LOC_DTYPE)
        _check(_lib.kv_pool_place(self._h, request, n_blocks, out.ctypes.data))
        return out[:n_blocks]

    def extend(self, request: int, n_new: int) -> np.ndarray:
        """Entries of the request's next n_new blocks, placed as an offload set of their own."""
        n_new = _block_count(n_new)
        out = np.zeros(max(n_new, 1), dtype=LOC_DTYPE)
        _check(_lib.kv_pool_extend(self._h, request, n_new, out.ctypes.data))
        return out[:n_new]

    def lookup(self, request: int, n_blocks: int) -> np.ndarray:
        n_blocks = _block_count(n_blocks)
        out = np.zeros(max(n_blocks, 1), dtype=LOC_DTYPE)
        _check(_lib.kv_pool_lookup(self._h, request, n_blocks, out.ctypes.data))
        return out[:n_blocks]

    def release(self, request: int) -> None:
        _check(_lib.kv_pool_release(self._h, request))

    # ---- data path
    def _transfer(self, fn, loc_map, table, num_slots, k_ptrs, v_ptrs, stream, layers=None):
        m = _loc_array(loc_map)
        t = _int_array(table, np.int32, "block table")
        if len(m) != len(t):
            raise ValueError("map and block table differ in length")
        ks, vs = _ptrs(k_ptrs), _ptrs(v_ptrs)
        if len(ks) != self.spec.num_layers or len(vs) != self.spec.num_layers:
            raise ValueError("one K and one V pointer per layer")
        args = [self._h, m.ctypes.data if len(m) else None, len(m), t.ctypes.data if len(t) else None, num_slots]
        if layers is not None:
            args += [layers[0], layers[1]]
        _check(fn(*args, ctypes.addressof(ks), ctypes.addressof(vs), stream or None))

    def store(self, loc_map, src_table, src_num_slots: int, k_ptrs, v_ptrs, stream: int = 0):
        self._transfer(_lib.kv_pool_store, loc_map, src_table, src_num_slots, k_ptrs, v_ptrs, stream)

    def retrieve(self, loc_map, dst_table, dst_num_slots: int, k_ptrs, v_ptrs, stream: int = 0):
        self._transfer(_lib.kv_pool_retrieve, loc_map, dst_table, dst_num_slots, k_ptrs, v_ptrs, stream)

    def retrieve_noalloc(self, loc_map, dst_table, dst_num_slots: int, k_ptrs, v_ptrs, stream: int = 0):
        self._transfer(_lib.kv_pool_retrieve_noalloc, loc_map, dst_table, dst_num_slots, k_ptrs, v_ptrs, stream)

    def retrieve_request(self, request: int, dst_table, dst_num_slots: int, k_ptrs, v_ptrs, stream: int = 0):
        t = _int_array(dst_table, np.int32, "block table")
        ks, vs = _ptrs(k_ptrs), _ptrs(v_ptrs)
        if len(ks) != self.spec.num_layers or len(vs) != self.spec.num_layers:
            raise ValueError("one K and one V pointer per layer")
        _check(_lib.kv_pool_retrieve_request(self._h, request, len(t), t.ctypes.data if len(t) else None,
                                             dst_num_slots, ctypes.addressof(ks), ctypes.addressof(vs),
                                             stream or None))

    def retrieve_layers(self, loc_map, dst_table, dst_num_slots: int, layer_begin: int, layer_end: int,
                        k_ptrs, v_ptrs, stream: int = 0):
        self._transfer(_lib.kv_pool_retrieve_layers, loc_map, dst_table, dst_num_slots, k_ptrs, v_ptrs, stream,
                       (layer_begin, layer_end))

    def store_layers(self, loc_map, src_table, src_num_slots: int, layer_begin: int, layer_end: int,
                     k_ptrs, v_ptrs, stream: int = 0):
        self._transfer(_lib.kv_pool_store_layers, loc_map, src_table, src_num_slots, k_ptrs, v_ptrs, stream,
                       (layer_begin, layer_end))

    # ---- introspection
    def region_info(self, region: int) -> dict:
        info = _RegionInfo()
        _check(_lib.kv_pool_region_info(self._h, region, ctypes.byref(info)))
        return {k: getattr(info, k) for k, _ in _RegionInfo._fields_}

    def region_read(self, region: int, offset: int, nbytes: int, out: np.ndarray | None = None) -> np.ndarray:
        if out is None:
            out = np.empty(nbytes, dtype=np.uint8)
        if not (out.flags.c_contiguous and out.nbytes >= nbytes):
            raise ValueError("out must be C-contiguous and hold nbytes")
        _check(_lib.kv_pool_region_read(self._h, region, offset, nbytes, out.ctypes.data))
        return out

    # ---- measured bandwidths
    def measure_bandwidth(self, probe_bytes: int = 256 << 20, flags: int = 0) -> np.ndarray:
        out = np.zeros(self.n_regions, dtype=np.uint64)
        _check(_lib.kv_pool_measure_bandwidth(self._h, probe_bytes, flags, out.ctypes.data))
        return out

    def set_bandwidths(self, bandwidths) -> None:
        bw = _int_array(bandwidths, np.uint64, "bandwidths")
        if len(bw) != self.n_regions:
            raise ValueError("one bandwidth per region")
        _check(_lib.kv_pool_set_bandwidths(self._h, bw.ctypes.data))

    # ---- launch configuration and timing
    def set_launch(self, cls: int, op: int, grid: int = 0, flags: int = 0) -> None:
        _check(_lib.kv_pool_set_launch(self._h, cls, op, grid, flags))

    def set_file_ring(self, slot_bytes: int) -> None:
        _check(_lib.kv_pool_set_file_ring(self._h, slot_bytes))

    def set_copy_ring(self, slot_bytes: int) -> None:
        _check(_lib.kv_pool_set_copy_ring(self._h, slot_bytes))

    def set_timing(self, enable: bool) -> None:
        _check(_lib.kv_pool_set_timing(self._h, 1 if enable else 0))

    def last_timing(self) -> dict:
        t = _Timing()
        _check(_lib.kv_pool_last_timing(self._h, ctypes.byref(t)))
        return {k: getattr(t, k) for k, _ in _Timing._fields_}

    def timing_summary(self) -> dict:
        t = _TimingSummary()
        _check(_lib.kv_pool_timing_summary(self._h, ctypes.byref(t)))
        return {k: getattr(t, k) for k, _ in _TimingSummary._fields_ if k != "reserved"}


def allowed_numa_nodes() -> list[int]:
    """NUMA nodes this process may allocate on (online nodes within Mems_allowed)."""
    def parse(s):
        out = set()
        for part in s.strip().split(","):
            if not part:
                continue
            if "-" in part:
                a, b = part.split("-")
                out.update(range(int(a), int(b) + 1))
            else:
                out.add(int(part))
        return out
    try:
        online = parse(open("/sys/devices/system/node/online").read())
    except OSError:
        online = {0}
    allowed = online
    try:
        for line in open("/proc/self/status"):
            if line.startswith("Mems_allowed_list:"):
                allowed = parse(line.split(":", 1)[1])
    except OSError:
        pass
    nodes = sorted(online & allowed)
    return nodes or [0]

"""Set one synthetic workload up on a GPU through the library.

A ``WorkloadRun`` owns the pool (``kv_pool_create``), the engine's source and
destination paged caches (torch tensors: device memory only), the placement
maps (``kv_pool_place``) and the offload (``kv_pool_store``).  Retrieval is a
single ``kv_pool_retrieve_request`` call per request (``kv_pool_retrieve``
with an explicit map when part of the context is absent).  The tests and the bench drive
the hot path through this class; it performs no copy of its own besides
putting the seeded source values into GPU memory.
"""
from __future__ import annotations

import numpy as np

import kvgen
from kvgen.workloads import Workload

from . import kvpool as K

SENTINEL = 0x7FA5  # a bf16 NaN pattern that the generator never produces


class WorkloadRun:
    def __init__(self, wl: Workload, device: int = 0, coherence: int = K.HOST_DEFAULT, numa_nodes=None,
                 file_dir=None, file_flags: int = 0):
        import os
        import tempfile
        import torch
        self.torch = torch
        self.wl = wl
        self.device = device
        sh = wl.shape
        nodes = list(numa_nodes) if numa_nodes else K.allowed_numa_nodes()
        self.regions = []
        self.file_paths = []
        for i, r in enumerate(wl.regions):
            if r.kind == "host":
                node = nodes[r.numa % len(nodes)] if r.numa >= 0 else -1
                self.regions.append(K.Region("host", r.capacity_bytes, node, coherence))
            elif r.kind == "file":     # a new file per region, created and removed by the pool
                path = os.path.join(file_dir or tempfile.gettempdir(),
                                    "kvpool-%d-%x-region%d.bin" % (os.getpid(), id(self), i))
                self.file_paths.append(path)
                self.regions.append(K.Region("file", r.capacity_bytes, -1, file_flags, path))
            else:
                self.regions.append(K.Region("staging", r.capacity_bytes))
        self.weights = [r.weight for r in wl.regions]
        self.spec = K.KVSpec(sh.layers, sh.kv_heads, sh.head_dim, sh.block_size, sh.elem_bytes, wl.layout)
        self.pool = K.KVPool(self.regions, self.weights, self.spec, device)
        dev = torch.device("cuda", device)
        shape = (sh.layers, 2)
        tail = (sh.kv_heads, sh.block_size, sh.head_dim)
        self.src = torch.empty(shape + (wl.src_num_slots,) + tail, dtype=torch.int16, device=dev)
        self.dst = torch.empty(shape + (wl.dst_num_slots,) + tail, dtype=torch.int16, device=dev)
        self._ptrs = {}           # id(cache) -> (K pointers, V pointers), computed once
        self.maps = {}            # request_id -> placed map (present prefix)
        self.retrieve_maps = {}   # request_id -> map of the whole context (absent tail)
        self._batch = None        # concatenated maps and tables of all requests (retrieve_batch)
        # one caller stream per concurrent request; a single-stream workload uses the current stream
        self.streams = [torch.cuda.Stream(device=dev) for _ in range(wl.n_streams)] if wl.n_streams > 1 else []

    # ---- pointers
    def layer_ptrs(self, cache):
        """Per-layer K and V base addresses of a [L][2][slots][H][bs][D] cache (cached per tensor)."""
        key = (cache.data_ptr(), tuple(cache.shape))
        if key not in self._ptrs:
            L = cache.shape[0]
            self._ptrs[key] = (tuple(cache[l, 0].data_ptr() for l in range(L)),
                               tuple(cache[l, 1].data_ptr() for l in range(L)))
        return self._ptrs[key]

    # ---- setup steps
    def fill_source(self, threads=None, keep_host=False):
        """Seeded values of every present block into the source cache (host generate, then copy)."""
        sh = self.wl.shape
        host = np.empty(tuple(self.src.shape), dtype=np.uint16)
        kp = [host[l, 0].ctypes.data for l in range(sh.layers)]
        vp = [host[l, 1].ctypes.data for l in range(sh.layers)]
        for q in self.wl.requests:
            kvgen.fill_cache(self.wl.seed, q.request_id, np.arange(q.n_present, dtype=np.uint64), q.src_slots,
                             sh.layers, sh.kv_heads, sh.block_size, sh.head_dim, kp, vp, threads)
        self.src.copy_(self.torch.from_numpy(host.view(np.int16)))
        self.torch.cuda.synchronize(self.device)
        return host if keep_host else None

    def fill_dst(self, value=SENTINEL):
        self.dst.fill_(np.int16(np.uint16(value).view(np.int16)).item())

    def place_all(self):
        self._batch = None
        for q in self.wl.requests:
            m = self.pool.place(q.request_id, q.n_present)
            self.maps[q.request_id] = m
            full = np.zeros(q.n_blocks, dtype=K.LOC_DTYPE)
            full[:q.n_present] = m
            full["region"][q.n_present:] = K.ABSENT
            self.retrieve_maps[q.request_id] = full

    def store_all(self, stream=None):
        kp, vp = self.layer_ptrs(self.src)
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        for q in self.wl.requests:
            self.pool.store(self.maps[q.request_id], q.src_slots, self.wl.src_num_slots, kp, vp, s.cuda_stream)

    def retrieve(self, q, stream=None):
        """One request: by request id (GLT lookup inside the library) when the
        whole context is present, else with the map whose tail is absent."""
        kp, vp = self.layer_ptrs(self.dst)
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        if q.n_present == q.n_blocks:
            self.pool.retrieve_request(q.request_id, q.dst_slots, self.wl.dst_num_slots, kp, vp, s.cuda_stream)
        else:
            self.pool.retrieve(self.retrieve_maps[q.request_id], q.dst_slots, self.wl.dst_num_slots, kp, vp,
                               s.cuda_stream)

    def retrieve_batch(self, stream=None):
        """Every request in one kv_pool_retrieve call: the maps (absent tails included) and the
        destination tables concatenated."""
        kp, vp = self.layer_ptrs(self.dst)
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        if self._batch is None:
            m = np.concatenate([self.retrieve_maps[q.request_id] for q in self.wl.requests])
            t = np.concatenate([q.dst_slots for q in self.wl.requests]).astype(np.int32)
            self._batch = (m, t)
        m, t = self._batch
        self.pool.retrieve(m, t, self.wl.dst_num_slots, kp, vp, s.cuda_stream)

    def retrieve_all(self):
        """One retrieve per request; request i on stream i % n_streams (forked from the current stream)."""
        torch = self.torch
        cur = torch.cuda.current_stream(self.device)
        if len(self.streams) <= 1:
            for q in self.wl.requests:
                self.retrieve(q, cur)
            return
        for s in self.streams:
            s.wait_stream(cur)
        for i, q in enumerate(self.wl.requests):
            self.retrieve(q, self.streams[q.stream % len(self.streams)])
        for s in self.streams:
            cur.wait_stream(s)

    def setup(self, threads=None, keep_host=False):
        host = self.fill_source(threads, keep_host)
        self.fill_dst()
        self.place_all()
        self.store_all()
        self.torch.cuda.synchronize(self.device)
        return host

    def close(self):
        self.pool.close()
        self.src = self.dst = None

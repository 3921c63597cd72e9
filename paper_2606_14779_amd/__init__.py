"""MI355X-native KV-cache retrieval from a bandwidth-striped KV pool.

The product is ``libkvpool.so`` (C ABI in ``include/kvpool.h``; HIP kernels
for gfx950 under ``csrc/``).  ``kvpool`` is its thin ctypes binding.
"""
from .kvpool import (KVPool, KVPoolError, KVSpec, Region, allowed_numa_nodes, counts,  # noqa: F401
                     probe_copy_kernel, probe_memcpy, LOC_DTYPE, ABSENT, EXPORTED)

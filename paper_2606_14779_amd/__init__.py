"""MI355X-native KV-cache retrieval from a bandwidth-striped KV pool.

The product is ``libkvpool.so`` (C ABI in ``include/kvpool.h``; HIP kernels
for gfx950 under ``csrc/``).  ``kvpool`` is its thin ctypes binding; it is
loaded on first use so that ``build`` can run before the library exists.
"""

_BINDING = ("KVPool", "KVPoolError", "KVSpec", "Region", "allowed_numa_nodes", "counts",
            "probe_copy_kernel", "probe_memcpy", "LOC_DTYPE", "ABSENT", "EXPORTED")


def __getattr__(name):
    if name in _BINDING:
        from . import kvpool
        return getattr(kvpool, name)
    raise AttributeError(name)

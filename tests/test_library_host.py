"""Host-side checks of libkvpool.so that need no GPU.

- every function the header declares is exported;
- placement in the library (placement-only pools make no HIP call) equals the
  oracle's placement bit for bit over random place/release sequences;
- argument validation returns the documented error codes.
"""
import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
from paper_2606_14779_amd import kvpool as K

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "kvpool.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kv_\w+)\s*\(", src)))


def test_header_symbols_exported():
    names = _declared_functions()
    assert len(names) >= 16
    lib = ctypes.CDLL(K.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(K.EXPORTED)


def _pool(weights, caps, bb_layers=1):
    spec = K.KVSpec(bb_layers, 1, 8, 16, 2, 0)      # chunk 256 B, block 512*L B
    regions = [K.Region("host" if i % 2 == 0 else "staging", c, -1) for i, c in enumerate(caps)]
    return K.KVPool(regions, weights, spec, device=-1), spec


def test_counts_match_oracle_random():
    rng = np.random.default_rng(1)
    for _ in range(500):
        N = int(rng.integers(1, 9))
        w = rng.integers(1, 1 << 40, size=N, dtype=np.uint64)
        n = int(rng.integers(0, 1 << 40))
        assert np.array_equal(K.counts(w, n), oracle.counts(w, n))


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(1, 9), min_size=1, max_size=6), st.integers(1, 4),
       st.lists(st.tuples(st.booleans(), st.integers(1, 90)), min_size=1, max_size=30))
def test_placement_equals_oracle(weights, layers, ops):
    bb = 2 * layers * 256
    caps = [(w * 60 + 7) * bb + 3000 for w in weights]
    lib_pool, spec = _pool(weights, caps, layers)
    assert spec.block_bytes == bb
    ora = oracle.Pool(weights, caps, bb)
    live, req = [], 100
    for is_release, n in ops:
        if is_release and live:
            r = live.pop(n % len(live))
            assert ora.release(r) == 0
            lib_pool.release(r)
            continue
        rc, om = ora.try_place(req, n)
        if rc == 0:
            lm = lib_pool.place(req, n)
            assert np.array_equal(lm.view(np.uint8), om.view(np.uint8))
            assert np.array_equal(lib_pool.lookup(req, n), om)
            live.append(req)
        else:
            with pytest.raises(K.KVPoolError) as ei:
                lib_pool.place(req, n)
            assert ei.value.code == rc == -3
        req += 1
    lib_pool.close()


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(1, 9), min_size=1, max_size=6), st.integers(1, 3),
       st.lists(st.tuples(st.sampled_from(["place", "extend", "extend", "release"]), st.integers(1, 60)),
                min_size=1, max_size=40))
def test_placement_with_extensions_equals_oracle(weights, layers, ops):
    """Place, extend (the next offload set of a placed request) and release in random order: every
    map, every full lookup and every refusal as the oracle's."""
    bb = 2 * layers * 256
    caps = [(w * 40 + 7) * bb + 3000 for w in weights]
    lib_pool, _ = _pool(weights, caps, layers)
    ora = oracle.Pool(weights, caps, bb)
    live, req = {}, 100                           # request -> blocks placed so far
    for op, n in ops:
        if op == "release" and live:
            r = sorted(live)[n % len(live)]
            del live[r]
            assert ora.release(r) == 0
            lib_pool.release(r)
        elif op == "extend" and live:
            r = sorted(live)[n % len(live)]
            rc, om = ora.try_extend(r, n)
            if rc == 0:
                lm = lib_pool.extend(r, n)
                assert np.array_equal(lm.view(np.uint8), om.view(np.uint8))
                live[r] += n
            else:
                with pytest.raises(K.KVPoolError) as ei:
                    lib_pool.extend(r, n)
                assert ei.value.code == rc == -3
            assert np.array_equal(lib_pool.lookup(r, live[r]), ora.lookup(r, live[r]))
        else:
            rc, om = ora.try_place(req, n)
            if rc == 0:
                assert np.array_equal(lib_pool.place(req, n).view(np.uint8), om.view(np.uint8))
                live[req] = n
            else:
                with pytest.raises(K.KVPoolError) as ei:
                    lib_pool.place(req, n)
                assert ei.value.code == rc == -3
            req += 1
    lib_pool.close()


def test_extend_errors():
    p, spec = _pool([2, 1], [8 * 4096, 4 * 4096], bb_layers=8)  # one block = one 4096-byte sector
    assert spec.block_bytes == 4096
    m = p.place(1, 6)
    assert _err(p.extend, 2, 3) == "NOTFOUND"
    assert _err(p.extend, 1, 0) == "INVALID"
    assert _err(p.extend, 1, 9) == "NOSPACE"                    # device 0 has room for 4 more only
    assert np.array_equal(p.lookup(1, 6), m)                     # nothing changed
    e = p.extend(1, 3)
    assert list(e["region"]) == [0, 1, 0] and set(e["gen"].tolist()) == {int(m["gen"][0])}
    assert np.array_equal(p.lookup(1, 9), np.concatenate([m, e]))
    assert _err(p.lookup, 1, 6) == "INVALID"                      # the count is now 9
    p.release(1)
    assert _err(p.extend, 1, 1) == "NOTFOUND"
    assert p.place(2, 12) is not None                            # every range came back
    p.close()


def test_maximum_counts():
    """The largest counts the ABI takes: 2^32-1 blocks are refused for room, and a request cannot grow
    past 2^32-1 blocks in all; nothing changes either way."""
    p, spec = _pool([3, 1], [1 << 20, 1 << 20])
    one = np.zeros(1, dtype=K.LOC_DTYPE)        # the library refuses before it writes the map
    raw = lambda fn, req, n: K.ERRORS.get(fn(p._h, req, n, one.ctypes.data), "OK")   # noqa: E731
    assert raw(K._lib.kv_pool_place, 1, 2 ** 32 - 1) == "NOSPACE"
    m = p.place(1, 5)
    assert raw(K._lib.kv_pool_extend, 1, 2 ** 32 - 5) == "INVALID"
    assert raw(K._lib.kv_pool_extend, 1, 2 ** 32 - 6) == "NOSPACE"
    assert np.array_equal(p.lookup(1, 5), m)
    p.close()


def test_extension_uses_the_current_weights():
    """After kv_pool_set_bandwidths, an extension is placed by the new weights, as a new placement is;
    the request's earlier blocks stay where they were."""
    p, spec = _pool([1, 1], [1 << 20, 1 << 20])
    first = p.place(1, 4)
    assert list(first["region"]) == [0, 1, 0, 1]
    p.set_bandwidths([1, 3])
    ext = p.extend(1, 4)
    assert sorted(ext["region"].tolist()) == [0, 1, 1, 1]          # Eq. 2 with the new weights
    assert np.array_equal(p.lookup(1, 8), np.concatenate([first, ext]))
    p.close()


def test_workload_scale_placement_equals_oracle():
    from kvgen import workloads
    for cfg in (1, 2, 3, 4, 5):
        wl = workloads.make(cfg)
        bb = wl.shape.block_bytes
        w = [r.weight for r in wl.regions]
        caps = [r.capacity_bytes for r in wl.regions]
        spec = K.KVSpec(wl.shape.layers, wl.shape.kv_heads, wl.shape.head_dim)
        lp = K.KVPool([K.Region(r.kind, r.capacity_bytes) for r in wl.regions], w, spec, device=-1)
        op = oracle.Pool(w, caps, bb)
        for q in wl.requests:
            assert np.array_equal(lp.place(q.request_id, q.n_present), op.place(q.request_id, q.n_present))
        lp.close()


def _err(fn, *a):
    with pytest.raises(K.KVPoolError) as ei:
        fn(*a)
    return ei.value.name


def test_create_validation():
    spec = K.KVSpec(2, 2, 8)
    ok = [K.Region("host", 1 << 20)]
    assert _err(K.KVPool, ok, [0], spec, -1) == "INVALID"                    # zero bandwidth
    assert _err(K.KVPool, [K.Region("host", 100)], [1], spec, -1) == "INVALID"  # below a sector
    assert _err(K.KVPool, ok, [1], K.KVSpec(2, 1, 3, 1, 2, 0), -1) == "INVALID"  # chunk 6 B
    assert _err(K.KVPool, ok, [1], K.KVSpec(2, 4, 4, 16, 2, 1), -1) == "INVALID"  # token-major row 8 B
    assert _err(K.KVPool, ok, [1], K.KVSpec(0, 2, 8), -1) == "INVALID"
    assert _err(K.KVPool, ok, [1], K.KVSpec(2, 2, 8, 16, 2, 2), -1) == "INVALID"  # layout 2
    assert _err(K.KVPool, [K.Region("staging", 1 << 20, 0)], [1], spec, -1) == "INVALID"
    assert _err(K.KVPool, [K.Region("host", 1 << 20, -2)], [1], spec, -1) == "INVALID"
    assert _err(K.KVPool, [], [], spec, -1) == "INVALID"
    assert _err(K.KVPool, ok, [1], spec, -5) == "INVALID"


def test_place_lookup_release_errors():
    p, spec = _pool([1, 1], [1 << 20, 1 << 20])
    assert _err(p.place, 1, 0) == "INVALID"
    m = p.place(1, 5)
    assert _err(p.place, 1, 5) == "INVALID"
    assert _err(p.lookup, 1, 4) == "INVALID"
    assert _err(p.lookup, 2, 5) == "NOTFOUND"
    assert _err(p.release, 2) == "NOTFOUND"
    assert _err(p.place, 3, 10 ** 6) == "NOSPACE"
    assert np.array_equal(p.lookup(1, 5), m)
    p.release(1)
    assert _err(p.lookup, 1, 5) == "NOTFOUND"
    # gen keeps counting across failures and releases
    assert int(p.place(4, 1)["gen"][0]) == 2
    p.close()


def test_transfers_rejected_without_device():
    p, spec = _pool([1], [1 << 20])
    m = p.place(1, 2)
    ptrs = [16 * 1024] * spec.num_layers
    assert _err(p.retrieve, m, [0, 1], 2, ptrs, ptrs) == "INVALID"
    assert _err(p.store, m, [0, 1], 2, ptrs, ptrs) == "INVALID"
    assert _err(p.set_timing, True) == "INVALID"
    assert _err(p.set_launch, 2, 0, 0, 0) == "INVALID"
    assert _err(p.set_launch, 0, 0, 0, 512) == "INVALID"                                     # unknown flag
    p.set_launch(0, 0, 64, K.LAUNCH_NT_LOAD)
    assert _err(p.set_launch, K.CLASS_HOST, K.OP_RETRIEVE, 0, K.LAUNCH_SDMA) == "INVALID"   # nothing to copy with
    assert _err(p.set_launch, K.CLASS_STAGING, K.OP_STORE, 0, K.LAUNCH_SDMA) == "INVALID"  # host class only
    assert _err(p.set_copy_ring, 1 << 20) == "INVALID"                                     # no device
    info = p.region_info(0)
    assert info["device_ptr"] is None and info["capacity_bytes"] == 1 << 20
    assert _err(p.region_info, 1) == "INVALID"
    assert _err(p.region_read, 0, 0, 16) == "INVALID"
    p.close()


def test_binding_rejects_integers_outside_their_c_type():
    """ctypes would wrap -1 to 2^32-1 (a slot count every table entry passes); the binding refuses it
    before the call, for every integer argument of every entry point."""
    p, spec = _pool([1], [1 << 20])
    ptrs = [16 * 1024] * spec.num_layers
    with pytest.raises(ValueError, match="outside"):
        p.place(1, -1)
    with pytest.raises(ValueError, match="outside"):
        p.place(-1, 2)
    with pytest.raises(ValueError, match="outside"):
        p.extend(1, 2 ** 32)
    m = p.place(1, 2)
    with pytest.raises(ValueError, match="outside"):
        p.retrieve(m, [0, 1], -1, ptrs, ptrs)
    with pytest.raises(ValueError, match="outside"):
        p.retrieve_layers(m, [0, 1], 2, 0, -1, ptrs, ptrs)
    with pytest.raises(ValueError, match="outside"):
        p.region_read(0, -16, 16)
    with pytest.raises(ValueError, match="outside"):
        K.counts([1, 1], -5)
    with pytest.raises(ValueError, match="outside"):
        p.set_launch(0, 0, 2 ** 32, 0)
    for name, (_, args) in K._SIGS.items():                       # every wrapper checks
        ints = [i for i, t in enumerate(args) if t in K._RANGES]
        if not ints:
            continue
        call = [None if t is K._vp else 0 for t in args]
        call[ints[-1]] = K._RANGES[args[ints[-1]]][1]                   # one past the type's maximum
        with pytest.raises(ValueError, match=name):
            getattr(K._lib, name)(*call)
    with pytest.raises(ValueError, match="block table"):            # int64 table: checked, not wrapped
        p.retrieve(m, np.array([0, 2 ** 32 + 1], np.int64), 2, ptrs, ptrs)
    with pytest.raises(ValueError, match="bandwidths"):
        p.set_bandwidths(np.array([-1], np.int64))
    with pytest.raises(ValueError, match="capacity_bytes"):
        K.KVPool([K.Region("host", -4096)], [1], spec, device=-1)
    with pytest.raises(ValueError, match="num_layers"):
        K.KVPool([K.Region("host", 1 << 20)], [1], K.KVSpec(-1, 1, 8), device=-1)
    assert np.array_equal(p.lookup(1, 2), m)                      # nothing reached the pool
    p.close()


def test_glt_survives_many_requests():
    """Table growth and backward-shift deletion keep every lookup exact."""
    p, spec = _pool([3, 1, 2], [1 << 34] * 3)
    rng = np.random.default_rng(0)
    maps = {}
    for r in range(400):
        n = int(rng.integers(1, 60))
        maps[r] = p.place(r, n)
        if r % 3 == 0:
            victim = int(rng.choice(list(maps)))
            p.release(victim)
            del maps[victim]
    for r, m in maps.items():
        assert np.array_equal(p.lookup(r, len(m)), m)
    p.close()


def test_set_bandwidths_changes_later_placements():
    p, spec = _pool([1, 1, 1], [1 << 24] * 3)
    p.set_bandwidths([5, 1, 2])
    ora = oracle.Pool([5, 1, 2], [1 << 24] * 3, spec.block_bytes)
    assert np.array_equal(p.place(1, 41), ora.place(1, 41))
    assert _err(p.set_bandwidths, [1, 0, 1]) == "INVALID"
    with pytest.raises(ValueError):
        p.set_bandwidths([1, 1])
    assert _err(p.measure_bandwidth) == "INVALID"          # no memory to measure
    p.close()
    with pytest.raises(K.KVPoolError):
        K.KVPool([K.Region("host", 1 << 20)], None, K.KVSpec(1, 1, 8), device=-1)


def test_placement_from_threads_keeps_invariants():
    """place / lookup / release from several threads: every live map stays valid."""
    import threading
    weights = [4, 4, 1, 1, 1, 1]
    bb = 512
    caps = [1 << 26] * 6
    p = K.KVPool([K.Region("host", c) for c in caps], weights, K.KVSpec(1, 1, 8), device=-1)
    live, lock, errs = {}, threading.Lock(), []

    def work(t):
        rng = np.random.default_rng(t)
        try:
            for i in range(150):
                req = t * 100000 + i
                n = int(rng.integers(1, 300))
                m = p.place(req, n)
                assert np.array_equal(p.lookup(req, n), m)
                with lock:
                    live[req] = m
                if rng.random() < 0.4:
                    with lock:
                        victim = live.pop(req)
                    p.release(req)
                    assert len(victim) == n
        except Exception as e:            # reported below
            errs.append(e)

    ts = [threading.Thread(target=work, args=(t,)) for t in range(6)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errs, errs
    spans = [[] for _ in weights]
    gens = set()
    for req, m in live.items():
        c = oracle.counts(weights, len(m))
        reg = m["region"].astype(np.int64)
        assert list(np.bincount(reg, minlength=6)) == [int(x) for x in c]
        gens.add(int(m["gen"][0]))
        for i in range(6):
            offs = np.sort(m["offset"][reg == i].astype(np.int64))
            if len(offs):
                assert np.all(offs == offs[0] + bb * np.arange(len(offs)))
                spans[i].append((int(offs[0]), int(offs[-1]) + bb))
        assert np.array_equal(p.lookup(req, len(m)), m)
    assert len(gens) == len(live)
    for s in spans:
        s.sort()
        assert all(a[1] <= b[0] for a, b in zip(s, s[1:]))
    p.close()


def test_header_is_c99_and_callable_from_c(tmp_path):
    """include/kvpool.h is plain C: a C99 program (-pedantic -Werror) includes it, links the library
    and places and extends a request on a placement-only pool."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("needs gcc")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    src = tmp_path / "c_client.c"
    src.write_text(r"""
#include "kvpool.h"
#include <stdio.h>
int main(void)
{
    kvp_kv_spec spec = {2, 1, 8, 16, 2, 0};
    kvp_region_desc r = {KVP_REGION_HOST, -1, 1u << 20, KVP_HOST_DEFAULT, 0};
    uint64_t bw = 1;
    kvp_pool *p = NULL;
    kvp_loc m[5];
    if (kv_pool_create(&r, &bw, 1, &spec, -1, &p) != KVP_OK) { printf("%s\n", kv_pool_last_error()); return 1; }
    if (kv_pool_place(p, 1, 3, m) != KVP_OK || kv_pool_extend(p, 1, 2, m + 3) != KVP_OK) return 2;
    if (kv_pool_lookup(p, 1, 5, m) != KVP_OK || kv_pool_lookup(p, 1, 4, m) != KVP_ERR_INVALID) return 3;
    kv_pool_destroy(p);
    printf("c client ok\n");
    return 0;
}
""")
    exe = str(tmp_path / "c_client")
    lib_dir = os.path.dirname(K.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(root, "include"),
                    str(src), "-o", exe, "-L", lib_dir, "-lkvpool", "-Wl,-rpath," + lib_dir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and "c client ok" in r.stdout, r.stdout + r.stderr


def test_binding_raises_without_the_library(tmp_path):
    """No fallback: the binding, imported from a package directory that holds no libkvpool.so,
    raises ImportError instead of loading anything else."""
    import shutil
    import subprocess
    import sys
    pkg = tmp_path / "kvp_copy"
    pkg.mkdir()
    (pkg / "__init__.py").write_text("")
    shutil.copy(os.path.join(ROOT, "paper_2606_14779_amd", "kvpool.py"), pkg / "kvpool.py")
    r = subprocess.run([sys.executable, "-c", "import kvp_copy.kvpool"], cwd=tmp_path, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "libkvpool.so is not built" in r.stderr, r.stderr

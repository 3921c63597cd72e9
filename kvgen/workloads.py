"""The five synthetic retrieval workloads, as data.

Each workload fixes a KV shape (layers, KV heads, head_dim, 16-token blocks,
bf16), a set of pool regions (pinned host or HBM staging, with integer
bandwidth weights and a logical NUMA node), and one or more requests with
their source and destination block tables.  Everything random is drawn from
seeded streams (``kvgen.subseed(seed, tag)``), so a workload is a pure
function of its config number and scale.

The paper evaluates on a long-document QA benchmark with inputs of 1K-128K
tokens; only that context-length range is used here.  Values are seeded
N(0,1) bf16 (``kvgen.c``), not model activations.

Nothing here computes the placement: region capacities use only the bound
"a region receives at most floor(w_i * n / W) + 1 blocks of a request",
which holds for any remainder rule that adds at most one block per region.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field

import numpy as np

from . import subseed

SECTOR = 4096  # the allocation granule of every pool region


@dataclass(frozen=True)
class KVShape:
    name: str
    layers: int
    kv_heads: int
    head_dim: int
    block_size: int = 16
    elem_bytes: int = 2

    @property
    def chunk_bytes(self) -> int:
        """Bytes of one (block, layer, K-or-V) chunk: [heads][block_size][head_dim]."""
        return self.kv_heads * self.block_size * self.head_dim * self.elem_bytes

    @property
    def block_bytes(self) -> int:
        """Bytes of one block across all layers, K and V."""
        return 2 * self.layers * self.chunk_bytes

    @property
    def bytes_per_token(self) -> int:
        return self.block_bytes // self.block_size


LLAMA_8B = KVShape("llama3.1-8b", 32, 8, 128)
GPT_OSS_20B = KVShape("gpt-oss-20b", 24, 8, 64)
QWEN3_30B_A3B = KVShape("qwen3-30b-a3b", 48, 4, 128)


@dataclass
class RegionSpec:
    kind: str            # "host" (pinned, zero-copy mapped) or "staging" (HBM)
    weight: int          # bandwidth weight b_i (positive integer)
    numa: int = -1       # logical NUMA node for host regions (-1 = any)
    capacity_bytes: int = 0


@dataclass
class RequestSpec:
    request_id: int
    n_blocks: int               # blocks in the request's context
    n_present: int              # present prefix (placed and stored); the rest is absent
    src_slots: np.ndarray       # int32[n_present], slot of each present block in the source cache
    dst_slots: np.ndarray       # int32[n_blocks], -1 for absent blocks
    stream: int = 0


@dataclass
class Workload:
    cfg: int
    name: str
    seed: int
    shape: KVShape
    layout: int                 # 0: pool chunks head-major; 1: token-major
    regions: list
    requests: list
    src_num_slots: int
    dst_num_slots: int
    occupied_dst_slots: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    n_streams: int = 1

    @property
    def present_blocks(self) -> int:
        return sum(r.n_present for r in self.requests)

    @property
    def retrieved_bytes(self) -> int:
        return self.present_blocks * self.shape.block_bytes

    def describe(self) -> dict:
        return {
            "workload": self.name, "cfg": self.cfg, "seed": self.seed,
            "shape": dataclasses.asdict(self.shape), "layout": self.layout,
            "regions": [(r.kind, r.weight, r.numa, r.capacity_bytes) for r in self.regions],
            "requests": [(q.request_id, q.n_blocks, q.n_present, q.stream) for q in self.requests],
            "src_num_slots": self.src_num_slots, "dst_num_slots": self.dst_num_slots,
            "occupied_dst_slots": int(len(self.occupied_dst_slots)),
        }


def _rng(seed: int, tag: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(subseed(seed, tag)))


def _round_up(x: int, a: int) -> int:
    return (x + a - 1) // a * a


def _size_regions(regions, present_counts, block_bytes, slack_blocks=0):
    """Give each region room for its share of every request (upper bound per request)."""
    total_w = sum(r.weight for r in regions)
    for r in regions:
        cap = 0
        for n in present_counts:
            if n == 0:
                continue
            blocks = r.weight * n // total_w + 1
            cap += _round_up(blocks * block_bytes, SECTOR)
        cap += _round_up(slack_blocks * block_bytes, SECTOR)
        r.capacity_bytes = max(cap, SECTOR)


def _scaled(n_full: int, max_blocks):
    return n_full if max_blocks is None else max(1, min(n_full, max_blocks))


def make(cfg: int, max_blocks: int | None = None, layout: int = 0, seed: int | None = None,
         context_tokens: int | None = None) -> Workload:
    """Build workload ``cfg`` (1..5).

    ``max_blocks`` caps the blocks of each request (same shapes, regions,
    weights and table recipes) for parity cases the oracle finishes in
    seconds; ``None`` gives the full size.  ``context_tokens`` (workload 3
    only) replaces its 128K-token context, keeping every other recipe.
    """
    if context_tokens is not None and cfg != 3:
        raise ValueError("context_tokens applies to workload 3 only")
    seed = 1000 + cfg if seed is None else seed
    if cfg == 1:
        shape = LLAMA_8B
        n = _scaled(16384 // 16, max_blocks)
        regions = [RegionSpec("host", 1, 0), RegionSpec("host", 1, 1)]
        src = _rng(seed, "src").permutation(n).astype(np.int32)
        dst = np.arange(n, dtype=np.int32)                        # identity table
        req = RequestSpec(1, n, n, src, dst)
        wl = Workload(1, "llama3.1-8b-kv-16k-2host", seed, shape, layout, regions, [req], n, n)
    elif cfg == 2:
        shape = LLAMA_8B
        n = _scaled(65536 // 16, max_blocks)
        regions = [RegionSpec("host", 4, 0), RegionSpec("host", 4, 1),
                   RegionSpec("staging", 1), RegionSpec("staging", 1)]
        src = _rng(seed, "src").permutation(n).astype(np.int32)
        dst = _rng(seed, "perm").permutation(n).astype(np.int32)  # permutation of free slots
        req = RequestSpec(1, n, n, src, dst)
        wl = Workload(2, "llama3.1-8b-kv-64k-4region", seed, shape, layout, regions, [req], n, n)
    elif cfg == 3:
        shape = LLAMA_8B
        ctx = 131072 if context_tokens is None else int(context_tokens)
        n = _scaled(ctx // 16, max_blocks)
        regions = [RegionSpec("host", 4, 0), RegionSpec("host", 4, 1)] + \
                  [RegionSpec("staging", 1) for _ in range(4)]
        n_occ = n // 4                      # 8192 blocks -> 10240 slots, 2048 occupied
        slots = n + n_occ
        occ = np.sort(_rng(seed, "frag").choice(slots, size=n_occ, replace=False)).astype(np.int32)
        free = np.setdiff1d(np.arange(slots, dtype=np.int32), occ)   # ascending free slots
        src = _rng(seed, "src").permutation(n).astype(np.int32)
        req = RequestSpec(1, n, n, src, free[:n].astype(np.int32))
        name = "llama3.1-8b-kv-128k-6region" if ctx == 131072 else "llama3.1-8b-kv-%dk-6region" % (ctx // 1024)
        wl = Workload(3, name, seed, shape, layout, regions, [req], n, slots, occupied_dst_slots=occ)
    elif cfg == 4:
        shape = GPT_OSS_20B
        n = _scaled(131072 // 16, max_blocks)
        regions = [RegionSpec("host", 3, 0), RegionSpec("host", 3, 1),
                   RegionSpec("staging", 1), RegionSpec("staging", 1)]
        src = _rng(seed, "src").permutation(n).astype(np.int32)
        dst = _rng(seed, "perm").permutation(n).astype(np.int32)
        req = RequestSpec(1, n, n, src, dst)
        wl = Workload(4, "gpt-oss-20b-kv-128k-4region", seed, shape, layout, regions, [req], n, n)
    elif cfg == 5:
        shape = QWEN3_30B_A3B
        regions = [RegionSpec("host", 4, 0), RegionSpec("host", 4, 1)] + \
                  [RegionSpec("staging", 1) for _ in range(4)]
        ctx_rng, pre_rng = _rng(seed, "ctx"), _rng(seed, "prefix")
        reqs_raw = []
        for i in range(4):
            ctx = int(ctx_rng.integers(16384, 131072 + 1))         # tokens, uniform
            nb = (ctx + shape.block_size - 1) // shape.block_size
            u = float(pre_rng.uniform(0.5, 1.0))
            present = int(np.floor(u * ctx / shape.block_size))
            present = max(1, min(nb, present))
            if max_blocks is not None:                             # shrink, keep the ratio
                scale = min(1.0, max_blocks / nb)
                nb_s = max(1, int(nb * scale))
                present = max(1, min(nb_s, int(present * scale)))
                nb = nb_s
            reqs_raw.append((nb, present))
        total_present = sum(p for _, p in reqs_raw)
        dst_slots_n = total_present + (total_present + 3) // 4      # +25 %
        dst_perm = _rng(seed, "perm").permutation(dst_slots_n).astype(np.int32)
        src_perm = _rng(seed, "src").permutation(total_present).astype(np.int32)
        reqs, at = [], 0
        for i, (nb, present) in enumerate(reqs_raw):
            dst = np.full(nb, -1, dtype=np.int32)
            dst[:present] = dst_perm[at:at + present]
            reqs.append(RequestSpec(i + 1, nb, present, src_perm[at:at + present].copy(), dst, stream=i))
            at += present
        wl = Workload(5, "qwen3-30b-a3b-kv-batch4-6region", seed, shape, layout, regions, reqs,
                      total_present, dst_slots_n, n_streams=4)
    else:
        raise ValueError("workload config must be 1..5, got %r" % (cfg,))
    _size_regions(wl.regions, [r.n_present for r in wl.requests], shape.block_bytes)
    return wl

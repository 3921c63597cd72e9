// KV pool engine: regions, placement bookkeeping, and the store / retrieve
// enqueue path.
//
// Retrieval follows Sec. 4.3 of the paper: look every block up, group the
// blocks by pool device, and read all devices in parallel.  Here the groups
// are the two region classes -- pinned host regions, read by a zero-copy
// kernel over the host link, and HBM staging regions, read by an HBM gather
// kernel -- and "in parallel" means the staging kernel is forked onto an
// internal HIP stream while the host kernel runs on the caller's stream, and
// the two are joined again on the caller's stream, so both kernels run at
// once and the caller sees one stream-ordered operation.  The per-call work list (one
// 16-byte item per block plus the 2L engine-buffer pointers) is written to a
// pinned buffer and uploaded with one asynchronous copy; buffers come from a
// small ring guarded by events, so a call only blocks when the ring wraps
// onto work that is still running.

#include <numaif.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstring>

#include "internal.hpp"

namespace kvp {

void fail(int code, const std::string &msg) { throw Error{code, msg}; }

// A failed HIP call also leaves its code as the thread's last error, which the
// caller's next launch check would report as its own: the library takes it.
void clear_hip_error() { (void)hipGetLastError(); }

void check_hip(hipError_t e, const char *what)
{
    if (e == hipSuccess) return;
    clear_hip_error();
    fail(KVP_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

constexpr uint64_t kSector = 4096;
constexpr uint32_t kRingSlots = 32;
constexpr size_t kSlotMin = 64 * 1024;
constexpr uint64_t kCreateProbeBytes = 256ull << 20;   // per-region read probe when no bandwidths are given
// Staging-class bytes below which the HBM kernel runs on the caller's stream
// ahead of the host-class kernel instead of being forked: forking costs about
// 25 us of host time per call, more than such a kernel takes (32 MiB read and
// written at ~2.5 TB/s copied: ~13 us).
constexpr uint64_t kForkMinBytes = 32ull << 20;

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Make `dev` the calling thread's device for the scope, then restore.
class DeviceScope {
public:
    explicit DeviceScope(int dev)
    {
        if (dev < 0) return;
        check_hip(hipGetDevice(&old_), "hipGetDevice");
        if (old_ != dev) check_hip(hipSetDevice(dev), "hipSetDevice");
        else old_ = -1;
    }
    ~DeviceScope()
    {
        if (old_ >= 0) (void)hipSetDevice(old_);
    }

private:
    int old_ = -1;
};

// Bind the calling thread's memory policy to one NUMA node for the scope.
class NumaScope {
public:
    explicit NumaScope(int node)
    {
        if (node < 0) return;
        if (node >= kMaxNodes) fail(KVP_ERR_INVALID, "NUMA node " + std::to_string(node) + " out of range");
        saved_ = syscall(SYS_get_mempolicy, &old_mode_, old_mask_, kMaxNodes + 1, nullptr, 0) == 0;
        unsigned long mask[kWords] = {};
        mask[node / 64] = 1ul << (node % 64);
        if (syscall(SYS_set_mempolicy, MPOL_BIND, mask, kMaxNodes + 1) != 0)
            fail(KVP_ERR_INVALID, "cannot bind memory to NUMA node " + std::to_string(node) + ": " +
                                      std::strerror(errno));
        active_ = true;
    }
    ~NumaScope()
    {
        if (!active_) return;
        if (saved_ && old_mode_ != MPOL_DEFAULT)
            syscall(SYS_set_mempolicy, old_mode_, old_mask_, kMaxNodes + 1);
        else
            syscall(SYS_set_mempolicy, MPOL_DEFAULT, nullptr, 0);
    }

private:
    static constexpr int kMaxNodes = 1024;
    static constexpr int kWords = kMaxNodes / 64;
    bool active_ = false, saved_ = false;
    int old_mode_ = MPOL_DEFAULT;
    unsigned long old_mask_[kWords] = {};
};

// NUMA node backing the page at p: move_pages() in query mode (no nodes
// given) reports where each page lives; get_mempolicy() is the fallback.
int page_node(void *p)
{
    void *pages[1] = {p};
    int status[1] = {-1};
    if (syscall(SYS_move_pages, 0, 1ul, pages, nullptr, status, 0) == 0 && status[0] >= 0) return status[0];
    int node = -1;
    if (syscall(SYS_get_mempolicy, &node, nullptr, 0, p, MPOL_F_NODE | MPOL_F_ADDR) != 0) return -1;
    return node;
}

void alloc_region(Region &r)
{
    if (r.desc.type == KVP_REGION_HOST) {
        unsigned flags = hipHostMallocMapped;
        const uint32_t coh = r.desc.flags;
        // Default: coarse-grained.  Nothing writes a region from the CPU while
        // a kernel reads it, and coarse-grained pages may be cached on the GPU.
        r.flags_used = coh == KVP_HOST_DEFAULT ? KVP_HOST_NONCOHERENT : coh;
        flags |= r.flags_used == KVP_HOST_COHERENT ? hipHostMallocCoherent : hipHostMallocNonCoherent;
        if (r.desc.numa_node >= 0) flags |= hipHostMallocNumaUser;
        void *p = nullptr;
        hipError_t e;
        {
            NumaScope bind(r.desc.numa_node);
            e = hipHostMalloc(&p, r.capacity, flags);
        }
        if (e != hipSuccess || !p) {
            clear_hip_error();
            fail(KVP_ERR_NOMEM, "hipHostMalloc of " + std::to_string(r.capacity) + " bytes: " + hipGetErrorString(e));
        }
        r.host = p;
        void *d = nullptr;
        check_hip(hipHostGetDevicePointer(&d, p, 0), "hipHostGetDevicePointer");
        r.dev = d;
        r.numa_actual = page_node(p);
    } else {
        void *d = nullptr;
        hipError_t e = hipMalloc(&d, r.capacity);
        if (e != hipSuccess || !d) {
            clear_hip_error();
            fail(KVP_ERR_NOMEM, "hipMalloc of " + std::to_string(r.capacity) + " bytes: " + hipGetErrorString(e));
        }
        r.dev = d;
    }
}

void free_slot(Slot &s)
{
    if (s.host) (void)hipHostFree(s.host);
    if (s.dev) (void)hipFree(s.dev);
    s.host = s.dev = nullptr;
    s.cap = 0;
}

// The copy-engine transport's ring and events (after the work on them).
void release_bounce(Pool &p)
{
    if (p.s_stage) (void)hipStreamSynchronize(p.s_stage);
    for (uint32_t j = 0; j < kBounceSlots; ++j) {
        if (p.bounce_free_rec[j] && p.bounce_free[j]) (void)hipEventSynchronize(p.bounce_free[j]);
        if (p.bounce_free[j]) (void)hipEventDestroy(p.bounce_free[j]);
        if (p.bounce_filled[j]) (void)hipEventDestroy(p.bounce_filled[j]);
        p.bounce_free[j] = p.bounce_filled[j] = nullptr;
        p.bounce_free_rec[j] = false;
    }
    if (p.bounce) (void)hipFree(p.bounce);
    p.bounce = nullptr;
    p.bounce_slot_bytes = 0;
    p.bounce_next = 0;
}

// Allocate the copy-engine transport's ring on first use.  Caller holds the
// lock and the device scope.
void ensure_bounce(Pool &p)
{
    if (p.bounce) return;
    const uint64_t slot = round_up(std::max(p.bounce_slot_request, p.block_bytes), kSector);
    try {
        void *mem = nullptr;
        if (hipMalloc(&mem, slot * kBounceSlots) != hipSuccess || !mem) {
            clear_hip_error();
            fail(KVP_ERR_NOMEM, "bounce ring of " + std::to_string(slot * kBounceSlots) + " bytes");
        }
        p.bounce = static_cast<char *>(mem);
        p.bounce_slot_bytes = slot;
        for (uint32_t j = 0; j < kBounceSlots; ++j) {
            check_hip(hipEventCreateWithFlags(&p.bounce_filled[j], hipEventDisableTiming), "hipEventCreate");
            check_hip(hipEventCreateWithFlags(&p.bounce_free[j], hipEventDisableTiming), "hipEventCreate");
        }
    } catch (...) {
        release_bounce(p);
        throw;
    }
}

void release_gpu(Pool &p)
{
    if (p.placement_only) return;
    release_bounce(p);
    if (p.s_stage) (void)hipStreamSynchronize(p.s_stage);
    for (auto &s : p.ring) {
        if (s.pending && s.done) (void)hipEventSynchronize(s.done);
        free_slot(s);
        if (s.done) (void)hipEventDestroy(s.done);
        s.done = nullptr;
    }
    for (auto &kv : p.requests) {
        if (kv.second->busy_rec) (void)hipEventSynchronize(kv.second->busy);
        if (kv.second->stored) (void)hipEventDestroy(kv.second->stored);
        if (kv.second->busy) (void)hipEventDestroy(kv.second->busy);
    }
    hipEvent_t *evs[] = {&p.fork, &p.stage_done, &p.link_done[0], &p.link_done[1]};
    for (auto e : evs)
        if (*e) (void)hipEventDestroy(*e), *e = nullptr;
    for (auto &tc : p.timed)
        for (int c = 0; c < 2; ++c) {
            if (tc.t0[c]) (void)hipEventDestroy(tc.t0[c]);
            if (tc.t1[c]) (void)hipEventDestroy(tc.t1[c]);
        }
    p.timed.clear();
    for (auto e : p.spare) (void)hipEventDestroy(e);
    p.spare.clear();
    if (p.s_stage) (void)hipStreamDestroy(p.s_stage);
    p.s_stage = nullptr;
    for (auto &r : p.regions) {
        if (r.host) (void)hipHostFree(r.host);
        else if (r.dev) (void)hipFree(r.dev);
        r.host = r.dev = nullptr;
    }
}

void check_spec(const kvp_kv_spec &s, uint64_t &chunk, uint64_t &block)
{
    if (s.num_layers == 0 || s.num_kv_heads == 0 || s.head_dim == 0 || s.block_size == 0 || s.elem_bytes == 0)
        fail(KVP_ERR_INVALID, "kv spec has a zero dimension");
    if (s.pool_layout > 1) fail(KVP_ERR_INVALID, "pool_layout must be 0 or 1");
    const unsigned __int128 c = static_cast<unsigned __int128>(s.num_kv_heads) * s.block_size * s.head_dim * s.elem_bytes;
    if (c % 16 != 0) fail(KVP_ERR_INVALID, "chunk bytes H*bs*D*elem_bytes must be a multiple of 16");
    if (c >= (static_cast<unsigned __int128>(1) << 36)) fail(KVP_ERR_INVALID, "chunk too large");
    if (s.pool_layout == 1 && (static_cast<uint64_t>(s.head_dim) * s.elem_bytes) % 16 != 0)
        fail(KVP_ERR_INVALID, "token-major pool layout needs head_dim*elem_bytes to be a multiple of 16");
    if (2ull * s.num_layers > (1u << 20)) fail(KVP_ERR_INVALID, "too many layers");
    chunk = static_cast<uint64_t>(c);
    block = 2ull * s.num_layers * chunk;
}

void measure_regions(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps);

}  // namespace

// ---------------------------------------------------------------- launch policy

uint32_t default_grid(uint32_t cls, uint32_t op, const kvp_kv_spec &spec)
{
    // Host class: the link needs only about its bandwidth-delay product in
    // flight; 12 workgroups x 32 KiB keep a PCIe 5.0 x16 link at its measured
    // peak, while more of them only queue reads in the shared memory path and
    // slow the HBM kernel running beside them.  The token-major store (host
    // writes in runs of whole chunks, reads from HBM by rows) wants 16.
    // Staging class: many workgroups so the HBM kernel keeps its share of
    // the memory queues while the host kernel runs -- 65536 half-chunk units
    // in flight for the plain retrieve (2.4 ms beside the host kernel, 2.22 ms
    // alone), 8192 otherwise.
    if (cls == KVP_CLASS_HOST) return (op == KVP_OP_STORE && spec.pool_layout == 1) ? 16u : 12u;
    return (op == KVP_OP_RETRIEVE && spec.pool_layout == 0) ? 65536u : 8192u;
}

uint32_t default_flags(uint32_t cls, uint32_t op, const kvp_kv_spec &spec)
{
    uint32_t f = 0;
    // zero-copy writes to host memory: non-temporal stores measured 0.5 %
    // faster and left the HBM kernel beside them less delayed
    if (cls == KVP_CLASS_HOST && op == KVP_OP_STORE) f |= KVP_LAUNCH_NT_STORE;
    // token-major pools stage each chunk through LDS (contiguous on both
    // sides), except the host-class store: there the direct conversion keeps
    // the host-link side contiguous and measured faster (207 vs 211 ms)
    if (spec.pool_layout == 1 && !(cls == KVP_CLASS_HOST && op == KVP_OP_STORE)) f |= KVP_LAUNCH_LDS;
    // plain HBM retrieve: half-chunk units (the copy shape that measured best)
    if (spec.pool_layout == 0 && cls == KVP_CLASS_STAGING && op == KVP_OP_RETRIEVE) f |= KVP_LAUNCH_SPLIT2;
    return f;
}

// ---------------------------------------------------------------- create / destroy

Pool *pool_create(const kvp_region_desc *regions, const uint64_t *bandwidths, uint32_t n_regions,
                  const kvp_kv_spec *spec, int hip_device)
{
    if (!regions || !spec) fail(KVP_ERR_INVALID, "null argument");
    if (!bandwidths && hip_device < 0) fail(KVP_ERR_INVALID, "a placement-only pool needs bandwidths");
    if (n_regions == 0 || n_regions > 4096) fail(KVP_ERR_INVALID, "n_regions must be in [1, 4096]");
    if (hip_device < -1) fail(KVP_ERR_INVALID, "hip_device must be >= -1");
    auto p = std::make_unique<Pool>();
    p->spec = *spec;
    check_spec(p->spec, p->chunk_bytes, p->block_bytes);
    p->regions.resize(n_regions);
    if (bandwidths)
        p->bandwidth.assign(bandwidths, bandwidths + n_regions);
    else
        p->bandwidth.assign(n_regions, 1);   // replaced by the measurement below
    for (uint32_t i = 0; i < n_regions; ++i) {
        const kvp_region_desc &d = regions[i];
        const std::string who = "region " + std::to_string(i) + ": ";
        if (d.type != KVP_REGION_HOST && d.type != KVP_REGION_STAGING) fail(KVP_ERR_INVALID, who + "bad type");
        if (p->bandwidth[i] == 0) fail(KVP_ERR_INVALID, who + "bandwidth must be positive");
        if (d.capacity_bytes < kSector) fail(KVP_ERR_INVALID, who + "capacity below one 4096-byte sector");
        if (d.numa_node < -1) fail(KVP_ERR_INVALID, who + "numa_node must be >= -1");
        if (d.type == KVP_REGION_HOST && d.flags > KVP_HOST_NONCOHERENT) fail(KVP_ERR_INVALID, who + "bad flags");
        if (d.type == KVP_REGION_STAGING && (d.flags != 0 || d.numa_node != -1))
            fail(KVP_ERR_INVALID, who + "staging regions take no flags and no NUMA node");
        if (d.reserved != 0) fail(KVP_ERR_INVALID, who + "reserved must be 0");
        Region &r = p->regions[i];
        r.desc = d;
        r.bandwidth = p->bandwidth[i];
        r.capacity = d.capacity_bytes / kSector * kSector;
        r.alloc = RangeAllocator(r.capacity);
    }
    for (uint32_t c = 0; c < 2; ++c)
        for (uint32_t o = 0; o < 2; ++o) p->launch[c][o] = LaunchCfg{default_grid(c, o, p->spec), default_flags(c, o, p->spec)};

    p->device = hip_device;
    p->placement_only = hip_device < 0;
    if (p->placement_only) return p.release();

    int n_dev = 0;
    check_hip(hipGetDeviceCount(&n_dev), "hipGetDeviceCount");
    if (hip_device >= n_dev) fail(KVP_ERR_INVALID, "hip_device " + std::to_string(hip_device) + " not present");
    DeviceScope dev(hip_device);
    try {
        for (auto &r : p->regions) alloc_region(r);
        check_hip(hipStreamCreateWithFlags(&p->s_stage, hipStreamNonBlocking), "hipStreamCreate");
        check_hip(hipEventCreateWithFlags(&p->fork, hipEventDisableTiming), "hipEventCreate");
        check_hip(hipEventCreateWithFlags(&p->stage_done, hipEventDisableTiming), "hipEventCreate");
        for (auto &e : p->link_done) check_hip(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate");
        p->ring.resize(kRingSlots);
        for (auto &s : p->ring) check_hip(hipEventCreateWithFlags(&s.done, hipEventDisableTiming), "hipEventCreate");
        if (!bandwidths) {
            // Eq. 1 from measured bandwidths: each region's read rate into HBM
            std::vector<uint64_t> mbps(n_regions);
            measure_regions(*p, kCreateProbeBytes, 0, mbps.data());
            for (uint32_t i = 0; i < n_regions; ++i) p->bandwidth[i] = p->regions[i].bandwidth = mbps[i];
        }
    } catch (...) {
        release_gpu(*p);
        throw;
    }
    return p.release();
}

void pool_destroy(Pool *p)
{
    if (!p) return;
    {
        std::lock_guard<std::mutex> lock(p->mu);
        if (!p->placement_only) {
            DeviceScope dev(p->device);
            release_gpu(*p);
        }
    }
    delete p;
}

// ---------------------------------------------------------------- place / lookup / release

void pool_place(Pool &p, uint64_t request, uint32_t n_blocks, kvp_loc *out)
{
    if (n_blocks == 0) fail(KVP_ERR_INVALID, "n_blocks must be positive");
    if (!out) fail(KVP_ERR_INVALID, "map_out is null");
    std::lock_guard<std::mutex> lock(p.mu);
    if (p.requests.count(request)) fail(KVP_ERR_INVALID, "request " + std::to_string(request) + " is already placed");
    const uint32_t N = static_cast<uint32_t>(p.regions.size());
    std::vector<uint64_t> counts(N);
    target_counts(p.bandwidth.data(), N, n_blocks, counts.data());

    // one contiguous, sector-rounded range per region with a nonzero share;
    // find them all before taking any, so a failure changes nothing
    std::vector<uint64_t> base(N, 0), len(N, 0);
    for (uint32_t i = 0; i < N; ++i) {
        len[i] = round_up(counts[i] * p.block_bytes, kSector);
        if (len[i] && !p.regions[i].alloc.first_fit(len[i], &base[i]))
            fail(KVP_ERR_NOSPACE, "region " + std::to_string(i) + " has no free range of " + std::to_string(len[i]) +
                                      " bytes");
    }

    auto rec = std::make_unique<RequestRec>();
    if (!p.placement_only) {
        DeviceScope dev(p.device);
        check_hip(hipEventCreateWithFlags(&rec->stored, hipEventDisableTiming), "hipEventCreate");
        hipError_t e = hipEventCreateWithFlags(&rec->busy, hipEventDisableTiming);
        if (e != hipSuccess) {
            (void)hipEventDestroy(rec->stored);
            check_hip(e, "hipEventCreate");
        }
    }
    rec->id = request;
    rec->n_blocks = n_blocks;
    rec->gen = p.next_gen++;
    rec->ranges.reserve(N);
    for (uint32_t i = 0; i < N; ++i) {
        if (!len[i]) continue;
        p.regions[i].alloc.take(base[i], len[i]);
        rec->ranges.push_back(Allocation{rec.get(), i, rec->gen, base[i], counts[i], len[i]});
    }
    for (auto &a : rec->ranges) p.regions[a.region].live[a.base] = &a;

    std::vector<uint32_t> region_of;
    stripe(counts, n_blocks, region_of);
    std::vector<uint64_t> next(N, 0);
    for (uint32_t j = 0; j < n_blocks; ++j) {
        const uint32_t r = region_of[j];
        const uint64_t off = base[r] + next[r]++ * p.block_bytes;
        out[j] = kvp_loc{r, rec->gen, off};
        p.glt.insert(GltEntry{request, j, r, p.regions[r].desc.type, rec->gen, off});
    }
    p.requests.emplace(request, std::move(rec));
}

namespace {

void lookup_locked(Pool &p, uint64_t request, uint32_t n_blocks, kvp_loc *out)
{
    auto it = p.requests.find(request);
    if (it == p.requests.end()) fail(KVP_ERR_NOTFOUND, "request " + std::to_string(request) + " is not placed");
    if (it->second->n_blocks != n_blocks)
        fail(KVP_ERR_INVALID, "request has " + std::to_string(it->second->n_blocks) + " blocks, not " +
                                  std::to_string(n_blocks));
    for (uint32_t j = 0; j < n_blocks; ++j) {
        const GltEntry *e = p.glt.find(request, j);
        if (!e) fail(KVP_ERR_NOTFOUND, "GLT entry missing");
        out[j] = kvp_loc{e->region, e->gen, e->offset};
    }
}

}  // namespace

void pool_lookup(Pool &p, uint64_t request, uint32_t n_blocks, kvp_loc *out)
{
    if (!out && n_blocks) fail(KVP_ERR_INVALID, "map_out is null");
    std::lock_guard<std::mutex> lock(p.mu);
    lookup_locked(p, request, n_blocks, out);
}

void pool_lookup_vector(Pool &p, uint64_t request, uint32_t n_blocks, std::vector<kvp_loc> &out)
{
    out.resize(n_blocks);
    std::lock_guard<std::mutex> lock(p.mu);
    lookup_locked(p, request, n_blocks, out.data());
}

void pool_release(Pool &p, uint64_t request)
{
    std::lock_guard<std::mutex> lock(p.mu);
    auto it = p.requests.find(request);
    if (it == p.requests.end()) fail(KVP_ERR_NOTFOUND, "request " + std::to_string(request) + " is not placed");
    RequestRec &rec = *it->second;
    if (!p.placement_only) {
        DeviceScope dev(p.device);
        if (rec.busy_rec) check_hip(hipEventSynchronize(rec.busy), "hipEventSynchronize");
        (void)hipEventDestroy(rec.stored);
        (void)hipEventDestroy(rec.busy);
    }
    for (auto &a : rec.ranges) {
        p.regions[a.region].live.erase(a.base);
        p.regions[a.region].alloc.give(a.base, a.len);
    }
    for (uint32_t j = 0; j < rec.n_blocks; ++j) p.glt.erase(request, j);
    p.requests.erase(it);
}

// ---------------------------------------------------------------- store / retrieve

namespace {

// The live allocation holding the block at map entry e, or an error.
const Allocation *resolve(const Pool &p, const kvp_loc &e, uint32_t b, const Allocation *hint)
{
    const uint32_t N = static_cast<uint32_t>(p.regions.size());
    if (e.region >= N)
        fail(KVP_ERR_INVALID, "map entry " + std::to_string(b) + ": region " + std::to_string(e.region) +
                                  " out of range");
    const Region &r = p.regions[e.region];
    if (e.offset % 16 != 0 || e.offset > r.capacity || r.capacity - e.offset < p.block_bytes)
        fail(KVP_ERR_INVALID, "map entry " + std::to_string(b) + ": offset outside region");
    const Allocation *a = hint;
    if (!(a && a->region == e.region && e.offset >= a->base && e.offset < a->base + a->blocks * p.block_bytes)) {
        auto it = r.live.upper_bound(e.offset);
        if (it == r.live.begin()) fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": no live placement there");
        a = std::prev(it)->second;
        if (e.offset >= a->base + a->blocks * p.block_bytes)
            fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": no live placement there");
    }
    if ((e.offset - a->base) % p.block_bytes != 0 || a->gen != e.gen)
        fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": stale generation or block boundary");
    return a;
}

constexpr size_t kMaxTimedCalls = 4096;

hipEvent_t timing_event(Pool &p)
{
    if (!p.spare.empty()) {
        hipEvent_t e = p.spare.back();
        p.spare.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    check_hip(hipEventCreate(&e), "hipEventCreate");
    return e;
}

// Wait for every recorded call, optionally summarise it, and recycle its events.
void drain_timed(Pool &p, kvp_timing_summary *sum)
{
    kvp_timing_summary s{};
    s.host_ms_min = s.staging_ms_min = -1.f;
    s.host_ms_max = s.staging_ms_max = -1.f;
    for (auto &tc : p.timed) {
        ++s.calls;
        for (int c = 0; c < 2; ++c) {
            if (!tc.ran[c]) continue;
            check_hip(hipEventSynchronize(tc.t1[c]), "hipEventSynchronize");
            float ms = 0.f;
            check_hip(hipEventElapsedTime(&ms, tc.t0[c], tc.t1[c]), "hipEventElapsedTime");
            float &mn = c == 0 ? s.host_ms_min : s.staging_ms_min;
            float &mx = c == 0 ? s.host_ms_max : s.staging_ms_max;
            (c == 0 ? s.host_ms_sum : s.staging_ms_sum) += ms;
            (c == 0 ? s.host_calls : s.staging_calls) += 1;
            mn = mn < 0.f ? ms : std::min(mn, ms);
            mx = std::max(mx, ms);
        }
    }
    for (auto &tc : p.timed)
        for (int c = 0; c < 2; ++c) {
            if (tc.t0[c]) p.spare.push_back(tc.t0[c]);
            if (tc.t1[c]) p.spare.push_back(tc.t1[c]);
        }
    p.timed.clear();
    if (sum) *sum = s;
}

Slot &acquire_slot(Pool &p, size_t bytes)
{
    Slot &s = p.ring[p.ring_next];
    p.ring_next = (p.ring_next + 1) % static_cast<uint32_t>(p.ring.size());
    if (s.pending) {
        check_hip(hipEventSynchronize(s.done), "hipEventSynchronize");
        s.pending = false;
    }
    if (s.cap < bytes) {
        free_slot(s);
        const size_t cap = round_up(std::max(bytes, kSlotMin), kSlotMin);
        void *h = nullptr, *d = nullptr;
        if (hipHostMalloc(&h, cap, hipHostMallocDefault) != hipSuccess || !h) {
            clear_hip_error();
            fail(KVP_ERR_NOMEM, "work-list pinned buffer");
        }
        if (hipMalloc(&d, cap) != hipSuccess || !d) {
            clear_hip_error();
            (void)hipHostFree(h);
            fail(KVP_ERR_NOMEM, "work-list device buffer");
        }
        s.host = h;
        s.dev = d;
        s.cap = cap;
    }
    return s;
}

}  // namespace

void pool_transfer(Pool &p, const kvp_loc *map, uint32_t n_blocks, const int32_t *table, uint32_t num_slots,
                   uint32_t layer_begin, uint32_t layer_end, void *const *k_layers, void *const *v_layers,
                   void *stream_ptr, bool gather)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool has no memory to copy");
    if (n_blocks && (!map || !table)) fail(KVP_ERR_INVALID, "null map or block table");
    const uint32_t L = p.spec.num_layers;
    if (layer_begin >= layer_end || layer_end > L)
        fail(KVP_ERR_INVALID, "layer range [" + std::to_string(layer_begin) + ", " + std::to_string(layer_end) +
                                  ") not inside [0, " + std::to_string(L) + ")");
    if (!k_layers || !v_layers) fail(KVP_ERR_INVALID, "null layer pointer array");
    for (uint32_t l = layer_begin; l < layer_end; ++l) {
        const uintptr_t k = reinterpret_cast<uintptr_t>(k_layers[l]), v = reinterpret_cast<uintptr_t>(v_layers[l]);
        if (!k || !v || (k & 15) || (v & 15))
            fail(KVP_ERR_INVALID, "layer " + std::to_string(l) + ": null or unaligned cache pointer");
    }
    if (static_cast<uint64_t>(n_blocks) * 4 * L >= (1ull << 32)) fail(KVP_ERR_INVALID, "request too large");

    std::lock_guard<std::mutex> lock(p.mu);
    DeviceScope dev(p.device);
    const uint32_t op = gather ? KVP_OP_RETRIEVE : KVP_OP_STORE;
    const bool sdma = (p.launch[KVP_CLASS_HOST][op].flags & KVP_LAUNCH_SDMA) != 0;
    if (sdma && !p.bounce)   // only after a kv_pool_set_copy_ring that could not allocate
        fail(KVP_ERR_NOMEM, "copy-engine ring not allocated: set a smaller ring or clear KVP_LAUNCH_SDMA");

    // GLT-resolved locations, grouped by region class (Sec. 4.3)
    std::vector<CopyItem> items[2];
    std::vector<HostBlock> host_blocks;   // copy-engine transport: placed in ring slots below
    std::vector<RequestRec *> touched;
    std::vector<uint64_t> targets;   // store: (region, offset) keys; retrieve: destination slots
    // one hint per region: a request's blocks in a region share one range,
    // while consecutive blocks of a striped map alternate between regions
    std::vector<const Allocation *> hints(p.regions.size(), nullptr);
    for (uint32_t b = 0; b < n_blocks; ++b) {
        const kvp_loc &e = map[b];
        if (e.region == KVP_ABSENT) continue;
        const Allocation *hint = resolve(p, e, b, e.region < hints.size() ? hints[e.region] : nullptr);
        hints[e.region] = hint;
        const int32_t slot = table[b];
        if (slot < 0 || static_cast<uint32_t>(slot) >= num_slots)
            fail(KVP_ERR_INVALID, "block table entry " + std::to_string(b) + " = " + std::to_string(slot) +
                                      " outside [0, " + std::to_string(num_slots) + ")");
        targets.push_back(gather ? static_cast<uint64_t>(slot)
                                 : (static_cast<uint64_t>(e.region) << 48) | (e.offset >> 4));
        if (std::find(touched.begin(), touched.end(), hint->owner) == touched.end()) touched.push_back(hint->owner);
        const Region &r = p.regions[e.region];
        const uint32_t cls = r.desc.type == KVP_REGION_HOST ? KVP_CLASS_HOST : KVP_CLASS_STAGING;
        if (cls == KVP_CLASS_HOST && sdma)
            host_blocks.push_back(HostBlock{e.region, e.offset, static_cast<uint32_t>(slot)});
        else
            items[cls].push_back(CopyItem{reinterpret_cast<uint64_t>(r.dev) + e.offset, static_cast<uint32_t>(slot), 0u});
    }
    // no two present entries may write the same place (a destination slot on
    // retrieve, a pool block on store): sorted keys, independent of num_slots
    std::sort(targets.begin(), targets.end());
    auto dup = std::adjacent_find(targets.begin(), targets.end());
    if (dup != targets.end())
        fail(KVP_ERR_INVALID, gather ? "destination slot " + std::to_string(*dup) + " named twice"
                                     : std::string("two map entries name the same pool block"));
    const uint64_t width = 2ull * (layer_end - layer_begin) * p.chunk_bytes;   // bytes moved per block
    const uint64_t skip = 2ull * layer_begin * p.chunk_bytes;
    std::vector<LinkRun> runs;
    std::vector<Batch> batches;
    if (!host_blocks.empty()) {
        const RingGeometry g{reinterpret_cast<uint64_t>(p.bounce), p.bounce_slot_bytes, kBounceSlots, p.bounce_next,
                             p.block_bytes, p.chunk_bytes};
        plan_bounce(g, host_blocks, width, 2 * layer_begin, items[KVP_CLASS_HOST], runs, batches);
    }

    const size_t n_items = items[0].size() + items[1].size();
    if (p.timing) {
        if (p.timed.size() >= kMaxTimedCalls) drain_timed(p, nullptr);   // bound the history
        TimedCall tc;
        for (int c = 0; c < 2; ++c) {
            tc.blocks[c] = static_cast<uint32_t>(items[c].size());
            if (!items[c].empty()) {
                tc.t0[c] = timing_event(p);
                tc.t1[c] = timing_event(p);
            }
        }
        p.timed.push_back(tc);
    }
    if (n_items == 0) return;

    // work list: [2L cache pointers][host items][staging items]
    const size_t ptr_bytes = round_up(2ull * L * sizeof(uint64_t), 16);
    const size_t bytes = ptr_bytes + n_items * sizeof(CopyItem);
    Slot &slot = acquire_slot(p, bytes);
    auto *ptrs = static_cast<uint64_t *>(slot.host);
    for (uint32_t l = 0; l < L; ++l) {
        const bool in = l >= layer_begin && l < layer_end;   // entries outside the range are never read
        ptrs[2 * l] = in ? reinterpret_cast<uint64_t>(k_layers[l]) : 0;
        ptrs[2 * l + 1] = in ? reinterpret_cast<uint64_t>(v_layers[l]) : 0;
    }
    auto *list = reinterpret_cast<CopyItem *>(static_cast<char *>(slot.host) + ptr_bytes);
    std::copy(items[0].begin(), items[0].end(), list);
    std::copy(items[1].begin(), items[1].end(), list + items[0].size());

    hipStream_t s = static_cast<hipStream_t>(stream_ptr);
    // ordering with earlier work on the same requests from any stream:
    // retrieve after store (read after write), store after store/retrieve
    for (RequestRec *rec : touched) {
        if (gather && rec->stored_rec) check_hip(hipStreamWaitEvent(s, rec->stored, 0), "hipStreamWaitEvent");
        if (!gather && rec->busy_rec) check_hip(hipStreamWaitEvent(s, rec->busy, 0), "hipStreamWaitEvent");
    }
    check_hip(hipMemcpyAsync(slot.dev, slot.host, bytes, hipMemcpyHostToDevice, s), "hipMemcpyAsync");
    slot.pending = true;  // from here on the slot is in use even if a launch fails
    // the internal stream takes work only for enough staging bytes or for ring batches
    const bool fork_staging = batches.empty() && items[KVP_CLASS_STAGING].size() * width >= kForkMinBytes;
    if (fork_staging || !batches.empty()) check_hip(hipEventRecord(p.fork, s), "hipEventRecord");

    const CopyItem *dev_list = reinterpret_cast<const CopyItem *>(static_cast<char *>(slot.dev) + ptr_bytes);
    // Staging class forked onto the internal stream first, then the host
    // class on the caller's stream itself; the caller's stream then waits for
    // the staging kernel.  One extra stream keeps the pool within the few
    // hardware queues a process gets, so caller streams (e.g. compute
    // overlapping a layerwise retrieve) are not serialised behind it.
    size_t first = 0;
    CopyArgs args[2] = {};
    for (uint32_t c = 0; c < 2; ++c) {
        CopyArgs &a = args[c];
        a.items = dev_list + first;
        a.cache = static_cast<const uint64_t *>(slot.dev);
        a.n_items = static_cast<uint32_t>(items[c].size());
        a.chunks = 2 * (layer_end - layer_begin);
        a.chunk0 = 2 * layer_begin;
        a.parts = 1;
        a.xcd_remap = 0;
        a.chunk_bytes = p.chunk_bytes;
        a.heads = p.spec.num_kv_heads;
        a.tokens = p.spec.block_size;
        a.row_vec = static_cast<uint32_t>(static_cast<uint64_t>(p.spec.head_dim) * p.spec.elem_bytes / 16);
        a.layout = p.spec.pool_layout;
        first += items[c].size();
    }
    TimedCall *tc = p.timing ? &p.timed.back() : nullptr;
    auto launch = [&](uint32_t c, hipStream_t st) {
        const LaunchCfg &lc = p.launch[c][op];
        if (tc) check_hip(hipEventRecord(tc->t0[c], st), "hipEventRecord");
        check_hip(launch_chunk_copy(args[c], c, gather, lc.grid, lc.flags, st), "kernel launch");
        if (tc) {
            check_hip(hipEventRecord(tc->t1[c], st), "hipEventRecord");
            tc->ran[c] = true;
        }
    };
    const bool staging = !items[KVP_CLASS_STAGING].empty();
    if (batches.empty()) {
        if (fork_staging) {
            check_hip(hipStreamWaitEvent(p.s_stage, p.fork, 0), "hipStreamWaitEvent");
            launch(KVP_CLASS_STAGING, p.s_stage);
            check_hip(hipEventRecord(p.stage_done, p.s_stage), "hipEventRecord");
        } else if (staging) {
            launch(KVP_CLASS_STAGING, s);   // small: in order on the caller's stream
        }
        if (!items[KVP_CLASS_HOST].empty()) {
            // one host-class kernel on the link at a time, in enqueue order:
            // two of them would only share its bandwidth and both end late
            if (p.link_rec[op] && p.link_stream[op] != s)
                check_hip(hipStreamWaitEvent(s, p.link_done[op], 0), "hipStreamWaitEvent");
            launch(KVP_CLASS_HOST, s);
            check_hip(hipEventRecord(p.link_done[op], s), "hipEventRecord");
            p.link_rec[op] = true;
            p.link_stream[op] = s;
        }
        if (fork_staging) check_hip(hipStreamWaitEvent(s, p.stage_done, 0), "hipStreamWaitEvent");
    } else {
        // Copy-engine transport: the host-link copies take the internal
        // stream (no stream beyond the kernel path's two) and every kernel
        // runs on the caller's stream -- the staging class first, then one
        // ring-slot kernel per batch.  A slot is refilled only after its
        // previous contents were consumed (by any call, either op).
        if (staging) launch(KVP_CLASS_STAGING, s);
        const LaunchCfg &lc = p.launch[KVP_CLASS_STAGING][op];
        const hipMemcpyKind kind = gather ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost;
        hipStream_t sc = p.s_stage;
        auto link_copies = [&](const Batch &bt) {
            char *ring = p.bounce + static_cast<uint64_t>(bt.ring) * p.bounce_slot_bytes;
            for (size_t i = bt.run0; i < bt.run0 + bt.runs; ++i) {
                const LinkRun &run = runs[i];
                char *host = static_cast<char *>(p.regions[run.region].host) + run.offset + skip;
                char *dev = ring + run.slot_offset;
                void *dst = gather ? static_cast<void *>(dev) : static_cast<void *>(host);
                const void *src = gather ? static_cast<const void *>(host) : static_cast<const void *>(dev);
                if (width == p.block_bytes)
                    check_hip(hipMemcpyAsync(dst, src, run.blocks * width, kind, sc), "hipMemcpyAsync");
                else
                    check_hip(hipMemcpy2DAsync(dst, gather ? width : p.block_bytes, src, gather ? p.block_bytes : width,
                                               width, run.blocks, kind, sc),
                              "hipMemcpy2DAsync");
            }
        };
        auto ring_kernel = [&](const Batch &bt) {
            CopyArgs a = args[KVP_CLASS_HOST];
            a.items = dev_list + bt.first;
            a.n_items = bt.n;
            check_hip(launch_chunk_copy(a, kClassRing, gather, lc.grid, lc.flags, s), "kernel launch");
        };
        if (gather) {
            check_hip(hipStreamWaitEvent(sc, p.fork, 0), "hipStreamWaitEvent");
            if (tc) check_hip(hipEventRecord(tc->t0[KVP_CLASS_HOST], sc), "hipEventRecord");
            for (const Batch &bt : batches) {
                if (p.bounce_free_rec[bt.ring])
                    check_hip(hipStreamWaitEvent(sc, p.bounce_free[bt.ring], 0), "hipStreamWaitEvent");
                link_copies(bt);
                check_hip(hipEventRecord(p.bounce_filled[bt.ring], sc), "hipEventRecord");
                check_hip(hipStreamWaitEvent(s, p.bounce_filled[bt.ring], 0), "hipStreamWaitEvent");
                ring_kernel(bt);
                check_hip(hipEventRecord(p.bounce_free[bt.ring], s), "hipEventRecord");
                p.bounce_free_rec[bt.ring] = true;
            }
        } else {
            if (tc) check_hip(hipEventRecord(tc->t0[KVP_CLASS_HOST], s), "hipEventRecord");
            for (const Batch &bt : batches) {
                if (p.bounce_free_rec[bt.ring])
                    check_hip(hipStreamWaitEvent(s, p.bounce_free[bt.ring], 0), "hipStreamWaitEvent");
                ring_kernel(bt);
                check_hip(hipEventRecord(p.bounce_filled[bt.ring], s), "hipEventRecord");
                check_hip(hipStreamWaitEvent(sc, p.bounce_filled[bt.ring], 0), "hipStreamWaitEvent");
                link_copies(bt);
                check_hip(hipEventRecord(p.bounce_free[bt.ring], sc), "hipEventRecord");
                p.bounce_free_rec[bt.ring] = true;
            }
            check_hip(hipEventRecord(p.stage_done, sc), "hipEventRecord");
            check_hip(hipStreamWaitEvent(s, p.stage_done, 0), "hipStreamWaitEvent");
        }
        p.bounce_next = static_cast<uint32_t>((p.bounce_next + batches.size()) % kBounceSlots);
        if (tc) {
            check_hip(hipEventRecord(tc->t1[KVP_CLASS_HOST], s), "hipEventRecord");
            tc->ran[KVP_CLASS_HOST] = true;
        }
    }
    check_hip(hipEventRecord(slot.done, s), "hipEventRecord");
    for (RequestRec *rec : touched) {
        check_hip(hipEventRecord(rec->busy, s), "hipEventRecord");
        rec->busy_rec = true;
        if (!gather) {
            check_hip(hipEventRecord(rec->stored, s), "hipEventRecord");
            rec->stored_rec = true;
        }
    }
}

// ---------------------------------------------------------------- measured bandwidths (Sec. 4.1.2)

namespace {

// Read rate of every region (bytes from the region into HBM per second, in
// MB/s): the region-class kernel's launch shape streams min(probe_bytes,
// capacity) bytes from the region into a scratch buffer; best of 3 after one
// warm-up.  Caller holds the pool lock and the device scope.
void measure_regions(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps)
{
    probe_bytes &= ~15ull;
    void *scratch = nullptr;
    if (hipMalloc(&scratch, probe_bytes) != hipSuccess || !scratch) {
        clear_hip_error();
        fail(KVP_ERR_NOMEM, "probe scratch of " + std::to_string(probe_bytes) + " bytes");
    }
    hipEvent_t e0 = nullptr, e1 = nullptr;
    try {
        check_hip(hipEventCreate(&e0), "hipEventCreate");
        check_hip(hipEventCreate(&e1), "hipEventCreate");
        uint32_t n_host = 0;
        for (size_t r = 0; r < p.regions.size(); ++r) {
            const Region &reg = p.regions[r];
            const uint32_t cls = reg.desc.type == KVP_REGION_HOST ? KVP_CLASS_HOST : KVP_CLASS_STAGING;
            n_host += cls == KVP_CLASS_HOST;
            hipStream_t st = p.s_stage;   // one probe at a time
            const uint64_t n = std::min<uint64_t>(probe_bytes, reg.capacity) & ~15ull;
            const LaunchCfg &lc = p.launch[cls][KVP_OP_RETRIEVE];
            float best = 0.f;
            for (int it = 0; it < 4; ++it) {
                check_hip(hipEventRecord(e0, st), "hipEventRecord");
                check_hip(launch_probe_copy(scratch, reg.dev, n, lc.grid, lc.flags & KVP_LAUNCH_NT_LOAD, st),
                          "probe launch");
                check_hip(hipEventRecord(e1, st), "hipEventRecord");
                check_hip(hipEventSynchronize(e1), "hipEventSynchronize");
                float ms = 0.f;
                check_hip(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
                if (it > 0 && (best == 0.f || ms < best)) best = ms;
            }
            const double rate = best > 0.f ? static_cast<double>(n) / (best * 1e3) : 1.0;   // MB/s
            mbps[r] = std::max<uint64_t>(1, static_cast<uint64_t>(rate + 0.5));
        }
        // host regions reach the GPU over one shared link: split what one measured alone
        if ((flags & KVP_MEASURE_SHARED_LINK) && n_host > 1)
            for (size_t r = 0; r < p.regions.size(); ++r)
                if (p.regions[r].desc.type == KVP_REGION_HOST) mbps[r] = std::max<uint64_t>(1, mbps[r] / n_host);
    } catch (...) {
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
        (void)hipFree(scratch);
        throw;
    }
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    (void)hipFree(scratch);
}

}  // namespace

void pool_measure(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps_out)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool has no memory to measure");
    if (!mbps_out) fail(KVP_ERR_INVALID, "null output");
    if (flags & ~KVP_MEASURE_SHARED_LINK) fail(KVP_ERR_INVALID, "unknown flags");
    if (probe_bytes < (1u << 16) || probe_bytes > (1ull << 36)) fail(KVP_ERR_INVALID, "probe_bytes outside [64 KiB, 64 GiB]");
    std::lock_guard<std::mutex> lock(p.mu);
    DeviceScope dev(p.device);
    measure_regions(p, probe_bytes, flags, mbps_out);
}

void pool_set_bandwidths(Pool &p, const uint64_t *bw)
{
    if (!bw) fail(KVP_ERR_INVALID, "null bandwidths");
    for (size_t i = 0; i < p.regions.size(); ++i)
        if (bw[i] == 0) fail(KVP_ERR_INVALID, "bandwidth of region " + std::to_string(i) + " is 0");
    std::lock_guard<std::mutex> lock(p.mu);
    for (size_t i = 0; i < p.regions.size(); ++i) {
        p.bandwidth[i] = bw[i];
        p.regions[i].bandwidth = bw[i];
    }
}

// ---------------------------------------------------------------- introspection, launch config, timing

void pool_region_info(const Pool &p, uint32_t region, kvp_region_info *out)
{
    if (!out) fail(KVP_ERR_INVALID, "null output");
    if (region >= p.regions.size()) fail(KVP_ERR_INVALID, "region index out of range");
    const Region &r = p.regions[region];
    *out = kvp_region_info{r.desc.type, r.desc.numa_node, r.numa_actual, r.flags_used, r.capacity,
                           r.bandwidth, r.host, r.dev};
}

void pool_region_read(Pool &p, uint32_t region, uint64_t offset, uint64_t bytes, void *dst)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool has no memory");
    if (region >= p.regions.size()) fail(KVP_ERR_INVALID, "region index out of range");
    const Region &r = p.regions[region];
    if (!dst && bytes) fail(KVP_ERR_INVALID, "null destination");
    if (offset > r.capacity || r.capacity - offset < bytes) fail(KVP_ERR_INVALID, "range outside region");
    if (!bytes) return;
    if (r.host) {
        std::memcpy(dst, static_cast<const char *>(r.host) + offset, bytes);
    } else {
        DeviceScope dev(p.device);
        check_hip(hipMemcpy(dst, static_cast<const char *>(r.dev) + offset, bytes, hipMemcpyDeviceToHost),
                  "hipMemcpy");
    }
}

void pool_set_launch(Pool &p, uint32_t cls, uint32_t op, uint32_t grid, uint32_t flags)
{
    if (cls > 1 || op > 1) fail(KVP_ERR_INVALID, "class and op must be 0 or 1");
    if (flags & ~(KVP_LAUNCH_NT_LOAD | KVP_LAUNCH_NT_STORE | KVP_LAUNCH_LDS | KVP_LAUNCH_SPLIT2 | KVP_LAUNCH_XCD |
                  KVP_LAUNCH_SDMA | KVP_LAUNCH_CHUNK_MAJOR))
        fail(KVP_ERR_INVALID, "unknown flags");
    if (grid > (1u << 20)) fail(KVP_ERR_INVALID, "grid too large");
    if ((flags & KVP_LAUNCH_SDMA) && cls != KVP_CLASS_HOST)
        fail(KVP_ERR_INVALID, "the copy-engine transport is for the host class");
    if ((flags & KVP_LAUNCH_SDMA) && p.placement_only)
        fail(KVP_ERR_INVALID, "placement-only pool launches nothing");
    std::lock_guard<std::mutex> lock(p.mu);
    if (flags & KVP_LAUNCH_SDMA) {
        DeviceScope dev(p.device);
        ensure_bounce(p);
    }
    p.launch[cls][op] = LaunchCfg{grid ? grid : default_grid(cls, op, p.spec), flags};  // flags taken as given
}

void pool_set_copy_ring(Pool &p, uint64_t slot_bytes)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool launches nothing");
    if (slot_bytes % kSector || slot_bytes < (64u << 10) || slot_bytes > (1ull << 36))
        fail(KVP_ERR_INVALID, "slot_bytes must be a multiple of 4096 in [64 KiB, 64 GiB]");
    std::lock_guard<std::mutex> lock(p.mu);
    DeviceScope dev(p.device);
    release_bounce(p);
    p.bounce_slot_request = slot_bytes;
    if ((p.launch[KVP_CLASS_HOST][KVP_OP_RETRIEVE].flags | p.launch[KVP_CLASS_HOST][KVP_OP_STORE].flags) &
        KVP_LAUNCH_SDMA)
        ensure_bounce(p);
}

void pool_set_timing(Pool &p, int enable)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool launches nothing");
    std::lock_guard<std::mutex> lock(p.mu);
    DeviceScope dev(p.device);
    drain_timed(p, nullptr);
    p.timing = enable != 0;
}

void pool_last_timing(Pool &p, kvp_timing *out)
{
    if (!out) fail(KVP_ERR_INVALID, "null output");
    std::lock_guard<std::mutex> lock(p.mu);
    if (!p.timing || p.timed.empty()) fail(KVP_ERR_INVALID, "no timed call");
    DeviceScope dev(p.device);
    const TimedCall &tc = p.timed.back();
    float ms[2] = {-1.f, -1.f};
    for (int c = 0; c < 2; ++c) {
        if (!tc.ran[c]) continue;
        check_hip(hipEventSynchronize(tc.t1[c]), "hipEventSynchronize");
        check_hip(hipEventElapsedTime(&ms[c], tc.t0[c], tc.t1[c]), "hipEventElapsedTime");
    }
    *out = kvp_timing{ms[0], ms[1], tc.blocks[0], tc.blocks[1]};
}

void pool_timing_summary(Pool &p, kvp_timing_summary *out)
{
    if (!out) fail(KVP_ERR_INVALID, "null output");
    std::lock_guard<std::mutex> lock(p.mu);
    if (!p.timing) fail(KVP_ERR_INVALID, "timing is off");
    DeviceScope dev(p.device);
    drain_timed(p, out);
}

}  // namespace kvp

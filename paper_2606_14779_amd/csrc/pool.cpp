// KV pool: regions, the pool's life cycle, and placement bookkeeping.
//
// A pool enumerates its regions (Sec. 4.1.1): pinned, GPU-mapped host buffers
// bound to a NUMA node, and HBM staging buffers standing in for SSDs.  Placing
// a request computes its Eq. 2 counts and striped map (placement.cpp), takes
// one contiguous range per region from an address-ordered first-fit allocator
// (the LBA-range rule of Sec. 4.2), and records every block in the GLT.
// The store / retrieve engine is in transfer.cpp; measured bandwidths,
// introspection and settings are in control.cpp.

#include <numaif.h>
#include <sys/syscall.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstdio>
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

constexpr uint32_t kRingSlots = 32;
constexpr uint64_t kCreateProbeBytes = 256ull << 20;   // per-region read probe when no bandwidths are given

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

// The online NUMA nodes, from /sys/devices/system/node/online ("0", "0-1",
// "0,2-3"); empty if unreadable.
std::vector<int> online_nodes()
{
    std::vector<int> nodes;
    FILE *f = std::fopen("/sys/devices/system/node/online", "r");
    if (!f) return nodes;
    char buf[256] = {};
    const bool ok = std::fgets(buf, sizeof buf, f) != nullptr;
    std::fclose(f);
    if (!ok) return nodes;
    char *save = nullptr;   // strtok_r: pools may be created from several threads at once
    for (char *tok = strtok_r(buf, ",\n", &save); tok; tok = strtok_r(nullptr, ",\n", &save)) {
        int a = -1, b = -1;
        const int got = std::sscanf(tok, "%d-%d", &a, &b);
        if (got == 1) b = a;
        if (got >= 1 && a >= 0 && b >= a && b - a < 4096)
            for (int n = a; n <= b; ++n) nodes.push_back(n);
    }
    return nodes;
}

// The node holding most of the pages of the mapping that contains p, from
// the "N<node>=<pages>" fields of its /proc/self/numa_maps line; -1 if none.
int numa_maps_node(const void *p)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    uintptr_t start = 0;
    bool found = false;
    if (FILE *m = std::fopen("/proc/self/maps", "r")) {   // the mapping's start address
        char line[512];
        while (std::fgets(line, sizeof line, m)) {
            unsigned long lo = 0, hi = 0;
            if (std::sscanf(line, "%lx-%lx", &lo, &hi) == 2 && a >= lo && a < hi) {
                start = lo;
                found = true;
                break;
            }
        }
        std::fclose(m);
    }
    if (!found) return -1;
    FILE *f = std::fopen("/proc/self/numa_maps", "r");
    if (!f) return -1;
    int best = -1;
    long best_pages = 0;
    char line[4096];
    while (std::fgets(line, sizeof line, f)) {
        unsigned long lo = 0;
        if (std::sscanf(line, "%lx", &lo) != 1 || lo != start) continue;
        char *save = nullptr;
        for (char *tok = strtok_r(line, " \n", &save); tok; tok = strtok_r(nullptr, " \n", &save)) {
            int node = -1;
            long pages = 0;
            if (std::sscanf(tok, "N%d=%ld", &node, &pages) == 2 && pages > best_pages) {
                best = node;
                best_pages = pages;
            }
        }
        break;
    }
    std::fclose(f);
    return best;
}

// NUMA node backing the page at p: move_pages() in query mode (no nodes
// given) reports where each page lives; get_mempolicy() and the mapping's
// page counts in /proc/self/numa_maps are the fallbacks.  Driver-pinned pages
// may be invisible to all three; on a machine with a single online node they
// can only be on that node.
int page_node(void *p)
{
    void *pages[1] = {p};
    int status[1] = {-1};
    if (syscall(SYS_move_pages, 0, 1ul, pages, nullptr, status, 0) == 0 && status[0] >= 0) return status[0];
    int node = -1;
    if (syscall(SYS_get_mempolicy, &node, nullptr, 0, p, MPOL_F_NODE | MPOL_F_ADDR) == 0 && node >= 0) return node;
    node = numa_maps_node(p);
    if (node >= 0) return node;
    const std::vector<int> online = online_nodes();
    return online.size() == 1 ? online[0] : -1;
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

}  // namespace

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

// The file regions' ring: kFileSlots pinned, GPU-mapped host buffers of
// slot_bytes each (raised to one block), and their events.  Caller holds the
// device scope; on failure nothing stays allocated.
void alloc_file_ring(Pool &p, uint64_t slot_bytes)
{
    const uint64_t slot = round_up(std::max(slot_bytes, p.block_bytes), kSector);
    void *h = nullptr;
    if (hipHostMalloc(&h, slot * kFileSlots, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess || !h) {
        clear_hip_error();
        fail(KVP_ERR_NOMEM, "file-region ring of " + std::to_string(slot * kFileSlots) + " bytes");
    }
    try {
        void *d = nullptr;
        check_hip(hipHostGetDevicePointer(&d, h, 0), "hipHostGetDevicePointer");
        for (uint32_t j = 0; j < kFileSlots; ++j)
            if (!p.file_free[j])
                check_hip(hipEventCreateWithFlags(&p.file_free[j], hipEventDisableTiming), "hipEventCreate");
        p.file_ring = static_cast<char *>(h);
        p.file_ring_dev = reinterpret_cast<uint64_t>(d);
        p.file_slot_bytes = slot;
        p.file_next = 0;
    } catch (...) {
        (void)hipHostFree(h);
        throw;
    }
}

// The file regions' ring, after the kernels and the reads / writes on it.
void free_file_ring(Pool &p)
{
    for (uint32_t j = 0; j < kFileSlots; ++j) {
        io_drain(p.file_io[j]);
        if (p.file_free_rec[j] && p.file_free[j]) (void)hipEventSynchronize(p.file_free[j]);
        p.file_free_rec[j] = false;
    }
    if (p.file_ring) (void)hipHostFree(p.file_ring);
    p.file_ring = nullptr;
    p.file_ring_dev = 0;
    p.file_slot_bytes = 0;
}

namespace {

void release_gpu(Pool &p)
{
    if (p.placement_only) return;
    release_bounce(p);
    free_file_ring(p);
    for (auto &e : p.file_free)
        if (e) (void)hipEventDestroy(e), e = nullptr;
    p.workers.reset();   // joins the file regions' worker threads
    for (auto &r : p.regions) close_file_region(r);
    if (p.s_stage) (void)hipStreamSynchronize(p.s_stage);
    for (auto &s : p.ring) {
        if (s.pending && s.done) (void)hipEventSynchronize(s.done);
        free_slot(s);
        if (s.done) (void)hipEventDestroy(s.done);
        s.done = nullptr;
    }
    for (int op = 0; op < 2; ++op)   // the last host-class kernel of each direction
        if (p.link_rec[op] && p.link_done[op]) (void)hipEventSynchronize(p.link_done[op]);
    for (auto &kv : p.requests) {
        if (kv.second->busy_rec) (void)hipEventSynchronize(kv.second->busy);
        if (kv.second->stored) (void)hipEventDestroy(kv.second->stored);
        if (kv.second->busy) (void)hipEventDestroy(kv.second->busy);
    }
    hipEvent_t *evs[] = {&p.fork, &p.stage_done, &p.uploaded, &p.link_done[0], &p.link_done[1]};
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

bool has_file_region(const Pool &p)
{
    for (const auto &r : p.regions)
        if (r.desc.type == KVP_REGION_FILE) return true;
    return false;
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

}  // namespace

// ---------------------------------------------------------------- launch policy

uint32_t default_grid(uint32_t cls, uint32_t op, const kvp_kv_spec &spec)
{
    // Host class: the link needs only about its bandwidth-delay product in
    // flight; 12 workgroups x 32 KiB keep a PCIe 5.0 x16 link at its measured
    // peak, while more of them only queue reads in the shared memory path and
    // slow the HBM kernel running beside them.  A token-major pool wants
    // more: its LDS-staged retrieve has no link reads in flight while a
    // workgroup writes its chunk out (128K LLaMA-shaped retrieve: 200.5-200.7
    // ms at 16, 201.7 at 12, 206 at 20, 216 at 24), and its store writes the
    // host side in runs of whole chunks while reading HBM by rows (205.3 ms
    // at 20 or 24, 207.4-208.7 at 16, 211.2 at 12).
    // Staging class: one unit per workgroup, with no grid-stride loop (the
    // launch caps the grid at the call's unit count), up to 2^20 workgroups.
    if (cls == KVP_CLASS_HOST) return spec.pool_layout == 1 ? (op == KVP_OP_STORE ? 20u : 16u) : 12u;
    return 1u << 20;
}

uint32_t default_flags(uint32_t cls, uint32_t op, const kvp_kv_spec &spec)
{
    uint32_t f = 0;
    // zero-copy writes to host memory: non-temporal stores measured 0.5 %
    // faster and left the HBM kernel beside them less delayed
    if (cls == KVP_CLASS_HOST && op == KVP_OP_STORE) f |= KVP_LAUNCH_NT_STORE;
    // token-major pools stage each chunk through LDS (contiguous on both
    // sides), except the host-class store: there the direct conversion keeps
    // the host-link side contiguous and measured faster (16 workgroups:
    // 207.4-208.7 ms against 210.6-211.9 through LDS)
    if (spec.pool_layout == 1 && !(cls == KVP_CLASS_HOST && op == KVP_OP_STORE)) f |= KVP_LAUNCH_LDS;
    // Staging class: non-temporal loads and stores, one unit per workgroup
    // (default_grid); head-major pools in half-chunk units, the retrieve in
    // chunk-major unit order.  Measured on a 128K-token LLaMA-shaped request
    // placed on measured weights (8145 staging blocks, 17 GB), HBM traffic of
    // the kernel alone: gather 5608 GB/s this way, 5526 in block order, 4907
    // with the XCD renumbering, 5166 in workgroup-owned tiles of 8 blocks;
    // store 5517 against 5418 in chunk-major order and 5103 for 8192
    // grid-stride workgroups; token-major through LDS, gather 5519 and store
    // 5353 against 5112 and 5111 in the earlier forms.  A plain copy on this
    // GPU peaks in the same form (16 KiB per workgroup, non-temporal both
    // ways) at 5.7 TB/s of traffic, where reads alone reach 7.2 and writes
    // alone 5.9.  Beside the host-class kernel of the same request the link
    // rate is unchanged.
    if (cls == KVP_CLASS_STAGING) {
        f |= KVP_LAUNCH_NT_LOAD | KVP_LAUNCH_NT_STORE;
        if (spec.pool_layout == 0) f |= KVP_LAUNCH_SPLIT2 | (op == KVP_OP_RETRIEVE ? KVP_LAUNCH_CHUNK_MAJOR : 0u);
    }
    return f;
}

// ---------------------------------------------------------------- create / destroy

Pool *pool_create(const kvp_region_desc *regions, const uint64_t *bandwidths, uint32_t n_regions,
                  const kvp_kv_spec *spec, int hip_device, const char *const *paths)
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
        if (d.type != KVP_REGION_HOST && d.type != KVP_REGION_STAGING && d.type != KVP_REGION_FILE)
            fail(KVP_ERR_INVALID, who + "bad type");
        if (p->bandwidth[i] == 0) fail(KVP_ERR_INVALID, who + "bandwidth must be positive");
        if (d.capacity_bytes < kSector) fail(KVP_ERR_INVALID, who + "capacity below one 4096-byte sector");
        if (d.numa_node < -1) fail(KVP_ERR_INVALID, who + "numa_node must be >= -1");
        if (d.type == KVP_REGION_HOST && d.flags > KVP_HOST_NONCOHERENT) fail(KVP_ERR_INVALID, who + "bad flags");
        if (d.type == KVP_REGION_STAGING && (d.flags != 0 || d.numa_node != -1))
            fail(KVP_ERR_INVALID, who + "staging regions take no flags and no NUMA node");
        if (d.type == KVP_REGION_FILE) {
            if (d.flags & ~KVP_FILE_BUFFERED) fail(KVP_ERR_INVALID, who + "bad flags");
            if (d.numa_node != -1) fail(KVP_ERR_INVALID, who + "file regions take no NUMA node");
            if ((2 * p->chunk_bytes) % kSector != 0)
                fail(KVP_ERR_INVALID, who + "a file region needs 2 x chunk bytes to be a multiple of 4096");
            if (hip_device >= 0 && (!paths || !paths[i] || !*paths[i]))
                fail(KVP_ERR_INVALID, who + "file region without a path");
        }
        if (d.reserved != 0) fail(KVP_ERR_INVALID, who + "reserved must be 0");
        Region &r = p->regions[i];
        r.desc = d;
        r.bandwidth = p->bandwidth[i];
        r.capacity = d.capacity_bytes / kSector * kSector;
        r.alloc = RangeAllocator(r.capacity);
    }
    for (uint32_t c = 0; c < 2; ++c)
        for (uint32_t o = 0; o < 2; ++o)
            p->launch[c][o] = LaunchCfg{default_grid(c, o, p->spec), default_flags(c, o, p->spec), true};

    p->device = hip_device;
    p->placement_only = hip_device < 0;
    if (p->placement_only) return p.release();

    int n_dev = 0;
    check_hip(hipGetDeviceCount(&n_dev), "hipGetDeviceCount");
    if (hip_device >= n_dev) fail(KVP_ERR_INVALID, "hip_device " + std::to_string(hip_device) + " not present");
    DeviceScope dev(hip_device);
    try {
        for (uint32_t i = 0; i < n_regions; ++i) {
            Region &r = p->regions[i];
            if (r.desc.type == KVP_REGION_FILE)
                open_file_region(r, paths[i]);
            else
                alloc_region(r);
        }
        if (has_file_region(*p)) {
            size_t n_files = 0;
            uint64_t largest = 0;
            for (auto &r : p->regions)
                if (r.desc.type == KVP_REGION_FILE) {
                    r.worker = static_cast<uint32_t>(n_files++);
                    largest = std::max(largest, r.capacity);
                }
            p->workers = std::make_unique<FileWorkers>(n_files);
            alloc_file_ring(*p, std::min(kFileSlotMax, round_up(largest, kSector)));
        }
        check_hip(hipStreamCreateWithFlags(&p->s_stage, hipStreamNonBlocking), "hipStreamCreate");
        check_hip(hipEventCreateWithFlags(&p->fork, hipEventDisableTiming), "hipEventCreate");
        check_hip(hipEventCreateWithFlags(&p->uploaded, hipEventDisableTiming), "hipEventCreate");
        check_hip(hipEventCreateWithFlags(&p->stage_done, hipEventDisableTiming), "hipEventCreate");
        for (auto &e : p->link_done) check_hip(hipEventCreateWithFlags(&e, hipEventDisableTiming), "hipEventCreate");
        p->ring.resize(kRingSlots);
        for (auto &s : p->ring) check_hip(hipEventCreateWithFlags(&s.done, hipEventDisableTiming), "hipEventCreate");
        (void)scratch_setup(hip_device);   // once per device: the static work-list scratch
        if (!bandwidths) {
            // Eq. 1 from measured bandwidths: each region's read rate into HBM
            std::vector<uint64_t> mbps(n_regions);
            measure_regions(*p, kCreateProbeBytes, KVP_MEASURE_SHARED_LINK | KVP_MEASURE_FILES_TOGETHER,
                            mbps.data());
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

namespace {

// One offload set (Alg. 1 on the blocks of one place or extend call; the
// KV caches of one decoding step in Sec. 4.1.3): Eq. 2 counts for the set,
// and per region with a share one contiguous, sector-rounded range (Sec. 4.2),
// found first fit.  reserve() finds them all and changes nothing, so a
// failure leaves the pool as it was; commit() takes them.
struct SetPlan {
    std::vector<uint64_t> counts, base, len;
};

SetPlan reserve_set(Pool &p, uint32_t n)
{
    const uint32_t N = static_cast<uint32_t>(p.regions.size());
    SetPlan s{std::vector<uint64_t>(N), std::vector<uint64_t>(N, 0), std::vector<uint64_t>(N, 0)};
    target_counts(p.bandwidth.data(), N, n, s.counts.data());
    for (uint32_t i = 0; i < N; ++i) {
        s.len[i] = round_up(s.counts[i] * p.block_bytes, kSector);
        if (s.len[i] && !p.regions[i].alloc.first_fit(s.len[i], &s.base[i]))
            fail(KVP_ERR_NOSPACE, "region " + std::to_string(i) + " has no free range of " + std::to_string(s.len[i]) +
                                      " bytes");
    }
    return s;
}

// Take the planned ranges for blocks first .. first+n-1 of rec, stripe the
// blocks over them (R3) and record their GLT entries.  All or nothing: every
// step that allocates host memory runs before the pool changes, or is undone
// if a later one fails; what follows them cannot fail.
void commit_set(Pool &p, RequestRec &rec, const SetPlan &s, uint32_t first, uint32_t n, kvp_loc *out)
{
    const uint32_t N = static_cast<uint32_t>(p.regions.size());
    std::vector<uint32_t> region_of;
    stripe(s.counts, n, region_of);
    std::vector<uint64_t> next(N, 0);
    p.glt.reserve(n);
    const size_t ranges_before = rec.ranges.size();
    uint32_t linked = 0;   // regions whose new range is in their live map
    try {
        for (uint32_t i = 0; i < N; ++i) {
            if (!s.len[i]) continue;
            rec.ranges.push_back(Allocation{&rec, i, rec.gen, s.base[i], s.counts[i], s.len[i]});
            p.regions[i].live.emplace(s.base[i], &rec.ranges.back());
            linked = i + 1;
        }
    } catch (...) {
        for (uint32_t i = 0; i < linked; ++i)
            if (s.len[i]) p.regions[i].live.erase(s.base[i]);
        while (rec.ranges.size() > ranges_before) rec.ranges.pop_back();
        throw;
    }
    for (uint32_t i = 0; i < N; ++i)
        if (s.len[i]) p.regions[i].alloc.take(s.base[i], s.len[i]);   // first-fit starts: no allocation
    for (uint32_t j = 0; j < n; ++j) {
        const uint32_t r = region_of[j];
        const uint64_t off = s.base[r] + next[r]++ * p.block_bytes;
        out[j] = kvp_loc{r, rec.gen, off};
        p.glt.insert(GltEntry{rec.id, first + j, r, p.regions[r].desc.type, rec.gen, off});   // reserved
    }
    rec.n_blocks = first + n;
}

}  // namespace

void pool_place(Pool &p, uint64_t request, uint32_t n_blocks, kvp_loc *out)
{
    if (n_blocks == 0) fail(KVP_ERR_INVALID, "n_blocks must be positive");
    if (!out) fail(KVP_ERR_INVALID, "map_out is null");
    std::lock_guard<std::mutex> lock(p.mu);
    if (p.requests.count(request)) fail(KVP_ERR_INVALID, "request " + std::to_string(request) + " is already placed");
    const SetPlan plan = reserve_set(p, n_blocks);

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
    rec->gen = p.next_gen;
    RequestRec *r = rec.get();
    const hipEvent_t stored = rec->stored, busy = rec->busy;   // the record may be gone in the handler
    try {
        auto slot = p.requests.emplace(request, std::move(rec)).first;
        try {
            commit_set(p, *r, plan, 0, n_blocks, out);
        } catch (...) {
            p.requests.erase(slot);
            throw;
        }
    } catch (...) {
        if (stored) (void)hipEventDestroy(stored);
        if (busy) (void)hipEventDestroy(busy);
        throw;
    }
    ++p.next_gen;
}

void pool_extend(Pool &p, uint64_t request, uint32_t n_new, kvp_loc *out)
{
    if (n_new == 0) fail(KVP_ERR_INVALID, "n_new must be positive");
    if (!out) fail(KVP_ERR_INVALID, "map_out is null");
    std::lock_guard<std::mutex> lock(p.mu);
    auto it = p.requests.find(request);
    if (it == p.requests.end()) fail(KVP_ERR_NOTFOUND, "request " + std::to_string(request) + " is not placed");
    RequestRec &rec = *it->second;
    if (static_cast<uint64_t>(rec.n_blocks) + n_new > 0xFFFFFFFFull) fail(KVP_ERR_INVALID, "request too large");
    const SetPlan plan = reserve_set(p, n_new);
    commit_set(p, rec, plan, rec.n_blocks, n_new, out);
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
    // the only steps that can fail come first; from the first change on, nothing can
    std::vector<size_t> gives(p.regions.size(), 0);
    for (const auto &a : rec.ranges) ++gives[a.region];
    for (size_t i = 0; i < gives.size(); ++i)
        if (gives[i]) p.regions[i].alloc.reserve_gives(gives[i]);
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

}  // namespace kvp

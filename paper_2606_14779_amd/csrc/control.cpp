// Runtime control and introspection of a pool: measured region bandwidths
// (Sec. 4.1.2, the pool organizer's input to Eq. 1), region information and
// reads, launch settings of the two kernel classes, the copy-engine ring, and
// the HIP-event timing of store / retrieve calls.

#include <fcntl.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cstring>

#include "internal.hpp"

namespace kvp {

// ---------------------------------------------------------------- measured bandwidths (Sec. 4.1.2)

// Read rates of file regions, MB/s, through the path a retrieve takes: the
// region's worker thread reads its file into the pool's pinned ring (through
// its own aligned buffer).  A created file is measured on a probe file of its
// own beside it, written first by the same worker, since a range that was
// never written reads without touching the device; a block device is read in
// place from its start.  Each region reads n bytes per pass (its share of the
// ring, at most probe_bytes), one pass to warm up and the best of 3 after it.
// Alone: one region at a time.  Together: every region at once, as a retrieve
// reads them, so that regions sharing a device each get the rate they sustain
// beside the others.  The GPU's move out of the ring is not timed; it runs
// far faster.  Caller holds the pool lock; nothing else uses the ring.
void measure_file_regions(Pool &p, uint64_t probe_bytes, bool together, uint64_t *mbps)
{
    std::vector<size_t> idx;
    for (size_t r = 0; r < p.regions.size(); ++r)
        if (p.regions[r].desc.type == KVP_REGION_FILE) idx.push_back(r);
    if (idx.empty()) return;
    if (!p.file_ring)   // only after a kv_pool_set_file_ring that could not allocate
        fail(KVP_ERR_NOMEM, "file-region ring not allocated: set a smaller one with kv_pool_set_file_ring");
    for (uint32_t j = 0; j < kFileSlots; ++j) {   // the ring is idle
        io_drain(p.file_io[j]);
        if (p.file_free_rec[j]) check_hip(hipEventSynchronize(p.file_free[j]), "hipEventSynchronize");
    }
    const uint64_t share = kFileSlots * p.file_slot_bytes / idx.size() / kSector * kSector;
    struct Probe {
        const Region *r = nullptr;
        uint64_t n = 0;
        char *buf = nullptr;      // its part of the ring
        int fd = -1;
        std::string path;         // own probe file, removed afterwards
        IoGroup g;
        double best = 0.0;
        ~Probe()
        {
            io_drain(g);
            if (!path.empty()) {
                if (fd >= 0) ::close(fd);
                ::unlink(path.c_str());
            }
        }
    };
    std::vector<std::unique_ptr<Probe>> ps;
    for (size_t i = 0; i < idx.size(); ++i) {
        ps.push_back(std::make_unique<Probe>());
        Probe &q = *ps.back();
        q.r = &p.regions[idx[i]];
        q.n = std::max<uint64_t>(kSector, std::min({probe_bytes, q.r->capacity, share}) / kSector * kSector);
        q.buf = p.file_ring + i * share;
        q.fd = q.r->fd;
        if (q.r->file_owned) {
            const std::string path = q.r->file_path + ".probe";
            const int oflags =
                O_RDWR | O_CLOEXEC | O_CREAT | O_EXCL | ((q.r->flags_used & KVP_FILE_BUFFERED) ? 0 : O_DIRECT);
            q.fd = ::open(path.c_str(), oflags, 0600);
            if (q.fd < 0) fail(KVP_ERR_IO, "cannot create probe file " + path + ": " + std::strerror(errno));
            q.path = path;
            std::memset(q.buf, 0x5a, static_cast<size_t>(q.n));
            p.workers->submit(q.r->worker, IoJob{q.fd, true, 0, q.n, q.buf, &q.g});
            io_wait(q.g);
            if (::fsync(q.fd) != 0) fail(KVP_ERR_IO, "probe file " + path + ": " + std::strerror(errno));
        }
    }
    auto start = [&](Probe &q) {
        p.workers->submit(q.r->worker, IoJob{q.fd, false, 0, q.n, q.buf, &q.g});
    };
    auto finish = [&](Probe &q, std::chrono::steady_clock::time_point t0, bool timed) {
        io_wait(q.g);
        const double s = std::chrono::duration<double>(q.g.done_at - t0).count();
        if (timed && s > 0.0 && (q.best == 0.0 || s < q.best)) q.best = s;
    };
    double group_best = 0.0;   // together: the time until the last region finished
    for (int it = 0; it < 4; ++it) {
        if (together) {
            const auto t0 = std::chrono::steady_clock::now();
            for (auto &q : ps) start(*q);
            double last = 0.0;
            for (auto &q : ps) {
                finish(*q, t0, false);
                last = std::max(last, std::chrono::duration<double>(q->g.done_at - t0).count());
            }
            if (it > 0 && last > 0.0 && (group_best == 0.0 || last < group_best)) group_best = last;
        } else {
            for (auto &q : ps) {
                const auto t0 = std::chrono::steady_clock::now();
                start(*q);
                finish(*q, t0, it > 0);
            }
        }
    }
    // together, each region is credited with its bytes over the whole group's time, so the
    // rates add up to what the regions deliver at once (a retrieve waits for the last one)
    for (size_t i = 0; i < idx.size(); ++i) {
        const double t = together ? group_best : ps[i]->best;
        const double rate = t > 0.0 ? static_cast<double>(ps[i]->n) / t / 1e6 : 1.0;
        mbps[idx[i]] = std::max<uint64_t>(1, static_cast<uint64_t>(rate + 0.5));
    }
}


// An HBM region is read over at least this many bytes: a shorter copy leaves
// much of its writes in the GPU's 256 MB last-level cache when the kernel
// ends, and measures above the sustained rate (3.0-3.4 TB/s copied at 128-256
// MiB with non-temporal loads, 2.6-2.8 from 512 MiB on, against about 2.8 for
// a 17 GB gather).
constexpr uint64_t kHbmProbeMin = 1ull << 30;

// Bytes the probe of region r streams.
static uint64_t probe_span(const Region &r, uint64_t probe_bytes)
{
    const uint64_t want = r.desc.type == KVP_REGION_STAGING ? std::max(probe_bytes, kHbmProbeMin) : probe_bytes;
    return std::min<uint64_t>(want, r.capacity) & ~15ull;
}

// Read rate of every region (bytes from the region into HBM per second, in
// MB/s): the region-class kernel's launch shape streams probe_span bytes from
// the region into a scratch buffer; best of 3 after one warm-up.  Caller
// holds the pool lock and the device scope.
void measure_regions(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps)
{
    probe_bytes &= ~15ull;
    uint64_t scratch_bytes = 16;
    for (const Region &r : p.regions)
        if (r.desc.type != KVP_REGION_FILE) scratch_bytes = std::max(scratch_bytes, probe_span(r, probe_bytes));
    void *scratch = nullptr;
    if (hipMalloc(&scratch, scratch_bytes) != hipSuccess || !scratch) {
        clear_hip_error();
        fail(KVP_ERR_NOMEM, "probe scratch of " + std::to_string(scratch_bytes) + " bytes");
    }
    hipEvent_t e0 = nullptr, e1 = nullptr;
    try {
        check_hip(hipEventCreate(&e0), "hipEventCreate");
        check_hip(hipEventCreate(&e1), "hipEventCreate");
        uint32_t n_host = 0, n_staging = 0;
        for (size_t r = 0; r < p.regions.size(); ++r) {
            const Region &reg = p.regions[r];
            if (reg.desc.type == KVP_REGION_FILE) continue;   // below, all file regions together or one by one
            const uint32_t cls = reg.desc.type == KVP_REGION_HOST ? KVP_CLASS_HOST : KVP_CLASS_STAGING;
            n_host += cls == KVP_CLASS_HOST;
            n_staging += cls == KVP_CLASS_STAGING;
            hipStream_t st = p.s_stage;   // one probe at a time
            const uint64_t n = probe_span(reg, probe_bytes);
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
        // file regions: their files read into the pinned ring by their workers
        measure_file_regions(p, probe_bytes, (flags & KVP_MEASURE_FILES_TOGETHER) != 0, mbps);
        // host regions reach the GPU over one shared link: split what one measured alone
        if ((flags & KVP_MEASURE_SHARED_LINK) && n_host > 1)
            for (size_t r = 0; r < p.regions.size(); ++r)
                if (p.regions[r].desc.type == KVP_REGION_HOST) mbps[r] = std::max<uint64_t>(1, mbps[r] / n_host);
        // staging regions are all read from the one GPU's HBM: the same split
        if ((flags & KVP_MEASURE_SHARED_HBM) && n_staging > 1)
            for (size_t r = 0; r < p.regions.size(); ++r)
                if (p.regions[r].desc.type == KVP_REGION_STAGING) mbps[r] = std::max<uint64_t>(1, mbps[r] / n_staging);
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

void pool_measure(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps_out)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool has no memory to measure");
    if (!mbps_out) fail(KVP_ERR_INVALID, "null output");
    if (flags & ~(KVP_MEASURE_SHARED_LINK | KVP_MEASURE_FILES_TOGETHER | KVP_MEASURE_SHARED_HBM))
        fail(KVP_ERR_INVALID, "unknown flags");
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
    std::lock_guard<std::mutex> lock(p.mu);   // the bandwidth may be set meanwhile
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
    if (r.desc.type == KVP_REGION_FILE) {
        file_region_read(r, offset, bytes, dst);
    } else if (r.host) {
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
                  KVP_LAUNCH_SDMA | KVP_LAUNCH_CHUNK_MAJOR | KVP_LAUNCH_UPLOAD | KVP_LAUNCH_TILE))
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
    p.launch[cls][op] = LaunchCfg{grid ? grid : default_grid(cls, op, p.spec), flags, grid == 0};   // flags as given
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

void pool_set_file_ring(Pool &p, uint64_t slot_bytes)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool launches nothing");
    if (slot_bytes % kSector || slot_bytes < (64u << 10) || slot_bytes > (1ull << 36))
        fail(KVP_ERR_INVALID, "slot_bytes must be a multiple of 4096 in [64 KiB, 64 GiB]");
    std::lock_guard<std::mutex> lock(p.mu);
    if (!p.workers) fail(KVP_ERR_INVALID, "the pool has no file region");
    DeviceScope dev(p.device);
    free_file_ring(p);
    alloc_file_ring(p, slot_bytes);
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

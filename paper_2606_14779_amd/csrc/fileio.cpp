// File-backed pool regions (KVP_REGION_FILE): the storage tier of the pool.
//
// The paper keeps part of the pool on SSDs and reaches them through its
// KV-passthrough (Sec. 4.2): each offload set of a device is one contiguous
// range of ceil(|set| * KV_size / sector) sectors, written and read directly
// by the device's own worker thread (Sec. 4.1.3, Algorithm 1's SSD store;
// Sec. 4.3, the SSD reads of a retrieval).  Here a file region is a file (or
// a block device) opened with O_DIRECT, so reads and writes bypass the page
// cache; each region has one worker thread that runs its reads and writes.
// A request's share of the region is the same contiguous, sector-aligned
// range the allocator gives every region type.
//
// Between the file and the engine cache the bytes pass through a ring of two
// pinned, GPU-mapped host buffers ("slots").  A retrieve reads a batch of
// blocks into a slot (the workers, in parallel over the regions), then a
// kernel moves the slot to the engine cache on the caller's stream while the
// next batch is read into the other slot.  A store runs the other way: the
// kernel fills a slot from the engine cache, the host waits for it, and the
// workers write the slot's spans while the kernel fills the other slot.
//
// Every region offset, block size and layer range of a pool with file
// regions is a multiple of the 4096-byte sector (kv_pool_create checks that
// twice the chunk size is), so every span is sector aligned and no span ever
// shares a sector with another.

#include <fcntl.h>
#include <linux/fs.h>
#include <sys/ioctl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <chrono>
#include <cstdlib>
#include <cstring>

#include "internal.hpp"

namespace kvp {

// ---------------------------------------------------------------- plan

void plan_file(const FileGeometry &g, std::vector<HostBlock> &blocks, uint64_t skip, uint64_t width, uint32_t chunk0,
               std::vector<CopyItem> &items, std::vector<FileSpan> &spans, std::vector<FileBatch> &batches)
{
    // by region, then by offset: neighbouring blocks of a region merge into one span
    std::stable_sort(blocks.begin(), blocks.end(), [](const HostBlock &a, const HostBlock &b) {
        return a.region != b.region ? a.region < b.region : a.offset < b.offset;
    });
    // Every batch takes each region's blocks in proportion to the region's share of the
    // call, so all of the regions' workers read (or write) during every batch.  The
    // regions are merged by each block's place in its own region, (2i + 1) / (2 n_r) for
    // the i-th of n_r blocks (ties by region); a batch is the next `per` blocks of that
    // order, grouped by region again, where each region's blocks stay in offset order.
    const uint64_t per = std::max<uint64_t>(1, g.slot_bytes / width);
    if (blocks.size() > per) {
        struct Ranked {
            HostBlock b;
            uint64_t i, n;   // place in its region, blocks of its region
        };
        std::vector<Ranked> order;
        order.reserve(blocks.size());
        for (size_t s = 0; s < blocks.size();) {
            size_t e = s;
            while (e < blocks.size() && blocks[e].region == blocks[s].region) ++e;
            for (size_t k = s; k < e; ++k) order.push_back(Ranked{blocks[k], k - s, e - s});
            s = e;
        }
        std::stable_sort(order.begin(), order.end(), [](const Ranked &a, const Ranked &b) {
            const unsigned __int128 x = static_cast<unsigned __int128>(2 * a.i + 1) * b.n;
            const unsigned __int128 y = static_cast<unsigned __int128>(2 * b.i + 1) * a.n;
            return x != y ? x < y : a.b.region < b.b.region;
        });
        for (size_t s = 0; s < order.size(); s += per) {
            const auto e = order.begin() + static_cast<std::ptrdiff_t>(std::min<uint64_t>(order.size(), s + per));
            std::stable_sort(order.begin() + static_cast<std::ptrdiff_t>(s), e,
                             [](const Ranked &a, const Ranked &b) { return a.b.region < b.b.region; });
        }
        for (size_t k = 0; k < order.size(); ++k) blocks[k] = order[k].b;
    }
    const uint64_t back = static_cast<uint64_t>(chunk0) * g.chunk_bytes;   // the kernel adds (chunk0 + k) chunks
    uint32_t ring = g.next;
    uint64_t used = g.slot_bytes;   // forces a new batch for the first block
    for (const HostBlock &b : blocks) {
        if (used + width > g.slot_bytes) {
            if (!batches.empty()) ring = (ring + 1) % g.slots;
            batches.push_back(FileBatch{ring, static_cast<uint32_t>(items.size()), 0, spans.size(), 0});
            used = 0;
        }
        FileBatch &bt = batches.back();
        const uint64_t file_off = b.offset + skip;
        if (bt.spans && width == g.block_bytes) {
            FileSpan &last = spans.back();
            if (last.region == b.region && last.file_off + last.len == file_off && last.slot_off + last.len == used) {
                last.len += width;   // the previous span reaches this block: extend it
            } else {
                spans.push_back(FileSpan{b.region, file_off, width, used});
                ++bt.spans;
            }
        } else {
            spans.push_back(FileSpan{b.region, file_off, width, used});
            ++bt.spans;
        }
        items.push_back(CopyItem{g.base + static_cast<uint64_t>(ring) * g.slot_bytes + used - back, b.slot, 0u});
        ++bt.n;
        used += width;
    }
}

// ---------------------------------------------------------------- worker threads

namespace {

constexpr uint64_t kWorkerBounce = 16ull << 20;   // per-worker buffer of the file side

// One read or write of a whole span; a short transfer is continued, an
// interrupted one retried.  With a bounce buffer, the file side reads into
// or writes from that (ordinary, page-aligned) buffer piece by piece and the
// piece is copied to or from j.buf: the pinned ring slots are driver memory,
// which direct I/O cannot pin (it fails with EFAULT).  Returns 0 or an
// errno, with a message.
int transfer(const IoJob &j, std::string &what, char *bounce = nullptr, uint64_t bounce_bytes = 0)
{
    uint64_t done = 0;
    while (done < j.len) {
        const uint64_t piece = std::min<uint64_t>(j.len - done, bounce ? bounce_bytes : (1ull << 30));
        char *io = bounce ? bounce : j.buf + done;
        if (bounce && j.write) std::memcpy(bounce, j.buf + done, piece);
        uint64_t got = 0;
        while (got < piece) {
            const size_t want = static_cast<size_t>(piece - got);
            const off_t at = static_cast<off_t>(j.off + done + got);
            const ssize_t r = j.write ? ::pwrite(j.fd, io + got, want, at) : ::pread(j.fd, io + got, want, at);
            if (r < 0) {
                if (errno == EINTR) continue;
                const int e = errno;
                what = std::string(j.write ? "write" : "read") + " of " + std::to_string(j.len) +
                       " bytes at offset " + std::to_string(j.off) + ": " + std::strerror(e);
                return e;
            }
            if (r == 0) {
                what = std::string(j.write ? "write" : "read") + " at offset " + std::to_string(j.off + done + got) +
                       ": end of file";
                return EIO;
            }
            got += static_cast<uint64_t>(r);
        }
        if (bounce && !j.write) std::memcpy(j.buf + done, bounce, piece);
        done += piece;
    }
    return 0;
}

}  // namespace

FileWorkers::FileWorkers(size_t n)
{
    w_.reserve(n);
    try {
        for (size_t i = 0; i < n; ++i) {
            w_.push_back(std::make_unique<Worker>());
            Worker *w = w_.back().get();
            w->th = std::thread([w] { run(*w); });
        }
    } catch (...) {
        shutdown();
        throw;
    }
}

FileWorkers::~FileWorkers() { shutdown(); }

void FileWorkers::shutdown()
{
    for (auto &w : w_) {
        {
            std::lock_guard<std::mutex> lock(w->mu);
            w->stop = true;
        }
        w->cv.notify_one();
    }
    for (auto &w : w_)
        if (w->th.joinable()) w->th.join();
    w_.clear();
}

void FileWorkers::submit(size_t worker, const IoJob &job)
{
    Worker &w = *w_.at(worker);
    {
        std::lock_guard<std::mutex> g(job.group->mu);
        ++job.group->pending;
    }
    try {
        std::lock_guard<std::mutex> lock(w.mu);
        w.q.push_back(job);
    } catch (...) {   // not queued: take it back off the count, or a wait on the group never ends
        std::lock_guard<std::mutex> g(job.group->mu);
        if (--job.group->pending == 0) job.group->cv.notify_all();
        throw;
    }
    w.cv.notify_one();
}

void FileWorkers::run(Worker &w)
{
    void *bounce = nullptr;   // the worker's own page-aligned buffer for the file side
    if (::posix_memalign(&bounce, kSector, kWorkerBounce) != 0) bounce = nullptr;
    for (;;) {
        IoJob j;
        {
            std::unique_lock<std::mutex> lock(w.mu);
            w.cv.wait(lock, [&] { return w.stop || !w.q.empty(); });
            if (w.q.empty()) {     // stopping, nothing left
                std::free(bounce);
                return;
            }
            j = w.q.front();
            w.q.pop_front();
        }
        std::string what;
        int err = 0;
        try {
            if (bounce)
                err = transfer(j, what, static_cast<char *>(bounce), kWorkerBounce);
            else {
                err = ENOMEM;
                what = "no buffer for the worker thread";
            }
        } catch (...) {   // a message that cannot be built: keep the code
            err = err ? err : ENOMEM;
        }
        {
            std::lock_guard<std::mutex> g(j.group->mu);
            if (err && !j.group->err) {
                j.group->err = err;
                try {
                    j.group->what.swap(what);
                } catch (...) {
                }
            }
            if (--j.group->pending == 0) j.group->done_at = std::chrono::steady_clock::now();
            // notified under the lock: a waiter that sees pending == 0 may destroy the
            // group at once, so the group is not touched after the lock is released
            j.group->cv.notify_all();
        }
    }
}

void io_wait(IoGroup &g)
{
    std::unique_lock<std::mutex> lock(g.mu);
    g.cv.wait(lock, [&] { return g.pending == 0; });
    if (g.err) {
        const std::string what = g.what.empty() ? std::string(std::strerror(g.err)) : g.what;
        g.err = 0;
        g.what.clear();
        fail(KVP_ERR_IO, "file region " + what);
    }
}

void io_drain(IoGroup &g) noexcept
{
    std::unique_lock<std::mutex> lock(g.mu);
    g.cv.wait(lock, [&] { return g.pending == 0; });
    g.err = 0;
    g.what.clear();
}

// ---------------------------------------------------------------- region life cycle

void open_file_region(Region &r, const char *path)
{
    if (!path || !*path) fail(KVP_ERR_INVALID, "file region without a path");
    const bool direct = !(r.desc.flags & KVP_FILE_BUFFERED);
    const int oflags = O_RDWR | O_CLOEXEC | (direct ? O_DIRECT : 0);
    struct stat st;
    if (::stat(path, &st) == 0) {
        // an existing path is used only if it is a block device (read and written in place)
        if (!S_ISBLK(st.st_mode))
            fail(KVP_ERR_INVALID, std::string("file region ") + path + " exists and is not a block device (not overwritten)");
        const int fd = ::open(path, oflags);
        if (fd < 0) fail(KVP_ERR_INVALID, std::string("cannot open ") + path + ": " + std::strerror(errno));
        uint64_t size = 0;
        if (::ioctl(fd, BLKGETSIZE64, &size) != 0 || size < r.capacity) {
            ::close(fd);
            fail(KVP_ERR_INVALID, std::string("block device ") + path + " is smaller than the region's capacity");
        }
        r.fd = fd;
        r.file_owned = false;
    } else {
        if (errno != ENOENT) fail(KVP_ERR_INVALID, std::string("cannot stat ") + path + ": " + std::strerror(errno));
        const int fd = ::open(path, oflags | O_CREAT | O_EXCL, 0600);
        if (fd < 0) {
            const int e = errno;
            fail(KVP_ERR_INVALID, std::string("cannot create ") + path + ": " + std::strerror(e) +
                                      (e == EINVAL && direct ? " (no O_DIRECT on this file system: KVP_FILE_BUFFERED)" : ""));
        }
        // the region's blocks are reserved on the disk now, so a later store cannot run out of
        // space part-way and writes do not allocate; a file system without fallocate gets a sparse file
        if (::fallocate(fd, 0, 0, static_cast<off_t>(r.capacity)) != 0) {
            const int e = errno;
            const bool unsupported = e == EOPNOTSUPP || e == ENOSYS || e == EINVAL;
            if (!unsupported || ::ftruncate(fd, static_cast<off_t>(r.capacity)) != 0) {
                const int e2 = unsupported ? errno : e;
                ::close(fd);
                ::unlink(path);
                fail(KVP_ERR_IO, std::string("cannot reserve ") + std::to_string(r.capacity) + " bytes for " + path +
                                     ": " + std::strerror(e2));
            }
        }
        r.fd = fd;
        r.file_owned = true;
    }
    r.file_path = path;
    r.flags_used = r.desc.flags;
}

void close_file_region(Region &r) noexcept
{
    if (r.fd >= 0) ::close(r.fd);
    if (r.file_owned && !r.file_path.empty()) ::unlink(r.file_path.c_str());
    r.fd = -1;
    r.file_owned = false;
}

void file_region_read(const Region &r, uint64_t offset, uint64_t bytes, void *dst)
{
    // O_DIRECT wants sector-aligned offsets, lengths and buffers: read the
    // aligned span into an aligned buffer, then copy out
    const uint64_t lo = offset / kSector * kSector, hi = round_up(offset + bytes, kSector);
    const uint64_t step = 64ull << 20;
    void *buf = nullptr;
    if (::posix_memalign(&buf, kSector, static_cast<size_t>(std::min(hi - lo, step))) != 0 || !buf)
        fail(KVP_ERR_NOMEM, "aligned read buffer");
    try {
        for (uint64_t at = lo; at < hi; at += step) {
            const uint64_t n = std::min(step, hi - at);
            IoJob j{r.fd, false, at, n, static_cast<char *>(buf), nullptr};
            std::string what;
            if (const int e = transfer(j, what)) {
                (void)e;
                fail(KVP_ERR_IO, "file region " + what);
            }
            const uint64_t from = std::max(at, offset), to = std::min(at + n, offset + bytes);
            if (from < to)
                std::memcpy(static_cast<char *>(dst) + (from - offset), static_cast<char *>(buf) + (from - at), to - from);
        }
    } catch (...) {
        std::free(buf);
        throw;
    }
    std::free(buf);
}

}  // namespace kvp

// The storage tier's host side, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_native_asan.py (CPU only):
//
//   plan_file     random file-class blocks, layer ranges and slot sizes: every
//                 block has exactly one work item; its part lies inside one
//                 span of its own region, at the span's matching place in the
//                 batch's slot; spans of a batch do not overlap in the slot and
//                 fit it; batches take the ring's slots in turn; whole blocks
//                 at consecutive offsets of a region share a span; every batch
//                 but the last is full, and after every batch each region has
//                 sent its proportional share of the blocks, to within the
//                 merge's bound (all regions busy in every batch)
//   FileWorkers   one worker per file, O_DIRECT files in a temporary
//                 directory: spans written from an aligned buffer by the
//                 workers and read back by them equal the bytes written; a
//                 read past the end of a file is reported by io_wait as
//                 KVP_ERR_IO with its message, and the group is usable again;
//                 two host threads submitting to the same workers at once,
//                 each with its own group, get their own spans back
//   file regions  open_file_region creates and sizes a file, refuses an
//                 existing regular file, and close_file_region removes what
//                 it created; file_region_read returns unaligned ranges
//
// Only fileio.cpp (and placement.cpp, for the Region it fills) is linked; the
// error helper they call is defined here.
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <string>
#include <thread>
#include <vector>

#include "internal.hpp"

namespace kvp {
void fail(int code, const std::string &msg) { throw Error{code, msg}; }
}  // namespace kvp

using namespace kvp;

#define CHECK(c)                                                                 \
    do {                                                                         \
        if (!(c)) {                                                              \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            std::exit(1);                                                        \
        }                                                                        \
    } while (0)

static void plan_properties(std::mt19937_64 &rng)
{
    for (int iter = 0; iter < 3000; ++iter) {
        const uint64_t chunk = kSector / 2 * (1 + rng() % 4);          // 2 * chunk is a sector multiple
        const uint32_t layers = 1 + rng() % 6;
        const uint64_t bb = 2ull * layers * chunk;
        const uint32_t l0 = rng() % layers, l1 = l0 + 1 + rng() % (layers - l0);
        const uint64_t skip = 2ull * l0 * chunk, width = 2ull * (l1 - l0) * chunk;
        const uint32_t n_regions = 1 + rng() % 4;
        const uint32_t n = rng() % 60;
        // blocks: per region a run of consecutive offsets, some holes, order shuffled or not
        std::vector<HostBlock> blocks;
        std::set<std::pair<uint32_t, uint64_t>> seen;
        for (uint32_t b = 0; b < n; ++b) {
            const uint32_t r = rng() % n_regions;
            uint64_t k = rng() % 80;
            while (seen.count({r, k})) k = (k + 1) % 4096;
            seen.insert({r, k});
            blocks.push_back(HostBlock{r, (r * 7 % 3) * 16 * kSector + k * bb, b});   // a base per region
        }
        const std::vector<HostBlock> orig = blocks;   // block b has slot b
        if (rng() % 2) std::shuffle(blocks.begin(), blocks.end(), rng);
        const uint64_t slot_bytes = width * (1 + rng() % 9) + (rng() % 2) * kSector;
        const uint32_t slots = 2, next = rng() % 2;
        const uint64_t base = 1ull << 40;
        const FileGeometry g{base, slot_bytes, slots, next, bb, chunk};
        std::vector<CopyItem> items;
        std::vector<FileSpan> spans;
        std::vector<FileBatch> batches;
        plan_file(g, blocks, skip, width, 2 * l0, items, spans, batches);
        CHECK(items.size() == orig.size());
        std::vector<int> hits(orig.size(), 0);
        uint32_t expect_ring = next;
        size_t items_seen = 0, spans_seen = 0;
        for (size_t bi = 0; bi < batches.size(); ++bi) {
            const FileBatch &bt = batches[bi];
            CHECK(bt.ring == expect_ring);
            expect_ring = (expect_ring + 1) % slots;
            CHECK(bt.first == items_seen && bt.span0 == spans_seen && bt.n > 0 && bt.spans > 0);
            items_seen += bt.n;
            spans_seen += bt.spans;
            // spans of the batch: sector aligned, inside the slot, disjoint in the slot
            std::vector<std::pair<uint64_t, uint64_t>> used;
            for (size_t s = bt.span0; s < bt.span0 + bt.spans; ++s) {
                const FileSpan &sp = spans[s];
                CHECK(sp.file_off % kSector == 0 && sp.len % kSector == 0 && sp.slot_off % kSector == 0 && sp.len > 0);
                CHECK(sp.slot_off + sp.len <= slot_bytes);
                for (auto &u : used) CHECK(sp.slot_off + sp.len <= u.first || u.second <= sp.slot_off);
                used.push_back({sp.slot_off, sp.slot_off + sp.len});
            }
            // every item: its block's part inside one span of the block's region, at the matching place
            for (uint32_t i = bt.first; i < bt.first + bt.n; ++i) {
                const CopyItem &it = items[i];
                CHECK(it.slot < orig.size());
                ++hits[it.slot];
                const HostBlock &blk = orig[it.slot];                 // slot numbers were the block indices
                const uint64_t in_slot = it.pool + 2ull * l0 * chunk - base - static_cast<uint64_t>(bt.ring) * slot_bytes;
                int found = 0;
                for (size_t s = bt.span0; s < bt.span0 + bt.spans; ++s) {
                    const FileSpan &sp = spans[s];
                    if (sp.region != blk.region) continue;
                    const uint64_t f = blk.offset + skip;
                    if (f >= sp.file_off && f + width <= sp.file_off + sp.len) {
                        CHECK(in_slot == sp.slot_off + (f - sp.file_off));
                        ++found;
                    }
                }
                CHECK(found == 1);
            }
        }
        CHECK(items_seen == items.size() && spans_seen == spans.size());
        for (int h : hits) CHECK(h == 1);
        // full batches, and each region's share of the first m blocks: |c_r - m n_r / n| <= 1/2 + R n_r / (2 n)
        const uint64_t per = slot_bytes / width;
        std::vector<int64_t> n_r(n_regions, 0), c_r(n_regions, 0);
        for (const HostBlock &b : orig) ++n_r[b.region];
        int64_t m = 0;
        const int64_t nn = static_cast<int64_t>(orig.size());
        for (size_t bi = 0; bi < batches.size(); ++bi) {
            if (bi + 1 < batches.size()) CHECK(batches[bi].n == per);
            for (uint32_t i = batches[bi].first; i < batches[bi].first + batches[bi].n; ++i) ++c_r[orig[items[i].slot].region];
            m += batches[bi].n;
            for (uint32_t r = 0; r < n_regions; ++r)
                CHECK(2 * std::llabs(c_r[r] * nn - m * n_r[r]) <= nn + static_cast<int64_t>(n_regions) * n_r[r]);
        }
        // whole blocks of one region at consecutive offsets in one slot: one span
        if (width == bb)
            for (size_t s = 1; s < spans.size(); ++s)
                if (spans[s].region == spans[s - 1].region && spans[s - 1].file_off + spans[s - 1].len == spans[s].file_off &&
                    spans[s - 1].slot_off + spans[s - 1].len == spans[s].slot_off) {
                    // allowed only across a batch boundary
                    bool boundary = false;
                    for (const FileBatch &bt : batches) boundary |= bt.span0 == s;
                    CHECK(boundary);
                }
    }
}

static std::string temp_dir()
{
    char tmpl[] = "/tmp/kvpool-fileio-XXXXXX";
    const char *d = ::mkdtemp(tmpl);
    CHECK(d != nullptr);
    return d;
}

static void workers_round_trip(std::mt19937_64 &rng, const std::string &dir)
{
    const int n_files = 3;
    const uint64_t file_bytes = 64 * kSector;
    std::vector<int> fds;
    std::vector<std::string> names;
    for (int f = 0; f < n_files; ++f) {
        names.push_back(dir + "/w" + std::to_string(f));
        int fd = ::open(names.back().c_str(), O_RDWR | O_CREAT | O_EXCL | O_DIRECT, 0600);
        bool direct = fd >= 0;
        if (fd < 0) fd = ::open(names.back().c_str(), O_RDWR | O_CREAT | O_EXCL, 0600);   // no O_DIRECT here
        CHECK(fd >= 0);
        (void)direct;
        CHECK(::ftruncate(fd, static_cast<off_t>(file_bytes)) == 0);
        fds.push_back(fd);
    }
    const uint64_t buf_bytes = n_files * file_bytes;
    char *out = nullptr, *in = nullptr;
    CHECK(::posix_memalign(reinterpret_cast<void **>(&out), kSector, buf_bytes) == 0);
    CHECK(::posix_memalign(reinterpret_cast<void **>(&in), kSector, buf_bytes) == 0);
    for (uint64_t i = 0; i < buf_bytes; ++i) out[i] = static_cast<char>(rng());
    std::memset(in, 0, buf_bytes);
    {
        FileWorkers w(n_files);
        IoGroup g;
        for (int round = 0; round < 20; ++round) {
            // random sector-aligned spans of every file, written, then read back into the same place
            std::vector<IoJob> jobs;
            for (int f = 0; f < n_files; ++f) {
                const uint64_t a = (rng() % 64) * kSector, len = (1 + rng() % (64 - a / kSector)) * kSector;
                jobs.push_back(IoJob{fds[f], true, a, len, out + f * file_bytes + a, &g});
            }
            for (size_t j = 0; j < jobs.size(); ++j) w.submit(j, jobs[j]);
            io_wait(g);
            for (size_t j = 0; j < jobs.size(); ++j) {
                IoJob r = jobs[j];
                r.write = false;
                r.buf = in + (r.buf - out);
                w.submit(j, r);
            }
            io_wait(g);
            for (const IoJob &j : jobs) CHECK(std::memcmp(in + (j.buf - out), j.buf, j.len) == 0);
        }
        // a read past the end of a file: reported once, then the group works again
        w.submit(0, IoJob{fds[0], false, file_bytes, kSector, in, &g});
        bool threw = false;
        try {
            io_wait(g);
        } catch (const Error &e) {
            threw = e.code == KVP_ERR_IO && e.msg.find("end of file") != std::string::npos;
        }
        CHECK(threw);
        w.submit(1, IoJob{fds[1], false, 0, kSector, in, &g});
        io_wait(g);
        // file 1's first sector: the bytes written there, or zeros if no span covered it
        bool zero = true;
        for (uint64_t i = 0; i < kSector; ++i) zero &= in[i] == 0;
        CHECK(zero || std::memcmp(in, out + file_bytes, kSector) == 0);

        // two submitters at once: each writes its own half of every file, then reads it back
        const uint64_t half = file_bytes / 2;
        std::vector<char> ok(2, 0);
        auto submitter = [&](int t) {
            IoGroup mine;
            char *src = out + t * half, *dst = in + t * half;   // [t*half, t*half + half) of each file's slice
            for (int round = 0; round < 10; ++round) {
                for (int f = 0; f < n_files; ++f)
                    w.submit(f, IoJob{fds[f], true, t * half, half, src + f * file_bytes, &mine});
                io_wait(mine);
                for (int f = 0; f < n_files; ++f)
                    w.submit(f, IoJob{fds[f], false, t * half, half, dst + f * file_bytes, &mine});
                io_wait(mine);
            }
            bool same = true;
            for (int f = 0; f < n_files; ++f)
                same &= std::memcmp(dst + f * file_bytes, src + f * file_bytes, half) == 0;
            ok[t] = same;
        };
        std::memset(in, 0, buf_bytes);
        std::thread t0(submitter, 0), t1(submitter, 1);
        t0.join();
        t1.join();
        CHECK(ok[0] && ok[1]);
    }
    for (int f = 0; f < n_files; ++f) {
        ::close(fds[f]);
        ::unlink(names[f].c_str());
    }
    std::free(out);
    std::free(in);
}

static void region_life_cycle(const std::string &dir)
{
    Region r;
    r.desc.type = KVP_REGION_FILE;
    r.desc.numa_node = -1;
    r.desc.flags = 0;
    r.capacity = 40 * kSector;
    const std::string path = dir + "/region.bin";
    open_file_region(r, path.c_str());
    struct stat st;
    CHECK(::stat(path.c_str(), &st) == 0 && static_cast<uint64_t>(st.st_size) == r.capacity && r.file_owned);
    // reserved on the disk where the file system can (st_blocks counts 512-byte units)
    std::printf("region file: %llu bytes, %llu allocated\n", (unsigned long long)st.st_size,
                (unsigned long long)st.st_blocks * 512ull);
    // bytes written through the descriptor come back through file_region_read at unaligned ranges
    char *buf = nullptr;
    CHECK(::posix_memalign(reinterpret_cast<void **>(&buf), kSector, r.capacity) == 0);
    for (uint64_t i = 0; i < r.capacity; ++i) buf[i] = static_cast<char>(i * 131 + 7);
    CHECK(::pwrite(r.fd, buf, r.capacity, 0) == static_cast<ssize_t>(r.capacity));
    std::vector<char> got(r.capacity);
    for (uint64_t off : {0ull, 1ull, 4095ull, 4096ull, 12345ull})
        for (uint64_t len : {1ull, 100ull, 4096ull, 9000ull}) {
            if (off + len > r.capacity) continue;
            file_region_read(r, off, len, got.data());
            CHECK(std::memcmp(got.data(), buf + off, len) == 0);
        }
    // an existing regular file is refused, not overwritten
    Region r2 = Region();
    r2.desc = r.desc;
    r2.capacity = r.capacity;
    bool refused = false;
    try {
        open_file_region(r2, path.c_str());
    } catch (const Error &e) {
        refused = e.code == KVP_ERR_INVALID;
    }
    CHECK(refused && r2.fd < 0);
    close_file_region(r);
    CHECK(::stat(path.c_str(), &st) != 0);
    std::free(buf);
}

int main()
{
    std::mt19937_64 rng(2606);
    plan_properties(rng);
    const std::string dir = temp_dir();
    workers_round_trip(rng, dir);
    region_life_cycle(dir);
    ::rmdir(dir.c_str());
    std::printf("all checks passed\n");
    return 0;
}

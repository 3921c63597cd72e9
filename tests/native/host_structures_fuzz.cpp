// Randomised check of the library's host-side data structures, built with
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_native_asan.py.
//
//   RangeAllocator   against a byte-granular model of the free space, taking
//                    ranges at and inside free runs, with and without spare
//                    nodes reserved for give()
//   Glt              against std::map, through inserts, finds and the
//                    backward-shift deletions
//   target_counts    sum and per-region bounds of Eq. 2
//   stripe           every region receives exactly its count
//   plan_bounce      the copy-engine plan: every block exactly once, runs of
//                    consecutive offsets in one region, every byte a copy or
//                    the kernel touches inside its ring slot, and the
//                    kernel's addresses equal to the copies' addresses
//
// Only placement.cpp, glt.cpp and bounce.cpp are linked; the two error
// helpers they call are defined here.  Exit status 0 means every check held.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <vector>

#include "internal.hpp"

namespace kvp {
void fail(int code, const std::string &msg) { throw Error{code, msg}; }
void check_hip(hipError_t, const char *) {}
}  // namespace kvp

#define CHECK(c)                                                        \
    do {                                                                \
        if (!(c)) {                                                     \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            std::exit(1);                                               \
        }                                                               \
    } while (0)

static void allocator_against_model(std::mt19937_64 &rng)
{
    const uint64_t cap = 1 + rng() % 4096;
    kvp::RangeAllocator a(cap);
    std::vector<char> used(cap, 0);
    std::vector<std::pair<uint64_t, uint64_t>> live;
    for (int step = 0; step < 400; ++step) {
        if (!live.empty() && rng() % 3 == 0) {
            const size_t k = rng() % live.size();
            if (rng() % 2) a.reserve_gives(rng() % 4);   // spare nodes for give()
            a.give(live[k].first, live[k].second);
            for (uint64_t i = 0; i < live[k].second; ++i) used[live[k].first + i] = 0;
            live.erase(live.begin() + k);
        } else {
            const uint64_t len = 1 + rng() % 64;
            uint64_t start = 0;
            // model: lowest start of a free run of length >= len that begins a maximal free run
            uint64_t expect = UINT64_MAX;
            for (uint64_t i = 0; i < cap;) {
                if (used[i]) { ++i; continue; }
                uint64_t j = i;
                while (j < cap && !used[j]) ++j;
                if (j - i >= len) { expect = i; break; }
                i = j;
            }
            const bool ok = a.first_fit(len, &start);
            CHECK(ok == (expect != UINT64_MAX));
            if (!ok) continue;
            CHECK(start == expect);
            // now and then a range from inside the free run instead of its start
            uint64_t run_end = start;
            while (run_end < cap && !used[run_end]) ++run_end;
            if (rng() % 4 == 0 && run_end - start > len) start += rng() % (run_end - start - len + 1);
            a.take(start, len);
            for (uint64_t i = 0; i < len; ++i) {
                CHECK(!used[start + i]);
                used[start + i] = 1;
            }
            live.push_back({start, len});
        }
        uint64_t best = 0;
        for (uint64_t i = 0; i < cap;) {
            if (used[i]) { ++i; continue; }
            uint64_t j = i;
            while (j < cap && !used[j]) ++j;
            best = std::max(best, j - i);
            i = j;
        }
        CHECK(a.largest() == best);
    }
}

static void glt_against_map(std::mt19937_64 &rng)
{
    kvp::Glt g;
    std::map<std::pair<uint64_t, uint32_t>, uint64_t> ref;
    for (int step = 0; step < 20000; ++step) {
        const uint64_t req = rng() % 64;
        const uint32_t blk = static_cast<uint32_t>(rng() % 256);
        const int op = static_cast<int>(rng() % 3);
        if (op == 0) {
            const uint64_t off = rng();
            g.insert(kvp::GltEntry{req, blk, 1, 0, 7, off});
            ref[{req, blk}] = off;
        } else if (op == 1) {
            const bool had = ref.erase({req, blk}) > 0;
            CHECK(g.erase(req, blk) == had);
        }
        const kvp::GltEntry *e = g.find(req, blk);
        auto it = ref.find({req, blk});
        CHECK((e != nullptr) == (it != ref.end()));
        if (e) CHECK(e->offset == it->second && e->request == req && e->block == blk);
        CHECK(g.size() == ref.size());
    }
    for (const auto &kv : ref) {
        const kvp::GltEntry *e = g.find(kv.first.first, kv.first.second);
        CHECK(e && e->offset == kv.second);
    }
}

static void counts_and_stripe(std::mt19937_64 &rng)
{
    for (int t = 0; t < 2000; ++t) {
        const uint32_t N = 1 + rng() % 8;
        std::vector<uint64_t> w(N), c(N);
        for (auto &x : w) x = 1 + rng() % 1000;
        const uint32_t n = static_cast<uint32_t>(rng() % 5000);
        kvp::target_counts(w.data(), N, n, c.data());
        uint64_t sum = 0, W = 0;
        for (uint32_t i = 0; i < N; ++i) sum += c[i], W += w[i];
        CHECK(sum == n);
        for (uint32_t i = 0; i < N; ++i) {
            const uint64_t fl = w[i] * n / W;
            CHECK(c[i] == fl || c[i] == fl + 1);
        }
        std::vector<uint32_t> region_of;
        kvp::stripe(c, n, region_of);
        CHECK(region_of.size() == n);
        std::vector<uint64_t> got(N, 0);
        for (uint32_t r : region_of) {
            CHECK(r < N);
            ++got[r];
        }
        for (uint32_t i = 0; i < N; ++i) CHECK(got[i] == c[i]);
    }
    bool threw = false;
    try {
        uint64_t w0[2] = {1, 0}, c0[2];
        kvp::target_counts(w0, 2, 5, c0);
    } catch (const kvp::Error &e) {
        threw = e.code == KVP_ERR_INVALID;
    }
    CHECK(threw);
}

static void bounce_plan(std::mt19937_64 &rng)
{
    for (int t = 0; t < 3000; ++t) {
        const uint64_t chunk = 16 * (1 + rng() % 64);
        const uint32_t L = 1 + rng() % 6;
        const uint64_t block = 2 * L * chunk;
        kvp::RingGeometry g{0x100000000ull + 4096 * (rng() % 1000), block * (1 + rng() % 9) + 16 * (rng() % 4), 
                            static_cast<uint32_t>(1 + rng() % 4), 0, block, chunk};
        g.next = static_cast<uint32_t>(rng() % g.slots);
        const uint32_t l0 = rng() % L, l1 = l0 + 1 + rng() % (L - l0);
        const uint64_t width = 2ull * (l1 - l0) * chunk;
        // a few regions, each with one range of blocks, some entries dropped, in shuffled order
        const uint32_t N = 1 + rng() % 5;
        std::vector<kvp::HostBlock> in;
        uint32_t slot = 0;
        for (uint32_t r = 0; r < N; ++r) {
            const uint64_t base = block * (rng() % 50);
            const uint32_t cnt = rng() % 40;
            for (uint32_t k = 0; k < cnt; ++k)
                if (rng() % 5) in.push_back(kvp::HostBlock{r, base + k * block, slot++});
        }
        std::shuffle(in.begin(), in.end(), rng);
        std::vector<kvp::HostBlock> blocks = in;
        std::vector<kvp::CopyItem> items;
        std::vector<kvp::LinkRun> runs;
        std::vector<kvp::Batch> batches;
        kvp::plan_bounce(g, blocks, width, 2 * l0, items, runs, batches);
        CHECK(items.size() == in.size());
        std::map<uint32_t, std::pair<uint32_t, uint64_t>> seen;   // slot -> (region, offset)
        size_t next_item = 0, next_run = 0;
        for (size_t b = 0; b < batches.size(); ++b) {
            const kvp::Batch &bt = batches[b];
            CHECK(bt.ring == (g.next + b) % g.slots);
            CHECK(bt.first == next_item && bt.n > 0 && bt.run0 == next_run && bt.runs > 0);
            CHECK(bt.n <= g.slot_bytes / width);
            const uint64_t slot_base = g.base + bt.ring * g.slot_bytes;
            uint64_t packed = 0;
            size_t it = bt.first;
            for (size_t q = bt.run0; q < bt.run0 + bt.runs; ++q) {
                const kvp::LinkRun &run = runs[q];
                CHECK(run.slot_offset == packed && run.blocks > 0);
                CHECK(run.slot_offset + run.blocks * width <= g.slot_bytes);
                if (q > bt.run0) {      // a new run only where the previous one cannot continue
                    const kvp::LinkRun &prev = runs[q - 1];
                    CHECK(prev.region != run.region || prev.offset + prev.blocks * block != run.offset);
                }
                for (uint32_t k = 0; k < run.blocks; ++k, ++it) {
                    const kvp::CopyItem &ci = items[it];
                    // the kernel reads / writes [pool + chunk0*C, + width): the copy's bytes
                    CHECK(ci.pool + 2ull * l0 * chunk == slot_base + run.slot_offset + k * width);
                    CHECK(seen.count(ci.slot) == 0);
                    seen[ci.slot] = {run.region, run.offset + k * block};
                }
                packed += run.blocks * width;
            }
            CHECK(packed == bt.n * width && it == bt.first + bt.n);
            next_item += bt.n;
            next_run += bt.runs;
        }
        CHECK(next_item == items.size() && next_run == runs.size());
        CHECK(seen.size() == in.size());
        for (const kvp::HostBlock &hb : in) {
            auto f = seen.find(hb.slot);
            CHECK(f != seen.end() && f->second.first == hb.region && f->second.second == hb.offset);
        }
        // regions appear in order, each region's blocks in their input order
        for (size_t q = 1; q < runs.size(); ++q) CHECK(runs[q - 1].region <= runs[q].region);
    }
}

int main()
{
    std::mt19937_64 rng(12345);
    for (int i = 0; i < 40; ++i) allocator_against_model(rng);
    glt_against_map(rng);
    counts_and_stripe(rng);
    bounce_plan(rng);
    std::puts("host structures: all checks passed");
    return 0;
}

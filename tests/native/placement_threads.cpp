// Several threads using one placement-only pool (no GPU) at once through the
// C ABI, built with ThreadSanitizer by tests/test_native_tsan.py.
//
// Each thread owns its own request ids and runs a seeded sequence of place,
// extend, lookup and release calls, checking every lookup against the maps
// it was given and that its error messages are its own (the message is
// thread-local).  Other threads meanwhile set the weights (to the values they
// already have), read region descriptions and compute Eq. 2 counts.  After the join, the blocks of all live requests must sit
// in distinct places, and releasing them all must give every byte back: a
// request that fills every region exactly then fits.
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <random>
#include <set>
#include <thread>
#include <utility>
#include <vector>

#include "kvpool.h"

#define CHECK(c)                                                                      \
    do {                                                                              \
        if (!(c)) {                                                                   \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);      \
            std::exit(1);                                                             \
        }                                                                             \
    } while (0)

namespace {

constexpr uint32_t kRegions = 4;
constexpr int kWorkers = 6;
constexpr uint64_t kBlockBytes = 2ull * 2 * 256;   // 2 layers, 256-byte chunks
constexpr uint64_t kCapBlocks = 60;                // per unit of weight: 240/240/60/60 blocks

struct Live {
    std::map<uint64_t, std::vector<kvp_loc>> maps;
};

void worker(kvp_pool *pool, int id, Live *out, std::atomic<uint64_t> *refusals)
{
    std::mt19937_64 rng(1000 + id);
    Live &live = *out;
    uint64_t next = (static_cast<uint64_t>(id) << 32) + 1;
    for (int op = 0; op < 400; ++op) {
        const int kind = live.maps.empty() ? 0 : static_cast<int>(rng() % 4);
        if (kind == 0) {
            const uint32_t n = 1 + rng() % 20;
            std::vector<kvp_loc> m(n);
            const int rc = kv_pool_place(pool, next, n, m.data());
            if (rc == KVP_OK) {
                live.maps[next] = m;
            } else {
                CHECK(rc == KVP_ERR_NOSPACE);
                CHECK(std::strstr(kv_pool_last_error(), "no free range") != nullptr);
                refusals->fetch_add(1);
            }
            ++next;
            continue;
        }
        auto it = live.maps.begin();
        std::advance(it, rng() % live.maps.size());
        if (kind == 1) {
            const uint32_t n = 1 + rng() % 10;
            std::vector<kvp_loc> m(n);
            const int rc = kv_pool_extend(pool, it->first, n, m.data());
            if (rc == KVP_OK) {
                for (const kvp_loc &e : m) CHECK(e.gen == it->second[0].gen);
                it->second.insert(it->second.end(), m.begin(), m.end());
            } else {
                CHECK(rc == KVP_ERR_NOSPACE);
                refusals->fetch_add(1);
            }
        } else if (kind == 2) {
            CHECK(kv_pool_release(pool, it->first) == KVP_OK);
            CHECK(kv_pool_last_error()[0] == '\0');
            std::vector<kvp_loc> one(1);
            CHECK(kv_pool_lookup(pool, it->first, 1, one.data()) == KVP_ERR_NOTFOUND);
            CHECK(std::strstr(kv_pool_last_error(), "not placed") != nullptr);
            live.maps.erase(it);
        } else {
            std::vector<kvp_loc> got(it->second.size());
            CHECK(kv_pool_lookup(pool, it->first, static_cast<uint32_t>(got.size()), got.data()) == KVP_OK);
            for (size_t j = 0; j < got.size(); ++j)
                CHECK(got[j].region == it->second[j].region && got[j].gen == it->second[j].gen &&
                      got[j].offset == it->second[j].offset);
        }
    }
}

void reader(kvp_pool *pool, const std::atomic<bool> *stop)
{
    const uint64_t w[kRegions] = {4, 4, 1, 1};
    uint64_t c[kRegions];
    while (!stop->load()) {
        CHECK(kv_pool_set_bandwidths(pool, w) == KVP_OK);   // the same weights: maps stay as they are
        for (uint32_t i = 0; i < kRegions; ++i) {
            kvp_region_info info;
            CHECK(kv_pool_region_info(pool, i, &info) == KVP_OK);
            CHECK(info.bandwidth == w[i]);
        }
        CHECK(kv_pool_counts(w, kRegions, 8192, c) == KVP_OK);
        CHECK(c[0] == 3277 && c[1] == 3277 && c[2] == 819 && c[3] == 819);
    }
}

}  // namespace

int main()
{
    const uint64_t w[kRegions] = {4, 4, 1, 1};
    kvp_region_desc regions[kRegions];
    for (uint32_t i = 0; i < kRegions; ++i)
        regions[i] = kvp_region_desc{KVP_REGION_HOST, -1, w[i] * kCapBlocks * kBlockBytes, 0, 0};
    kvp_kv_spec spec = {2, 1, 8, 16, 2, 0};
    kvp_pool *pool = nullptr;
    CHECK(kv_pool_create(regions, w, kRegions, &spec, -1, &pool) == KVP_OK);

    std::vector<Live> live(kWorkers);
    std::atomic<uint64_t> refusals{0};
    std::atomic<bool> stop{false};
    std::vector<std::thread> threads;
    for (int t = 0; t < 2; ++t) threads.emplace_back(reader, pool, &stop);
    std::vector<std::thread> workers;
    for (int t = 0; t < kWorkers; ++t) workers.emplace_back(worker, pool, t, &live[t], &refusals);
    for (auto &t : workers) t.join();
    stop.store(true);
    for (auto &t : threads) t.join();

    std::set<std::pair<uint32_t, uint64_t>> used;
    size_t blocks = 0;
    for (const Live &l : live)
        for (const auto &kv : l.maps)
            for (const kvp_loc &e : kv.second) {
                CHECK(used.insert({e.region, e.offset}).second);   // no two live blocks share a place
                ++blocks;
            }
    for (const Live &l : live)
        for (const auto &kv : l.maps) CHECK(kv_pool_release(pool, kv.first) == KVP_OK);
    // everything free again: one request filling every region exactly
    uint64_t total = 0;
    for (uint32_t i = 0; i < kRegions; ++i) total += w[i] * kCapBlocks;
    std::vector<kvp_loc> all(total);
    CHECK(kv_pool_place(pool, 1ull << 62, static_cast<uint32_t>(total), all.data()) == KVP_OK);
    kv_pool_destroy(pool);
    std::printf("%zu live blocks at the join, %llu refusals\n", blocks, (unsigned long long)refusals.load());
    CHECK(blocks > 100 && refusals.load() > 10);
    std::printf("all checks passed\n");
    return 0;
}

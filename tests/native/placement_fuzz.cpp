// Placement-only pools (no GPU) through the C ABI of the host-sanitized
// library: random place / extend / release / lookup sequences, checked against
// a model of the live blocks.  Any memory or undefined-behaviour error in the
// placement bookkeeping (ranges per offload set, the regions' live maps, the
// GLT) stops the run under AddressSanitizer / UndefinedBehaviorSanitizer.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <random>
#include <set>
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

int main()
{
    std::mt19937_64 rng(2026);
    uint64_t placed = 0, extended = 0, refused = 0, released = 0;
    for (int round = 0; round < 60; ++round) {
        const uint32_t N = 1 + rng() % 6, L = 1u << (rng() % 4);
        kvp_kv_spec spec = {L, 1, 8, 16, 2, 0};              // chunk 256 B, block 512 * L B
        const uint64_t bb = 2ull * L * 256;
        std::vector<uint64_t> w(N), cap(N);
        std::vector<kvp_region_desc> regions(N);
        for (uint32_t i = 0; i < N; ++i) {
            w[i] = 1 + rng() % 9;
            cap[i] = (w[i] * 30 + 7) * bb + (rng() % 3) * 4096 + 4096;
            regions[i] = kvp_region_desc{i % 2 ? KVP_REGION_STAGING : KVP_REGION_HOST, -1, cap[i], 0, 0};
        }
        kvp_pool *pool = nullptr;
        CHECK(kv_pool_create(regions.data(), w.data(), N, &spec, -1, &pool) == KVP_OK);
        std::map<uint64_t, std::vector<kvp_loc>> live;
        std::set<std::pair<uint32_t, uint64_t>> used;   // (region, offset) of every live block
        uint64_t next_req = 1;
        auto add = [&](const std::vector<kvp_loc> &m, uint32_t gen) {
            for (const kvp_loc &e : m) {
                CHECK(e.region < N && e.gen == gen && e.offset % 16 == 0 && e.offset + bb <= cap[e.region]);
                CHECK(used.insert({e.region, e.offset}).second);   // no block shares a place
            }
        };
        for (int op = 0; op < 200; ++op) {
            const int kind = static_cast<int>(rng() % 4);
            if (kind == 0 || live.empty()) {
                const uint32_t n = 1 + rng() % 60;
                std::vector<kvp_loc> m(n);
                const int rc = kv_pool_place(pool, next_req, n, m.data());
                if (rc == KVP_OK) {
                    add(m, m[0].gen);
                    live[next_req] = m;
                    ++placed;
                } else {
                    CHECK(rc == KVP_ERR_NOSPACE);
                    ++refused;
                }
                ++next_req;
            } else {
                auto it = live.begin();
                std::advance(it, rng() % live.size());
                const uint64_t r = it->first;
                std::vector<kvp_loc> &have = it->second;
                if (kind == 1) {                                     // the next offload set
                    const uint32_t n = 1 + rng() % 40;
                    std::vector<kvp_loc> m(n);
                    const int rc = kv_pool_extend(pool, r, n, m.data());
                    if (rc == KVP_OK) {
                        add(m, have[0].gen);
                        have.insert(have.end(), m.begin(), m.end());
                        ++extended;
                    } else {
                        CHECK(rc == KVP_ERR_NOSPACE);
                        ++refused;
                    }
                } else if (kind == 2) {
                    CHECK(kv_pool_release(pool, r) == KVP_OK);
                    for (const kvp_loc &e : have) used.erase({e.region, e.offset});
                    live.erase(it);
                    ++released;
                    continue;
                }
                std::vector<kvp_loc> got(have.size());
                CHECK(kv_pool_lookup(pool, r, static_cast<uint32_t>(have.size()), got.data()) == KVP_OK);
                for (size_t j = 0; j < have.size(); ++j)
                    CHECK(got[j].region == have[j].region && got[j].gen == have[j].gen &&
                          got[j].offset == have[j].offset);
                CHECK(kv_pool_lookup(pool, r, static_cast<uint32_t>(have.size()) + 1, got.data()) ==
                      KVP_ERR_INVALID);
            }
        }
        std::vector<kvp_loc> one(1);
        CHECK(kv_pool_extend(pool, next_req + 1000, 1, one.data()) == KVP_ERR_NOTFOUND);
        if (!live.empty()) CHECK(kv_pool_extend(pool, live.begin()->first, 0, one.data()) == KVP_ERR_INVALID);
        kv_pool_destroy(pool);
    }
    std::printf("placed %llu, extended %llu, refused %llu, released %llu\n", (unsigned long long)placed,
                (unsigned long long)extended, (unsigned long long)refused, (unsigned long long)released);
    CHECK(placed > 100 && extended > 100 && refused > 10 && released > 50);
    std::printf("all checks passed\n");
    return 0;
}

// Host allocation failures inside place and extend, through the C ABI of the
// host-sanitized library on placement-only pools (no GPU).
//
// Creating a pool and computing Eq. 2 counts are tried the same way first
// (a failed create returns no pool and leaks nothing; a failed count writes
// nothing).  Then two pools go through the same random sequence of place /
// extend / release calls.  On pool A every call is first tried with the k-th host allocation
// made inside it failing (k = 0, 1, 2, ... until the call makes fewer than k
// allocations); each such try must return KVP_ERR_NOMEM (or the call's own
// error code, with a fixed message, when the failure hits the copy of its
// message) and leave the pool exactly as it was.  Pool B never fails.  "Exactly as it
// was" is checked two ways: the lookups of every live request are unchanged
// after each failed try, and the call that finally runs on A returns the same
// code and the same map as on B -- which a leaked or half-taken range, or a
// stale GLT entry, would change then or at a later call.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <new>
#include <random>
#include <vector>

#include "kvpool.h"

#define CHECK(c)                                                                      \
    do {                                                                              \
        if (!(c)) {                                                                   \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);      \
            std::exit(1);                                                             \
        }                                                                             \
    } while (0)

// One-shot failure of the k-th throwing operator new after arming (the library's host
// allocations resolve to these definitions).  Single-threaded driver.
static long g_countdown = -1;

void *operator new(std::size_t n)
{
    if (g_countdown >= 0 && g_countdown-- == 0) throw std::bad_alloc();
    void *p = std::malloc(n ? n : 1);
    if (!p) throw std::bad_alloc();
    return p;
}
void *operator new[](std::size_t n) { return operator new(n); }
// The non-throwing forms (e.g. the scratch buffer of std::stable_sort, which
// copes with a null return) are left out of the injection.
void *operator new(std::size_t n, const std::nothrow_t &) noexcept { return std::malloc(n ? n : 1); }
void *operator new[](std::size_t n, const std::nothrow_t &) noexcept { return std::malloc(n ? n : 1); }
void operator delete(void *p) noexcept { std::free(p); }
void operator delete[](void *p) noexcept { std::free(p); }
void operator delete(void *p, std::size_t) noexcept { std::free(p); }
void operator delete[](void *p, std::size_t) noexcept { std::free(p); }

static bool same(const std::vector<kvp_loc> &a, const std::vector<kvp_loc> &b)
{
    if (a.size() != b.size()) return false;
    for (size_t j = 0; j < a.size(); ++j)
        if (a[j].region != b[j].region || a[j].gen != b[j].gen || a[j].offset != b[j].offset) return false;
    return true;
}

static std::vector<kvp_loc> lookup(kvp_pool *p, uint64_t r, size_t n)
{
    std::vector<kvp_loc> m(n);
    CHECK(kv_pool_lookup(p, r, static_cast<uint32_t>(n), m.data()) == KVP_OK);
    return m;
}

int main()
{
    std::mt19937_64 rng(4242);
    uint64_t injected = 0, ops = 0;
    for (int round = 0; round < 12; ++round) {
        const uint32_t N = 1 + rng() % 6, L = 1u << (rng() % 3);
        kvp_kv_spec spec = {L, 1, 8, 16, 2, 0};                // block 512 * L bytes
        const uint64_t bb = 2ull * L * 256;
        std::vector<uint64_t> w(N);
        std::vector<kvp_region_desc> regions(N);
        for (uint32_t i = 0; i < N; ++i) {
            w[i] = 1 + rng() % 9;
            regions[i] = kvp_region_desc{KVP_REGION_HOST, -1, (w[i] * 20 + 5) * bb + 4096, 0, 0};
        }
        kvp_pool *A = nullptr, *B = nullptr;
        for (long k = 0;; ++k) {                            // create: nothing leaks, no pool comes back
            g_countdown = k;
            const int rc = kv_pool_create(regions.data(), w.data(), N, &spec, -1, &A);
            const bool failed_here = g_countdown < 0;
            g_countdown = -1;
            if (!failed_here) {
                CHECK(rc == KVP_OK && A);
                break;
            }
            CHECK(rc == KVP_ERR_NOMEM && A == nullptr);
            ++injected;
            CHECK(k < 100000);
        }
        std::vector<uint64_t> c(N, 7), c_ok(N);               // Eq. 2 counts: all written or none
        CHECK(kv_pool_counts(w.data(), N, 1000, c_ok.data()) == KVP_OK);
        for (long k = 0;; ++k) {
            g_countdown = k;
            const int rc = kv_pool_counts(w.data(), N, 1000, c.data());
            const bool failed_here = g_countdown < 0;
            g_countdown = -1;
            if (!failed_here) {
                CHECK(rc == KVP_OK && c == c_ok);
                break;
            }
            CHECK(rc == KVP_ERR_NOMEM);
            for (uint64_t x : c) CHECK(x == 7);
            ++injected;
        }
        CHECK(kv_pool_create(regions.data(), w.data(), N, &spec, -1, &B) == KVP_OK);
        std::map<uint64_t, std::vector<kvp_loc>> live;      // request -> its map on both pools
        uint64_t next_req = 1;
        auto all_unchanged = [&] {
            for (const auto &kv : live) CHECK(same(lookup(A, kv.first, kv.second.size()), kv.second));
        };
        for (int op = 0; op < 60; ++op) {
            const int kind = live.empty() ? 0 : static_cast<int>(rng() % 3);
            if (kind == 2) {
                auto it = live.begin();
                std::advance(it, rng() % live.size());
                for (long k = 0;; ++k) {
                    g_countdown = k;
                    const int rc = kv_pool_release(A, it->first);
                    const bool failed_here = g_countdown < 0;
                    g_countdown = -1;
                    if (!failed_here) {
                        CHECK(rc == KVP_OK);
                        break;
                    }
                    CHECK(rc == KVP_ERR_NOMEM);
                    ++injected;
                    all_unchanged();                              // the request is still whole
                    CHECK(k < 100000);
                }
                CHECK(kv_pool_release(B, it->first) == KVP_OK);
                live.erase(it);
                ++ops;
                continue;
            }
            const bool place = kind == 0;
            uint64_t r = next_req;
            if (!place) {
                auto it = live.begin();
                std::advance(it, rng() % live.size());
                r = it->first;
            }
            const uint32_t n = 1 + rng() % 30;
            std::vector<kvp_loc> ma(n), mb(n);
            int rc = KVP_OK;
            for (long k = 0;; ++k) {
                g_countdown = k;
                rc = place ? kv_pool_place(A, r, n, ma.data()) : kv_pool_extend(A, r, n, ma.data());
                const bool failed_here = g_countdown < 0;     // the armed allocation was reached
                g_countdown = -1;
                if (!failed_here) break;
                // NOMEM, or the call's own NOSPACE when the failure hit the copy of its message
                CHECK(rc == KVP_ERR_NOMEM ||
                      (rc == KVP_ERR_NOSPACE && std::strncmp(kv_pool_last_error(), "out of host memory", 18) == 0));
                ++injected;
                all_unchanged();
                if (place) {
                    std::vector<kvp_loc> one(1);
                    CHECK(kv_pool_lookup(A, r, 1, one.data()) == KVP_ERR_NOTFOUND);
                }
                CHECK(k < 100000);
            }
            const int rb = place ? kv_pool_place(B, r, n, mb.data()) : kv_pool_extend(B, r, n, mb.data());
            CHECK(rc == rb);
            ++ops;
            if (rc == KVP_OK) {
                CHECK(same(ma, mb));
                if (place) {
                    live[r] = ma;
                    ++next_req;
                } else {
                    live[r].insert(live[r].end(), ma.begin(), ma.end());
                }
            } else {
                CHECK(rc == KVP_ERR_NOSPACE);
                if (place) ++next_req;
            }
            all_unchanged();
        }
        kv_pool_destroy(A);
        kv_pool_destroy(B);
    }
    std::printf("%llu calls, %llu injected failures\n", (unsigned long long)ops, (unsigned long long)injected);
    CHECK(ops > 300 && injected > 3000);
    std::printf("all checks passed\n");
    return 0;
}

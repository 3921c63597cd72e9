/* The oracle under AddressSanitizer / UndefinedBehaviorSanitizer (CPU only):
 * random place / extend / release sequences on small pools, each placed set
 * stored from and gathered back into exactly-sized buffers (both chunk
 * layouts), with a round-trip check.  Prototypes are restated here: the
 * oracle has no header, and this driver is test code. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    uint32_t region;
    uint32_t gen;
    uint64_t offset;
} oracle_loc;
typedef struct opool opool;

int oracle_counts(const uint64_t *bandwidth, uint32_t n_dev, uint64_t n_kv, uint64_t *count);
opool *oracle_pool_new(uint32_t n_dev, const uint64_t *bandwidth, const uint64_t *capacity, uint64_t block_bytes);
void oracle_pool_free(opool *p);
int oracle_place(opool *p, uint64_t request, uint32_t n_blocks, oracle_loc *out);
int oracle_extend(opool *p, uint64_t request, uint32_t n_new, oracle_loc *out);
int oracle_lookup(const opool *p, uint64_t request, uint32_t n_blocks, oracle_loc *out);
int oracle_release(opool *p, uint64_t request);
void oracle_store(uint32_t n_blocks, const oracle_loc *map, const int32_t *src_slot, uint8_t *const *region_mem,
                  const uint8_t *const *k_layers, const uint8_t *const *v_layers, uint32_t L, uint32_t H,
                  uint32_t bs, uint32_t D, uint32_t elem_bytes, uint32_t layout);
void oracle_gather(uint32_t n_blocks, const oracle_loc *map, const int32_t *dst_slot, const uint8_t *const *region_mem,
                   uint8_t *const *k_layers, uint8_t *const *v_layers, uint32_t L, uint32_t H, uint32_t bs,
                   uint32_t D, uint32_t elem_bytes, uint32_t layout);

#define CHECK(c)                                                                \
    do {                                                                        \
        if (!(c)) {                                                             \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);     \
            exit(1);                                                            \
        }                                                                       \
    } while (0)

static uint64_t state = 88172645463325252ull;
static uint64_t rnd(void)
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return state;
}

int main(void)
{
    unsigned checks = 0;
    for (int round = 0; round < 40; ++round) {
        const uint32_t N = 1 + rnd() % 5, L = 1 + rnd() % 3, H = 1 + rnd() % 3, bs = 1 + rnd() % 4, D = 8 * (1 + rnd() % 3);
        const uint32_t layout = rnd() % 2, elem = 2;
        const uint64_t C = (uint64_t)H * bs * D * elem, bb = 2ull * L * C;
        uint64_t w[5], cap[5];
        uint8_t *mem[5];
        for (uint32_t i = 0; i < N; ++i) {
            w[i] = 1 + rnd() % 9;
            cap[i] = ((w[i] * 40 + 9) * bb + 4095) / 4096 * 4096;
            mem[i] = (uint8_t *)malloc(cap[i]);
            CHECK(mem[i]);
        }
        opool *p = oracle_pool_new(N, w, cap, bb);
        CHECK(p);
        for (int op = 0; op < 60; ++op) {
            const uint64_t req = 1 + rnd() % 6;
            const uint32_t n = 1 + rnd() % 30;
            oracle_loc *m = (oracle_loc *)malloc(n * sizeof(oracle_loc));
            int placed_set = 0;   /* m holds a set placed by this op */
            if (rnd() % 3 == 0) {
                (void)oracle_release(p, req);
            } else {
                int rc = oracle_extend(p, req, n, m);
                if (rc == -4) rc = oracle_place(p, req, n, m);
                CHECK(rc == 0 || rc == -3);
                placed_set = rc == 0;
            }
            if (placed_set && op % 2 == 0) {
                /* exactly-sized source and destination: n slots per layer and K/V */
                uint8_t **src = (uint8_t **)malloc(2 * L * sizeof(uint8_t *));
                uint8_t **dst = (uint8_t **)malloc(2 * L * sizeof(uint8_t *));
                int32_t *slots = (int32_t *)malloc(n * sizeof(int32_t));
                for (uint32_t b = 0; b < n; ++b) slots[b] = (int32_t)(n - 1 - b);
                for (uint32_t k = 0; k < 2 * L; ++k) {
                    src[k] = (uint8_t *)malloc(n * C);
                    dst[k] = (uint8_t *)calloc(n, C);
                    for (uint64_t e = 0; e < n * C; ++e) src[k][e] = (uint8_t)(rnd() >> 11);
                }
                {
                    for (uint32_t b = 0; b < n; ++b) CHECK(m[b].region < N && m[b].offset + bb <= cap[m[b].region]);
                    oracle_store(n, m, slots, mem, (const uint8_t *const *)src, (const uint8_t *const *)(src + L),
                                 L, H, bs, D, elem, layout);
                    oracle_gather(n, m, slots, (const uint8_t *const *)mem, dst, dst + L, L, H, bs, D, elem, layout);
                    for (uint32_t k = 0; k < 2 * L; ++k) CHECK(memcmp(src[k], dst[k], n * C) == 0);
                    ++checks;
                }
                for (uint32_t k = 0; k < 2 * L; ++k) {
                    free(src[k]);
                    free(dst[k]);
                }
                free(src);
                free(dst);
                free(slots);
            }
            free(m);
        }
        oracle_pool_free(p);
        for (uint32_t i = 0; i < N; ++i) free(mem[i]);
    }
    printf("%u round trips\n", checks);
    CHECK(checks > 100);
    printf("all checks passed\n");
    return 0;
}

/*
 * kvgen.c -- seeded synthetic KV-cache values, shared by the tests, the bench
 * and the oracle side of every parity check.
 *
 * This file holds no part of the KV-pool method (no placement, no store, no
 * gather).  It only defines the *input*: the bf16 contents of every logical
 * KV element of a request, as a pure function of
 *     (seed, request, block, layer, kv, head, token, dim).
 * Any block can therefore be regenerated on its own, which is what lets a
 * full-size run be checked on sampled blocks.
 *
 * Definition (counter based, no generator state):
 *   key(seed, q, b)   = sm64(sm64(sm64(seed) ^ q) ^ b)
 *   element index e   = ((((l*2 + kv)*H + h)*bs + t)*D + d)
 *   pair m = e / 2,   r = sm64(key ^ m)
 *   u1 = ((r >> 40) + 1) / 2^24        in (0, 1]
 *   u2 = ((r >> 16) & 0xFFFFFF) / 2^24 in [0, 1)
 *   Box-Muller (Box & Muller, 1958), in float:
 *     rad = sqrtf(-2 logf(u1));  z0 = rad cosf(2 pi u2);  z1 = rad sinf(2 pi u2)
 *   element 2m takes z0, element 2m+1 takes z1, each rounded to bf16 with
 *   round-to-nearest-even.
 * sm64 is the splitmix64 output function (Steele, Lea & Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014).
 *
 * The values are generated once on the host; both the GPU path and the oracle
 * read those same bytes, so no bit of the comparison depends on a GPU libm.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t sm64(uint64_t x)
{
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

static inline uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) /* NaN: keep quiet */
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7FFFu + lsb;
    return (uint16_t)(u >> 16);
}

uint64_t kvgen_block_key(uint64_t seed, uint64_t request, uint64_t block)
{
    return sm64(sm64(sm64(seed) ^ request) ^ block);
}

/* Two N(0,1) bf16 values for pair m of a block key. */
static inline void pair_values(uint64_t key, uint64_t m, uint16_t *v0, uint16_t *v1)
{
    uint64_t r = sm64(key ^ m);
    float u1 = (float)((r >> 40) + 1) * (1.0f / 16777216.0f);
    float u2 = (float)((r >> 16) & 0xFFFFFFull) * (1.0f / 16777216.0f);
    float rad = sqrtf(-2.0f * logf(u1));
    float ang = 6.28318530717958647692f * u2;
    *v0 = f32_to_bf16_rne(rad * cosf(ang));
    *v1 = f32_to_bf16_rne(rad * sinf(ang));
}

/*
 * Fill elements [e0, e0 + count) of block (seed, request, block) into out[0..count).
 * Elements are bf16 (uint16).  e0 may be odd.
 */
void kvgen_fill_elems(uint64_t seed, uint64_t request, uint64_t block,
                      uint64_t e0, uint64_t count, uint16_t *out)
{
    uint64_t key = kvgen_block_key(seed, request, block);
    uint64_t e = e0, end = e0 + count;
    uint16_t a, b;
    if (e < end && (e & 1)) {
        pair_values(key, e >> 1, &a, &b);
        *out++ = b;
        e++;
    }
    for (; e + 1 < end; e += 2) {
        pair_values(key, e >> 1, &a, &b);
        out[0] = a;
        out[1] = b;
        out += 2;
    }
    if (e < end) {
        pair_values(key, e >> 1, &a, &b);
        *out = a;
    }
}

/*
 * Fill the engine-layout source cache for n_blocks logical blocks of one
 * request.  Layout per layer and per K/V: [num_slots][H][bs][D] of
 * elem_bytes == 2 elements; block b goes to slot slot_of_block[b].
 * k_layers[l] / v_layers[l] are host pointers.  Work is split over n_threads
 * POSIX threads by block.
 */
typedef struct {
    uint64_t seed, request;
    uint32_t L, H, bs, D;
    const int32_t *slot_of_block;
    uint16_t *const *k_layers;
    uint16_t *const *v_layers;
    const uint64_t *block_ids;   /* logical block index used in the key (NULL = b) */
    uint32_t b_begin, b_end;
} fill_job;

static void *fill_worker(void *arg)
{
    const fill_job *j = (const fill_job *)arg;
    const uint64_t chunk = (uint64_t)j->H * j->bs * j->D;
    for (uint32_t b = j->b_begin; b < j->b_end; ++b) {
        uint64_t blk = j->block_ids ? j->block_ids[b] : b;
        uint64_t slot = (uint64_t)j->slot_of_block[b];
        for (uint32_t l = 0; l < j->L; ++l) {
            kvgen_fill_elems(j->seed, j->request, blk, (uint64_t)(2 * l) * chunk, chunk,
                             j->k_layers[l] + slot * chunk);
            kvgen_fill_elems(j->seed, j->request, blk, (uint64_t)(2 * l + 1) * chunk, chunk,
                             j->v_layers[l] + slot * chunk);
        }
    }
    return 0;
}

int kvgen_fill_cache(uint64_t seed, uint64_t request, uint32_t n_blocks,
                     const uint64_t *block_ids, const int32_t *slot_of_block,
                     uint32_t L, uint32_t H, uint32_t bs, uint32_t D,
                     uint16_t *const *k_layers, uint16_t *const *v_layers,
                     uint32_t n_threads)
{
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    if (n_threads > n_blocks) n_threads = n_blocks ? n_blocks : 1;
    pthread_t tid[256];
    fill_job jobs[256];
    uint32_t per = n_blocks / n_threads, extra = n_blocks % n_threads, at = 0;
    for (uint32_t i = 0; i < n_threads; ++i) {
        uint32_t take = per + (i < extra ? 1u : 0u);
        fill_job j = {seed, request, L, H, bs, D, slot_of_block, k_layers, v_layers,
                      block_ids, at, at + take};
        jobs[i] = j;
        at += take;
    }
    uint32_t started = 0;
    for (uint32_t i = 1; i < n_threads; ++i) {
        if (pthread_create(&tid[i], 0, fill_worker, &jobs[i]) != 0) break;
        started = i;
    }
    fill_worker(&jobs[0]);
    for (uint32_t i = 1; i <= started; ++i) pthread_join(tid[i], 0);
    /* any thread that failed to start: run its share here */
    for (uint32_t i = started + 1; i < n_threads; ++i) fill_worker(&jobs[i]);
    return 0;
}

/* Fill a host buffer with a repeated 16-bit pattern using n_threads threads. */
typedef struct { uint16_t *p; uint64_t n; uint16_t v; } pat_job;
static void *pat_worker(void *arg)
{
    pat_job *j = (pat_job *)arg;
    for (uint64_t i = 0; i < j->n; ++i) j->p[i] = j->v;
    return 0;
}

void kvgen_fill_u16(uint16_t *p, uint64_t n, uint16_t v, uint32_t n_threads)
{
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t tid[256];
    pat_job jobs[256];
    uint64_t per = n / n_threads;
    for (uint32_t i = 0; i < n_threads; ++i) {
        jobs[i].p = p + per * i;
        jobs[i].n = (i == n_threads - 1) ? n - per * i : per;
        jobs[i].v = v;
    }
    uint32_t started = 0;
    for (uint32_t i = 1; i < n_threads; ++i) {
        if (pthread_create(&tid[i], 0, pat_worker, &jobs[i]) != 0) break;
        started = i;
    }
    pat_worker(&jobs[0]);
    for (uint32_t i = 1; i <= started; ++i) pthread_join(tid[i], 0);
    for (uint32_t i = started + 1; i < n_threads; ++i) pat_worker(&jobs[i]);
}

uint64_t kvgen_sm64(uint64_t x) { return sm64(x); }

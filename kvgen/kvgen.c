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
 *   r = sm64(key ^ (e / 4)),  u = bits [16*(e%4), 16*(e%4)+16) of r
 *   value = Q[u],  Q[i] = bf16_rne( Phi^-1( (i + 0.5) / 65536 ) )
 * i.e. a standard normal sampled by inversion on a 16-bit uniform grid (the
 * tails beyond about 4.3 sigma are cut, which is invisible at bf16
 * resolution for this purpose).  Phi^-1 is Wichura's algorithm AS 241
 * (PPND16, Applied Statistics 37, 1988), accurate to about 1e-16 in double.
 * sm64 is the splitmix64 output function (Steele, Lea & Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014).
 *
 * The values are generated on the host; both the GPU path and the oracle read
 * those same bytes.
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

static uint16_t f64_to_bf16_rne(double v)
{
    /* Nearest bf16 to a double (ties to even), without double rounding:
     * the two bf16 neighbours of the nearest float bracket v, and the
     * distances to them are compared exactly in double. */
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, 4);
    uint32_t lo = u & 0xFFFF0000u, hi = lo + 0x10000u;
    float flo, fhi;
    memcpy(&flo, &lo, 4);
    memcpy(&fhi, &hi, 4);
    double dlo = fabs(v - (double)flo), dhi = fabs((double)fhi - v);
    if (dlo < dhi) return (uint16_t)(lo >> 16);
    if (dhi < dlo) return (uint16_t)(hi >> 16);
    return (uint16_t)(((lo >> 16) & 1u) ? (hi >> 16) : (lo >> 16)); /* tie: even */
}

/* Wichura AS 241 PPND16: the p-quantile of the standard normal. */
double kvgen_ppnd16(double p)
{
    const double q = p - 0.5;
    if (fabs(q) <= 0.425) {
        const double r = 0.180625 - q * q;
        return q * (((((((2509.0809287301226727 * r + 33430.575583588128105) * r + 67265.770927008700853) * r +
                        45921.953931549871457) * r + 13731.693765509461125) * r + 1971.5909503065514427) * r +
                     133.14166789178437745) * r + 3.387132872796366608) /
               (((((((5226.495278852545925 * r + 28729.085735721942674) * r + 39307.89580009271061) * r +
                    21213.794301586595867) * r + 5394.1960214247511077) * r + 687.1870074920579083) * r +
                 42.313330701600911252) * r + 1.0);
    }
    double r = q < 0 ? p : 1.0 - p;
    r = sqrt(-log(r));
    double val;
    if (r <= 5.0) {
        r -= 1.6;
        val = (((((((7.7454501427834140764e-4 * r + 0.0227238449892691845833) * r + 0.24178072517745061177) * r +
                   1.27045825245236838258) * r + 3.64784832476320460504) * r + 5.7694972214606914055) * r +
                4.6303378461565452959) * r + 1.42343711074968357734) /
              (((((((1.05075007164441684324e-9 * r + 5.475938084995344946e-4) * r + 0.0151986665636164571966) * r +
                   0.14810397642748007459) * r + 0.68976733498510000455) * r + 1.6763848301838038494) * r +
                2.05319162663775882187) * r + 1.0);
    } else {
        r -= 5.0;
        val = (((((((2.01033439929228813265e-7 * r + 2.71155556874348757815e-5) * r + 0.0012426609473880784386) * r +
                   0.026532189526576123093) * r + 0.29656057182850489123) * r + 1.7848265399172913358) * r +
                5.4637849111641143699) * r + 6.6579046435011037772) /
              (((((((2.04426310338993978564e-15 * r + 1.4215117583164458887e-7) * r + 1.8463183175100546818e-5) * r +
                   7.868691311456132591e-4) * r + 0.0148753612908506148525) * r + 0.13692988092273580531) * r +
                0.59983220655588793769) * r + 1.0);
    }
    return q < 0 ? -val : val;
}

static uint16_t g_table[65536];
static pthread_once_t g_once = PTHREAD_ONCE_INIT;

static void build_table(void)
{
    for (int i = 0; i < 65536; ++i) g_table[i] = f64_to_bf16_rne(kvgen_ppnd16((i + 0.5) / 65536.0));
}

void kvgen_normal_table(uint16_t *out)
{
    pthread_once(&g_once, build_table);
    memcpy(out, g_table, sizeof(g_table));
}

uint64_t kvgen_block_key(uint64_t seed, uint64_t request, uint64_t block)
{
    return sm64(sm64(sm64(seed) ^ request) ^ block);
}

/* Elements [e0, e0 + count) of block (seed, request, block) into out. */
void kvgen_fill_elems(uint64_t seed, uint64_t request, uint64_t block, uint64_t e0, uint64_t count,
                      uint16_t *out)
{
    pthread_once(&g_once, build_table);
    const uint64_t key = kvgen_block_key(seed, request, block);
    uint64_t e = e0;
    const uint64_t end = e0 + count;
    while (e < end && (e & 3)) {
        const uint64_t r = sm64(key ^ (e >> 2));
        *out++ = g_table[(r >> (16 * (e & 3))) & 0xFFFF];
        ++e;
    }
    for (; e + 4 <= end; e += 4) {
        const uint64_t r = sm64(key ^ (e >> 2));
        out[0] = g_table[r & 0xFFFF];
        out[1] = g_table[(r >> 16) & 0xFFFF];
        out[2] = g_table[(r >> 32) & 0xFFFF];
        out[3] = g_table[r >> 48];
        out += 4;
    }
    for (; e < end; ++e) {
        const uint64_t r = sm64(key ^ (e >> 2));
        *out++ = g_table[(r >> (16 * (e & 3))) & 0xFFFF];
    }
}

/*
 * Fill the engine-layout source cache for n_blocks blocks of one request.
 * Layout per layer and per K/V: [num_slots][H][bs][D] of 2-byte elements;
 * block block_ids[b] (logical block index) goes to slot slot_of_block[b].
 * k_layers[l] / v_layers[l] are host pointers.  Work is split over
 * n_threads POSIX threads by block.
 */
typedef struct {
    uint64_t seed, request;
    uint32_t L, H, bs, D;
    const uint64_t *block_ids;
    const int32_t *slot_of_block;
    uint16_t *const *k_layers;
    uint16_t *const *v_layers;
    uint32_t b_begin, b_end;
} fill_job;

static void *fill_worker(void *arg)
{
    const fill_job *j = (const fill_job *)arg;
    const uint64_t chunk = (uint64_t)j->H * j->bs * j->D;
    for (uint32_t b = j->b_begin; b < j->b_end; ++b) {
        const uint64_t blk = j->block_ids[b];
        const uint64_t slot = (uint64_t)j->slot_of_block[b];
        for (uint32_t l = 0; l < j->L; ++l) {
            kvgen_fill_elems(j->seed, j->request, blk, (uint64_t)(2 * l) * chunk, chunk,
                             j->k_layers[l] + slot * chunk);
            kvgen_fill_elems(j->seed, j->request, blk, (uint64_t)(2 * l + 1) * chunk, chunk,
                             j->v_layers[l] + slot * chunk);
        }
    }
    return 0;
}

int kvgen_fill_cache(uint64_t seed, uint64_t request, uint32_t n_blocks, const uint64_t *block_ids,
                     const int32_t *slot_of_block, uint32_t L, uint32_t H, uint32_t bs, uint32_t D,
                     uint16_t *const *k_layers, uint16_t *const *v_layers, uint32_t n_threads)
{
    pthread_once(&g_once, build_table);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    if (n_blocks && n_threads > n_blocks) n_threads = n_blocks;
    pthread_t tid[256];
    fill_job jobs[256];
    uint32_t per = n_blocks / n_threads, extra = n_blocks % n_threads, at = 0;
    for (uint32_t i = 0; i < n_threads; ++i) {
        uint32_t take = per + (i < extra ? 1u : 0u);
        fill_job j = {seed, request, L, H, bs, D, block_ids, slot_of_block, k_layers, v_layers, at, at + take};
        jobs[i] = j;
        at += take;
    }
    char started[256] = {0};
    for (uint32_t i = 1; i < n_threads; ++i) started[i] = pthread_create(&tid[i], 0, fill_worker, &jobs[i]) == 0;
    fill_worker(&jobs[0]);
    for (uint32_t i = 1; i < n_threads; ++i) {
        if (started[i])
            pthread_join(tid[i], 0);
        else
            fill_worker(&jobs[i]);
    }
    return 0;
}

/* Fill a host buffer with a repeated 16-bit pattern using n_threads threads. */
typedef struct {
    uint16_t *p;
    uint64_t n;
    uint16_t v;
} pat_job;

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
    char started[256] = {0};
    for (uint32_t i = 1; i < n_threads; ++i) started[i] = pthread_create(&tid[i], 0, pat_worker, &jobs[i]) == 0;
    pat_worker(&jobs[0]);
    for (uint32_t i = 1; i < n_threads; ++i) {
        if (started[i])
            pthread_join(tid[i], 0);
        else
            pat_worker(&jobs[i]);
    }
}

uint64_t kvgen_sm64(uint64_t x) { return sm64(x); }

/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU statement of what the KV-pool
 * retrieval path computes, written from the paper (Unified KV Pooling,
 * Sec. 4.1-4.3).  Only the test suite, the smoke check and the bench's CPU
 * baseline call it.  It shares no source, header or helper with the GPU
 * library; the two meet only through the seeded inputs and the comparison
 * in the tests.
 *
 * Contents
 *   oracle_counts    Eq. (1) placement ratio and Eq. (2) target counts,
 *                    remainder per Algorithm 1 (counting part).
 *   oracle_pool_*    pool bookkeeping: per-request placement map
 *   oracle_place     Algorithm 1 (partition part) + one contiguous range
 *                    per (request, device) as in Sec. 4.2 + GLT record
 *                    (Table "Fields of the GLT").
 *   oracle_extend    the next offload set of a placed request (the KV
 *                    caches of a later decoding step, Sec. 4.1.3): the same
 *                    steps on the new blocks alone, their own ranges.
 *   oracle_release   return all of a request's ranges.
 *   oracle_store     offload copy, Algorithm 1 (store part, MemStore).
 *   oracle_gather    retrieval copy, Sec. 4.3 "KV Retrieval".
 *
 * Readings of the paper taken here (where it is silent or ambiguous):
 *  R1 remainder: after flooring, the r leftover blocks go one each to the r
 *     devices with the largest p_i (the prose of Sec. 4.1.3 speaks of several
 *     devices; the algorithm's per-leftover step names the largest-p_i one).
 *  R2 ties in p_i: lower device index first.
 *  R3 which device a block goes to: blocks are taken in index order and
 *     block j goes to the device with room that has the largest deficit
 *     (j+1)*c_i - n*a_i  (a_i = blocks already given to i); ties to the
 *     lower index.  This stripes every request over all devices.
 *  R4 bandwidths are positive integers; p_i = b_i / sum b is never rounded:
 *     floor(p_i * n) is computed as floor(b_i * n / W) exactly.
 *  R5 placement unit: one block (block_size tokens, all layers, K and V).
 *  R6 offload set: the blocks of one place or extend call.  Counts, the
 *     interleave and the ranges of R7 are taken per set, so an extension
 *     never moves earlier blocks; all sets of a request share its gen.
 *  R7 location: a byte offset inside the device, both for host memory and
 *     for the SSD stand-in; each (request, device) gets one contiguous range
 *     of ceil(c_i * block_bytes / 4096) sectors of 4096 bytes, taken first fit
 *     from an address-ordered free list; block k of that device's share sits
 *     at base + k * block_bytes.
 *  R9 a map entry whose region is 0xFFFFFFFF is absent: skipped on store and
 *     retrieve, its destination untouched.
 *  gen: every successful place call takes the next value of a pool-wide
 *     counter starting at 1; all entries of that request carry it.
 *
 * Data layouts
 *   engine cache, per layer l and K/V: [num_slots][H][bs][D] (elem_bytes each)
 *   pool block at region + offset: for l in layers, kv in {K, V}: one chunk
 *     of C = H*bs*D*elem_bytes bytes at offset + (2l+kv)*C.  Inside a chunk
 *     layout 0 (head-major) is [H][bs][D], layout 1 (token-major) [bs][H][D].
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_ABSENT 0xFFFFFFFFu
#define ORACLE_SECTOR 4096ull

typedef struct {
    uint32_t region;
    uint32_t gen;
    uint64_t offset;
} oracle_loc;

/* ---------------------------------------------------------------- counts */

/*
 * Eq. (1): p_i = b_i / sum_j b_j.   Eq. (2): |set_i| = floor(p_i * n) + r_i,
 * with sum over i equal to n.  Returns 0, or -1 on bad input.
 */
int oracle_counts(const uint64_t *bandwidth, uint32_t n_dev, uint64_t n_kv, uint64_t *count)
{
    if (n_dev == 0) return -1;
    unsigned __int128 total = 0;
    for (uint32_t i = 0; i < n_dev; ++i) {
        if (bandwidth[i] == 0) return -1;
        total += bandwidth[i];
    }
    /* Algorithm 1, counting part: floor first */
    uint64_t assigned = 0;
    for (uint32_t i = 0; i < n_dev; ++i) {
        unsigned __int128 prod = (unsigned __int128)bandwidth[i] * n_kv;
        count[i] = (uint64_t)(prod / total);
        assigned += count[i];
    }
    /* then the remaining_count leftovers, one per device in order of
     * decreasing p_i (R1), ties to the lower index (R2) */
    uint64_t remaining = n_kv - assigned;
    char *got = (char *)calloc(n_dev, 1);
    if (!got) return -1;
    for (uint64_t k = 0; k < remaining; ++k) {
        uint32_t best = n_dev;
        for (uint32_t i = 0; i < n_dev; ++i) {
            if (got[i]) continue;
            if (best == n_dev || bandwidth[i] > bandwidth[best]) best = i;
        }
        if (best == n_dev) { free(got); return -1; } /* cannot happen: remaining < n_dev */
        got[best] = 1;
        count[best] += 1;
    }
    free(got);
    return 0;
}

/* ---------------------------------------------------------------- pool state */

typedef struct {
    uint64_t start, len;
} orange;

typedef struct {
    orange *r;
    uint32_t n, cap;
} ofreelist;

typedef struct {
    uint64_t request;
    uint32_t n_blocks;
    uint32_t gen;
    oracle_loc *map;
    uint32_t n_sets; /* offload sets placed (place, then each extend) */
    uint64_t *base;  /* [set][device]: range start (if len > 0) */
    uint64_t *len;   /* [set][device]: range length in bytes (0 = none) */
} orecord;

typedef struct {
    uint32_t n_dev;
    uint64_t *bandwidth;
    uint64_t *capacity;
    uint64_t block_bytes;
    ofreelist *free;
    orecord *rec;
    uint32_t n_rec, cap_rec;
    uint32_t next_gen;
} opool;

static int fl_insert(ofreelist *f, uint32_t at, orange v)
{
    if (f->n == f->cap) {
        uint32_t nc = f->cap ? f->cap * 2 : 8;
        orange *nr = (orange *)realloc(f->r, nc * sizeof(orange));
        if (!nr) return -1;
        f->r = nr;
        f->cap = nc;
    }
    memmove(f->r + at + 1, f->r + at, (f->n - at) * sizeof(orange));
    f->r[at] = v;
    f->n++;
    return 0;
}

static void fl_erase(ofreelist *f, uint32_t at)
{
    memmove(f->r + at, f->r + at + 1, (f->n - at - 1) * sizeof(orange));
    f->n--;
}

opool *oracle_pool_new(uint32_t n_dev, const uint64_t *bandwidth, const uint64_t *capacity,
                       uint64_t block_bytes)
{
    if (n_dev == 0 || block_bytes == 0) return 0;
    opool *p = (opool *)calloc(1, sizeof(opool));
    if (!p) return 0;
    p->n_dev = n_dev;
    p->block_bytes = block_bytes;
    p->bandwidth = (uint64_t *)malloc(n_dev * sizeof(uint64_t));
    p->capacity = (uint64_t *)malloc(n_dev * sizeof(uint64_t));
    p->free = (ofreelist *)calloc(n_dev, sizeof(ofreelist));
    p->next_gen = 1;
    for (uint32_t i = 0; i < n_dev; ++i) {
        p->bandwidth[i] = bandwidth[i];
        p->capacity[i] = capacity[i] / ORACLE_SECTOR * ORACLE_SECTOR;
        if (p->capacity[i] > 0) {
            orange whole = {0, p->capacity[i]};
            fl_insert(&p->free[i], 0, whole);
        }
    }
    return p;
}

void oracle_pool_free(opool *p)
{
    if (!p) return;
    for (uint32_t i = 0; i < p->n_rec; ++i) {
        free(p->rec[i].map);
        free(p->rec[i].base);
        free(p->rec[i].len);
    }
    for (uint32_t i = 0; i < p->n_dev; ++i) free(p->free[i].r);
    free(p->rec);
    free(p->free);
    free(p->bandwidth);
    free(p->capacity);
    free(p);
}

static int find_record(const opool *p, uint64_t request)
{
    for (uint32_t i = 0; i < p->n_rec; ++i)
        if (p->rec[i].request == request) return (int)i;
    return -1;
}

/* first fit in address order: index of the first free range with len >= need */
static int first_fit(const ofreelist *f, uint64_t need)
{
    for (uint32_t k = 0; k < f->n; ++k)
        if (f->r[k].len >= need) return (int)k;
    return -1;
}

static void give_back(ofreelist *f, uint64_t start, uint64_t len)
{
    /* insert keeping address order, then merge with neighbours */
    uint32_t at = 0;
    while (at < f->n && f->r[at].start < start) at++;
    orange v = {start, len};
    fl_insert(f, at, v);
    if (at + 1 < f->n && f->r[at].start + f->r[at].len == f->r[at + 1].start) {
        f->r[at].len += f->r[at + 1].len;
        fl_erase(f, at + 1);
    }
    if (at > 0 && f->r[at - 1].start + f->r[at - 1].len == f->r[at].start) {
        f->r[at - 1].len += f->r[at].len;
        fl_erase(f, at);
    }
}

/*
 * One offload set of n blocks (Algorithm 1 on the set): Eq. 2 counts, one
 * contiguous sector-rounded range per device with a share (Sec. 4.2, first
 * fit), then the blocks in index order to the device with room and the
 * largest deficit (R3).  Fills out[0..n) with gen and base/len[0..N).
 * Returns 0, -1 (bad input) or -3 (some device has no range large enough;
 * nothing changes).
 */
static int place_set(opool *p, uint32_t n, uint32_t gen, oracle_loc *out, uint64_t *base, uint64_t *len)
{
    const uint32_t N = p->n_dev;
    uint64_t *count = (uint64_t *)calloc(N, sizeof(uint64_t));
    uint64_t *given = (uint64_t *)calloc(N, sizeof(uint64_t));
    int *slot = (int *)malloc(N * sizeof(int));
    if (!count || !given || !slot || oracle_counts(p->bandwidth, N, n, count)) {
        free(count); free(given); free(slot);
        return -1;
    }

    /* Sec. 4.2: one contiguous range of ceil(c_i * KV_size / sector) sectors
     * per device.  Check every device first so that a failure changes nothing. */
    for (uint32_t i = 0; i < N; ++i) {
        base[i] = 0;
        len[i] = (count[i] * p->block_bytes + ORACLE_SECTOR - 1) / ORACLE_SECTOR * ORACLE_SECTOR;
        slot[i] = -1;
        if (len[i] == 0) continue;
        slot[i] = first_fit(&p->free[i], len[i]);
        if (slot[i] < 0) {
            free(count); free(given); free(slot);
            return -3;
        }
    }
    for (uint32_t i = 0; i < N; ++i) {
        if (len[i] == 0) continue;
        orange *fr = &p->free[i].r[slot[i]];
        base[i] = fr->start;
        fr->start += len[i];
        fr->len -= len[i];
        if (fr->len == 0) fl_erase(&p->free[i], (uint32_t)slot[i]);
    }

    /* Algorithm 1, partition part: blocks in index order, each to the device
     * with room and the largest deficit (R3). */
    for (uint32_t j = 0; j < n; ++j) {
        uint32_t best = N;
        __int128 best_score = 0;
        for (uint32_t i = 0; i < N; ++i) {
            if (given[i] >= count[i]) continue;
            __int128 score = (__int128)(j + 1) * (__int128)count[i] - (__int128)n * (__int128)given[i];
            if (best == N || score > best_score) {
                best = i;
                best_score = score;
            }
        }
        out[j].region = best;
        out[j].gen = gen;
        out[j].offset = base[best] + given[best] * p->block_bytes;
        given[best] += 1;
    }
    free(count);
    free(given);
    free(slot);
    return 0;
}

/*
 * Place the n_blocks blocks of one request.  Return codes: 0 ok, -1 bad
 * input or request already placed, -3 some device has no contiguous range
 * large enough (nothing changes in that case).
 */
int oracle_place(opool *p, uint64_t request, uint32_t n_blocks, oracle_loc *out)
{
    if (!p || n_blocks == 0 || find_record(p, request) >= 0) return -1;
    const uint32_t N = p->n_dev;
    uint64_t *base = (uint64_t *)calloc(N, sizeof(uint64_t));
    uint64_t *len = (uint64_t *)calloc(N, sizeof(uint64_t));
    if (!base || !len) {
        free(base); free(len);
        return -1;
    }
    const int rc = place_set(p, n_blocks, p->next_gen, out, base, len);
    if (rc) {
        free(base); free(len);
        return rc;
    }
    const uint32_t gen = p->next_gen++;

    /* UpdateGLT: keep the record */
    if (p->n_rec == p->cap_rec) {
        uint32_t nc = p->cap_rec ? p->cap_rec * 2 : 8;
        orecord *nr = (orecord *)realloc(p->rec, nc * sizeof(orecord));
        if (!nr) abort();
        p->rec = nr;
        p->cap_rec = nc;
    }
    orecord *r = &p->rec[p->n_rec++];
    r->request = request;
    r->n_blocks = n_blocks;
    r->gen = gen;
    r->map = (oracle_loc *)malloc(n_blocks * sizeof(oracle_loc));
    memcpy(r->map, out, n_blocks * sizeof(oracle_loc));
    r->n_sets = 1;
    r->base = base;
    r->len = len;
    return 0;
}

/*
 * The next offload set of a placed request: blocks n_old .. n_old+n_new-1,
 * placed as one set on their own (R6) with the request's gen.  out[0..n_new)
 * receives their entries.  Return codes: 0 ok, -1 bad input, -4 request not
 * placed, -3 no range large enough (nothing changes).
 */
int oracle_extend(opool *p, uint64_t request, uint32_t n_new, oracle_loc *out)
{
    if (!p || n_new == 0) return -1;
    const int k = find_record(p, request);
    if (k < 0) return -4;
    orecord *r = &p->rec[k];
    if ((uint64_t)r->n_blocks + n_new > 0xFFFFFFFFull) return -1;
    const uint32_t N = p->n_dev;
    uint64_t *base = (uint64_t *)realloc(r->base, (size_t)(r->n_sets + 1) * N * sizeof(uint64_t));
    if (!base) return -1;
    r->base = base;
    uint64_t *len = (uint64_t *)realloc(r->len, (size_t)(r->n_sets + 1) * N * sizeof(uint64_t));
    if (!len) return -1;
    r->len = len;
    oracle_loc *map = (oracle_loc *)realloc(r->map, (size_t)(r->n_blocks + n_new) * sizeof(oracle_loc));
    if (!map) return -1;
    r->map = map;
    const int rc = place_set(p, n_new, r->gen, out, r->base + (size_t)r->n_sets * N, r->len + (size_t)r->n_sets * N);
    if (rc) return rc;
    memcpy(r->map + r->n_blocks, out, n_new * sizeof(oracle_loc));
    r->n_blocks += n_new;
    r->n_sets += 1;
    return 0;
}

/* GLT read: the map recorded by oracle_place.  -4 if the request is unknown,
 * -1 if n_blocks differs from the placed count. */
int oracle_lookup(const opool *p, uint64_t request, uint32_t n_blocks, oracle_loc *out)
{
    int k = find_record(p, request);
    if (k < 0) return -4;
    if (p->rec[k].n_blocks != n_blocks) return -1;
    memcpy(out, p->rec[k].map, n_blocks * sizeof(oracle_loc));
    return 0;
}

int oracle_release(opool *p, uint64_t request)
{
    int k = find_record(p, request);
    if (k < 0) return -4;
    orecord *r = &p->rec[k];
    for (uint32_t set = 0; set < r->n_sets; ++set)
        for (uint32_t i = 0; i < p->n_dev; ++i) {
            const size_t at = (size_t)set * p->n_dev + i;
            if (r->len[at]) give_back(&p->free[i], r->base[at], r->len[at]);
        }
    free(r->map);
    free(r->base);
    free(r->len);
    p->rec[k] = p->rec[p->n_rec - 1];
    p->n_rec--;
    return 0;
}

/* largest free range of a device (for capacity tests) */
uint64_t oracle_largest_free(const opool *p, uint32_t dev)
{
    uint64_t best = 0;
    for (uint32_t k = 0; k < p->free[dev].n; ++k)
        if (p->free[dev].r[k].len > best) best = p->free[dev].r[k].len;
    return best;
}

/* ---------------------------------------------------------------- copies */

/* element (h, t) row of D elements inside a pool chunk, per layout */
static uint64_t pool_row(uint32_t layout, uint32_t H, uint32_t bs, uint32_t h, uint32_t t)
{
    return layout == 0 ? (uint64_t)h * bs + t : (uint64_t)t * H + h;
}

/*
 * Store (offload), Algorithm 1 store part: for every present block b and
 * every layer l, K and V: the chunk of slot src_slot[b] of the engine cache
 * goes to region[r_b] + off_b + (2l+kv)*C, in the pool's chunk layout.
 */
void oracle_store(uint32_t n_blocks, const oracle_loc *map, const int32_t *src_slot,
                  uint8_t *const *region_mem,
                  const uint8_t *const *k_layers, const uint8_t *const *v_layers,
                  uint32_t L, uint32_t H, uint32_t bs, uint32_t D, uint32_t elem_bytes,
                  uint32_t layout)
{
    const uint64_t row = (uint64_t)D * elem_bytes;
    const uint64_t C = (uint64_t)H * bs * row;
    for (uint32_t b = 0; b < n_blocks; ++b) {
        if (map[b].region == ORACLE_ABSENT) continue;
        uint8_t *blk = region_mem[map[b].region] + map[b].offset;
        for (uint32_t l = 0; l < L; ++l) {
            for (uint32_t kv = 0; kv < 2; ++kv) {
                const uint8_t *src = (kv == 0 ? k_layers[l] : v_layers[l]) + (uint64_t)src_slot[b] * C;
                uint8_t *dst = blk + (uint64_t)(2 * l + kv) * C;
                if (layout == 0) {
                    memcpy(dst, src, C);
                } else {
                    for (uint32_t h = 0; h < H; ++h)
                        for (uint32_t t = 0; t < bs; ++t)
                            memcpy(dst + pool_row(layout, H, bs, h, t) * row,
                                   src + ((uint64_t)h * bs + t) * row, row);
                }
            }
        }
    }
}

/*
 * Retrieve (Sec. 4.3): for every present block b, every layer l, K and V:
 * dst_k[l] / dst_v[l] slot dst_slot[b] <- region[r_b] + off_b + (2l+kv)*C,
 * converted from the pool's chunk layout to [H][bs][D].  Absent entries and
 * every slot not named by a present block are left untouched.
 */
void oracle_gather(uint32_t n_blocks, const oracle_loc *map, const int32_t *dst_slot,
                   const uint8_t *const *region_mem,
                   uint8_t *const *k_layers, uint8_t *const *v_layers,
                   uint32_t L, uint32_t H, uint32_t bs, uint32_t D, uint32_t elem_bytes,
                   uint32_t layout)
{
    const uint64_t row = (uint64_t)D * elem_bytes;
    const uint64_t C = (uint64_t)H * bs * row;
    for (uint32_t b = 0; b < n_blocks; ++b) {
        if (map[b].region == ORACLE_ABSENT) continue;
        const uint8_t *blk = region_mem[map[b].region] + map[b].offset;
        for (uint32_t l = 0; l < L; ++l) {
            for (uint32_t kv = 0; kv < 2; ++kv) {
                const uint8_t *src = blk + (uint64_t)(2 * l + kv) * C;
                uint8_t *dst = (kv == 0 ? k_layers[l] : v_layers[l]) + (uint64_t)dst_slot[b] * C;
                if (layout == 0) {
                    memcpy(dst, src, C);
                } else {
                    for (uint32_t h = 0; h < H; ++h)
                        for (uint32_t t = 0; t < bs; ++t)
                            memcpy(dst + ((uint64_t)h * bs + t) * row,
                                   src + pool_row(layout, H, bs, h, t) * row, row);
                }
            }
        }
    }
}

/*
 * kvpool.h -- C ABI of the MI355X (gfx950) KV-pool retrieval library.
 *
 * The library implements the data path of "Unified KV Pooling to Accelerate
 * Long-Context LLM Serving": a request's offloaded KV blocks are spread over
 * several pool regions in proportion to each region's bandwidth (Sec. 4.1.2,
 * Eq. 1; Sec. 4.1.3, Eq. 2 and Algorithm 1), recorded in a global lookup
 * table (Sec. 4.1.1, Table "Fields of the GLT"), and gathered back into the
 * GPU's paged KV cache by looking the blocks up, grouping them by region and
 * reading all regions in parallel (Sec. 4.3, "KV Retrieval").
 *
 * Pool regions ("pool devices" in the paper) are
 *   - KVP_REGION_HOST: pinned host memory bound to a NUMA node and mapped
 *     into the GPU's address space; GPU kernels read it directly over the
 *     host link (zero copy);
 *   - KVP_REGION_STAGING: a buffer in HBM that stands in for an SSD; or
 *   - KVP_REGION_FILE: a file or a block device, the storage tier, read and
 *     written with O_DIRECT by one worker thread per region (see
 *     kv_pool_create_files).
 *
 * Conventions for every function
 *   - Return 0 (KVP_OK) on success or a negative KVP_ERR_* code.  Nothing
 *     throws across the ABI.  kv_pool_last_error() gives a message for the
 *     calling thread's last failure.
 *   - All arguments are checked before any GPU work is enqueued.  A call
 *     that fails (its checks, or the library's host memory running out) has
 *     no side effects, with two exceptions: a HIP runtime error (KVP_ERR_HIP)
 *     met while a store or retrieve enqueues its work, and a failed read or
 *     write of a file region (KVP_ERR_IO), may leave part of that work
 *     enqueued or done.  The call still orders what it enqueued before later
 *     work on its stream and before a release of the requests it touched.
 *   - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 *   - Host arrays passed in (maps, block tables, pointer tables) may be freed
 *     as soon as the call returns: the library copies what it keeps.
 *   - The pool owns its regions, internal streams, events, GLT and work-list
 *     buffers.  The caller owns maps, block tables, the engine caches and
 *     its streams.
 *
 * Engine cache layout (destination of retrieve, source of store): for every
 * layer l there is one K and one V buffer in device memory, each laid out
 * [num_slots][num_kv_heads][block_size][head_dim] of elem_bytes-sized
 * elements; a "slot" is one block of block_size tokens.  Pointers must be
 * 16-byte aligned.
 *
 * Pool block layout: a placed block occupies block_bytes = 2 * L * C bytes
 * at (region, offset), C = num_kv_heads * block_size * head_dim * elem_bytes.
 * Chunk (layer l, K=0/V=1) sits at offset + (2l + kv) * C.  Inside a chunk,
 * pool_layout 0 stores [heads][tokens][head_dim] (head-major, the engine's
 * order) and pool_layout 1 stores [tokens][heads][head_dim] (token-major);
 * retrieve converts to the engine layout and store converts from it.
 */
#ifndef KVPOOL_H
#define KVPOOL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ---- */
#define KVP_OK            0
#define KVP_ERR_INVALID  -1   /* bad argument, shape, pointer, index or state */
#define KVP_ERR_NOMEM    -2   /* host or device allocation failed */
#define KVP_ERR_NOSPACE  -3   /* a region has no contiguous range large enough */
#define KVP_ERR_NOTFOUND -4   /* unknown request */
#define KVP_ERR_STALE    -5   /* map entry refers to a released or reused range */
#define KVP_ERR_HIP      -6   /* a HIP runtime call failed */
#define KVP_ERR_IO       -7   /* a read or write of a file region failed */

/* ---- region types and flags ---- */
#define KVP_REGION_HOST     0u  /* pinned, NUMA-bound, GPU-mapped host memory */
#define KVP_REGION_STAGING  1u  /* HBM buffer standing in for an SSD */
#define KVP_REGION_FILE     2u  /* a file or block device, read and written with O_DIRECT (storage tier) */

#define KVP_HOST_DEFAULT      0u  /* library's choice of host-memory coherence */
#define KVP_HOST_COHERENT     1u  /* fine-grained (coherent) pinned memory */
#define KVP_HOST_NONCOHERENT  2u  /* coarse-grained (non-coherent) pinned memory */

#define KVP_FILE_BUFFERED     1u  /* file regions: through the page cache (no O_DIRECT) */

#define KVP_ABSENT 0xFFFFFFFFu    /* kvp_loc.region of a block that is not in the pool */

/* One pool region ("pool device", Sec. 4.1.1: each gets a unique index). */
typedef struct {
    uint32_t type;            /* KVP_REGION_HOST, KVP_REGION_STAGING or KVP_REGION_FILE */
    int32_t  numa_node;       /* host: NUMA node whose memory backs it; -1 = no binding */
    uint64_t capacity_bytes;  /* usable bytes, rounded down to a multiple of 4096 */
    uint32_t flags;           /* host: KVP_HOST_*; staging: 0; file: 0 or KVP_FILE_BUFFERED */
    uint32_t reserved;        /* 0 */
} kvp_region_desc;

/* Shape of the KV cache being pooled. */
typedef struct {
    uint32_t num_layers;      /* L >= 1 */
    uint32_t num_kv_heads;    /* H >= 1 */
    uint32_t head_dim;        /* D >= 1 */
    uint32_t block_size;      /* tokens per block, >= 1 */
    uint32_t elem_bytes;      /* bytes per element (2 for bf16) */
    uint32_t pool_layout;     /* 0 head-major chunks, 1 token-major chunks */
} kvp_kv_spec;

/* Location of one block (the GLT's device_idx and location, Table "Fields of
 * the GLT"; the location is a byte offset inside the region for both region
 * types).  16 bytes. */
typedef struct {
    uint32_t region;          /* region index, or KVP_ABSENT */
    uint32_t gen;             /* placement generation; detects stale maps */
    uint64_t offset;          /* byte offset of the block inside the region */
} kvp_loc;

typedef struct kvp_pool kvp_pool;   /* opaque */

/*
 * Create a pool (Sec. 4.1.1: enumerate the pool devices, index them, and
 * initialise the GLT; Sec. 4.1.2, Eq. 1: placement ratio p_i = b_i / sum b_j).
 *   regions[n_regions]   region descriptions; region i gets index i.
 *   bandwidths[n_regions] positive integer bandwidth weights b_i (any unit,
 *                        e.g. MB/s).  Integers keep floor(p_i * n) exact.
 *                        NULL: measure them (kv_pool_measure_bandwidth with
 *                        256 MiB per region and KVP_MEASURE_SHARED_LINK |
 *                        KVP_MEASURE_FILES_TOGETHER) and use the result (not
 *                        allowed for placement-only pools).
 *   spec                 KV shape; C = H*bs*D*elem_bytes must be a multiple
 *                        of 16 (and, for pool_layout 1, so must D*elem_bytes).
 *   hip_device           GPU ordinal.  -1 creates a placement-only pool: no
 *                        memory is allocated and no HIP call is made; place,
 *                        lookup and release work, store and retrieve return
 *                        KVP_ERR_INVALID.
 *   out                  receives the pool handle.
 * Host regions are allocated with hipHostMalloc under an MPOL_BIND policy for
 * numa_node, staging regions with hipMalloc.  Errors: INVALID (bad
 * description or NUMA node not available), NOMEM, HIP.
 */
int kv_pool_create(const kvp_region_desc *regions, const uint64_t *bandwidths,
                   uint32_t n_regions, const kvp_kv_spec *spec, int hip_device,
                   kvp_pool **out);

/*
 * Create a pool whose regions may include the storage tier (Sec. 4.2, the
 * KV-passthrough to SSDs; Sec. 4.1.3, one worker per device).  Arguments as
 * kv_pool_create, plus:
 *   paths[n_regions]     for each KVP_REGION_FILE region, the file to create
 *                        or the block device to use; ignored (may be NULL)
 *                        for other regions; paths may be NULL if there is no
 *                        file region.  A path that does not exist is created
 *                        (mode 0600) and sized to the capacity, and removed
 *                        by kv_pool_destroy.  An existing path must be a
 *                        block device at least that large: it is read and
 *                        written in place and kept.  An existing regular file
 *                        is refused (KVP_ERR_INVALID), never overwritten.
 * A file region's numa_node must be -1; its flags are 0 (O_DIRECT: reads and
 * writes bypass the page cache) or KVP_FILE_BUFFERED (page cache, for file
 * systems without O_DIRECT).  A pool with a file region needs 2 * C to be a
 * multiple of 4096, so that every block, layer range and range of a request
 * is sector aligned.  Its file regions share a ring of two pinned, GPU-mapped
 * host buffers (min(256 MiB, the largest file region) each, at least one
 * block; kv_pool_set_file_ring) between the files and the engine cache.
 *
 * Retrieve and store of file-region blocks: the call runs the file reads
 * (retrieve) or writes (store) itself, by the regions' worker threads, batch
 * by batch through the ring.  A retrieve returns once every read is done and
 * the kernels moving the slots into the engine cache are enqueued on
 * `stream`; a store returns once every write is done (it waits for its own
 * kernels, and for work enqueued on `stream` before it).  Blocks of the
 * other region types in the same call are moved as kv_pool_retrieve /
 * kv_pool_store move them.  kv_pool_retrieve_noalloc refuses file-region
 * entries (KVP_ERR_INVALID); the copy-engine transport, the small-call launch
 * and kv_pool_set_timing do not cover them.  A failed file read or write
 * returns KVP_ERR_IO; batches enqueued before it may have reached the engine
 * cache (retrieve) or the file (store).
 * Errors: as kv_pool_create, plus IO (creating a file or reserving its space).
 */
int kv_pool_create_files(const kvp_region_desc *regions, const uint64_t *bandwidths,
                         uint32_t n_regions, const kvp_kv_spec *spec, int hip_device,
                         const char *const *paths, kvp_pool **out);

/*
 * Place the n_blocks blocks of one request (Algorithm 1 without the writes):
 * target counts c_i = floor(p_i * n) + r_i (Eq. 2), the r leftovers one each
 * to the regions with the largest p_i (ties: lower index); blocks taken in
 * index order, block j to the region with room whose deficit
 * (j+1)*c_i - n*a_i is largest (ties: lower index), a_i counting blocks
 * already given to region i; each region's share is one contiguous range of
 * ceil(c_i * block_bytes / 4096) sectors (Sec. 4.2), first fit in address
 * order; block k of region i's share sits at base_i + k*block_bytes.  The
 * GLT records every block (UpdateGLT).
 *   map_out[n_blocks]    caller-owned, receives (region, gen, offset).
 * Atomic: on any error (KVP_ERR_NOSPACE, or KVP_ERR_NOMEM when the library's
 * own host memory runs out) nothing is placed.  Errors: INVALID (n_blocks
 * == 0 or request already placed), NOSPACE, NOMEM, HIP.
 */
int kv_pool_place(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks, kvp_loc *map_out);

/*
 * Extend a placed request by its next n_new blocks (Sec. 4.1.3: the KV
 * caches offloaded at each decoding step form an offload set of their own,
 * and Algorithm 1 runs on that set).  Blocks n_old .. n_old+n_new-1 are
 * placed exactly as kv_pool_place places a request of n_new blocks on the
 * pool as it stands -- Eq. 2 counts of the set, the same block order, one
 * new contiguous range per region with a share -- while earlier blocks keep
 * their places.  Every entry carries the request's gen, so earlier maps stay
 * valid; kv_pool_lookup, kv_pool_retrieve_request and kv_pool_release then
 * cover all n_old + n_new blocks.  Small sets follow Eq. 2 literally: a
 * one-block set goes to the region with the largest p_i (lowest index on
 * ties).
 *   map_out[n_new]    caller-owned, receives the new blocks' entries.
 * Atomic: on any error nothing changes.  Errors: INVALID (n_new == 0, more
 * than 2^32-1 blocks in all), NOTFOUND, NOSPACE, NOMEM.
 */
int kv_pool_extend(kvp_pool *pool, uint64_t request_id, uint32_t n_new, kvp_loc *map_out);

/*
 * GLT read (Sec. 4.3, the lookup that starts a retrieval): the map of a placed
 * request.  n_blocks must equal its block count over all its offload sets
 * (kv_pool_place, then each kv_pool_extend), whose maps it returns in that
 * order.  Errors: NOTFOUND, INVALID.
 */
int kv_pool_lookup(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks, kvp_loc *map_out);

/*
 * Store (offload; Algorithm 1 store part, MemStore / SSD write): for every
 * present entry b of map and every layer l, K and V, copy slot
 * src_block_table[b] of the engine cache into the pool at
 * map[b].offset + (2l+kv)*C of region map[b].region, in pool_layout order.
 * Entries with region == KVP_ABSENT are skipped.
 *   map[n_blocks], src_block_table[n_blocks]   host arrays.
 *   src_num_slots        slots in each engine buffer; table entries of
 *                        present blocks must lie in [0, src_num_slots).
 *   k_layers[L], v_layers[L]  host arrays of device pointers.
 *   stream               work is ordered on it; the call returns after
 *                        enqueueing.  A later retrieve of these blocks on any
 *                        stream waits for this store.
 * Map entries must be blocks of live placements (else STALE) and distinct.
 * n_blocks * 4 * L may not exceed 2^31 (INVALID), for this call and for
 * kv_pool_retrieve and their layerwise forms.
 * Errors: INVALID, STALE, HIP.
 */
int kv_pool_store(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks,
                  const int32_t *src_block_table, uint32_t src_num_slots,
                  void *const *k_layers, void *const *v_layers, void *stream);

/*
 * Retrieve (Sec. 4.3, "KV Retrieval"): group the present entries by region
 * type, then read the host regions (zero-copy kernel, on `stream`) and the
 * staging regions (HBM gather kernel, on the pool's internal stream forked
 * from `stream` and joined back into it) in parallel.  A small call (see
 * kv_pool_set_launch) runs both in one launch on `stream`; otherwise a call
 * with under 32 MiB of staging-region bytes runs its HBM kernel on `stream`
 * ahead of the host-region kernel, since forking costs more.  Every chunk
 * lands in slot dst_block_table[b] of layer l's K or V buffer in the engine
 * layout.
 * Absent entries are skipped and every slot not named by a present entry is
 * left untouched.  Entries may belong to several requests: a batch retrieved
 * by one call shares one work list and one kernel per region class.
 *   map[n_blocks], dst_block_table[n_blocks]   host arrays; destination slots
 *                        of present entries must be distinct and lie in
 *                        [0, dst_num_slots).
 *   k_layers[L], v_layers[L]  host arrays of device pointers.
 * Stream ordered; returns after enqueueing.  Errors: INVALID, STALE, HIP.
 */
int kv_pool_retrieve(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks,
                     const int32_t *dst_block_table, uint32_t dst_num_slots,
                     void *const *k_layers, void *const *v_layers, void *stream);

/*
 * Allocation-free retrieve, for callers that cannot allocate memory during the
 * call (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, semantics, validation, stream ordering
 * and results as kv_pool_retrieve, except:
 *   - The work list (the engine pointers of the moved chunks, 8 bytes each,
 *     rounded up to 16, then 16 bytes per present block) goes through a
 *     static device array of KVP_NOALLOC_SCRATCH_BYTES (1 MiB) that the
 *     library holds once per GPU from the first kv_pool_create on that GPU
 *     until the process ends, with a pinned host buffer of the same size set
 *     up beside it.  A call whose list is larger -- more than 65,504 present
 *     blocks for a 32-layer model -- fails with KVP_ERR_INVALID before any
 *     work is enqueued.
 *   - The call makes no device or pinned allocation (no hipMalloc,
 *     hipHostMalloc, hipFree or other allocating routine) and creates no
 *     stream or event.  The host class always runs the zero-copy kernel
 *     (KVP_LAUNCH_SDMA is ignored: its ring is memory of its own); the call
 *     is never a small-call launch and is not timed.
 *   - The array is shared by every pool and every call on that GPU, and it
 *     keeps the last call's list; nothing in it needs to start at zero.  The
 *     library orders its users: a call's upload waits on the device for the
 *     kernels of the previous such call on that GPU (any pool, any stream),
 *     and the host waits, if need be, until the previous call's upload has
 *     left the pinned buffer.  Calls on one GPU therefore run in the order
 *     they were enqueued rather than overlapping.
 * Errors: as kv_pool_retrieve.
 */
#define KVP_NOALLOC_SCRATCH_BYTES (1u << 20)
int kv_pool_retrieve_noalloc(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks,
                             const int32_t *dst_block_table, uint32_t dst_num_slots,
                             void *const *k_layers, void *const *v_layers, void *stream);

/*
 * Retrieve by request (Sec. 4.3 as one call): read the GLT entries of blocks
 * 0..n_blocks-1 of request_id, then retrieve them exactly as kv_pool_retrieve
 * does with that map.  n_blocks must equal the request's block count over
 * all its offload sets.
 *   dst_block_table[n_blocks]  destination slot of every block.
 * Errors: NOTFOUND, INVALID, HIP.
 */
int kv_pool_retrieve_request(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks,
                             const int32_t *dst_block_table, uint32_t dst_num_slots,
                             void *const *k_layers, void *const *v_layers, void *stream);

/*
 * Layer-range variants for layerwise pipelining (Sec. 2.2.1: the engine
 * computes layer N while the KV cache of layer N+1 is fetched).  They move
 * only layers [layer_begin, layer_end) of every present block -- chunks
 * 2*layer_begin .. 2*layer_end-1 of each pool block -- with the same
 * semantics, validation and stream ordering as kv_pool_retrieve /
 * kv_pool_store.  k_layers / v_layers still have L entries; entries outside
 * the range are not read (may be NULL).  A caller overlapping compute with
 * I/O enqueues one call per layer (or per group of layers) and records its
 * own event after each.  Errors: as kv_pool_retrieve / kv_pool_store, plus
 * INVALID for an empty or out-of-range layer range.
 */
int kv_pool_retrieve_layers(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks,
                            const int32_t *dst_block_table, uint32_t dst_num_slots,
                            uint32_t layer_begin, uint32_t layer_end,
                            void *const *k_layers, void *const *v_layers, void *stream);
int kv_pool_store_layers(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks,
                         const int32_t *src_block_table, uint32_t src_num_slots,
                         uint32_t layer_begin, uint32_t layer_end,
                         void *const *k_layers, void *const *v_layers, void *stream);

/*
 * Release a request: its ranges go back to the regions' free lists (merged
 * with free neighbours) and its GLT entries are removed.  Waits for store /
 * retrieve work already enqueued on this request to finish.  Maps of it
 * become stale.  Atomic: on any error the request stays placed and whole.
 * Errors: NOTFOUND, NOMEM, HIP.
 */
int kv_pool_release(kvp_pool *pool, uint64_t request_id);

/* Destroy the pool: waits for its internal streams and for every store / retrieve
 * it enqueued, then frees everything.  NULL is a no-op.  No other call on the
 * pool may be running in another thread, or start afterwards. */
void kv_pool_destroy(kvp_pool *pool);

/* Message for the calling thread's last failed call ("" if none). */
const char *kv_pool_last_error(void);

/* ---- introspection ---- */

typedef struct {
    uint32_t type;            /* KVP_REGION_* */
    int32_t  numa_node;       /* requested node (-1 none) */
    int32_t  numa_node_actual;/* node backing the first page, -1 if unknown */
    uint32_t flags;           /* KVP_HOST_* actually used */
    uint64_t capacity_bytes;  /* usable bytes */
    uint64_t bandwidth;       /* b_i */
    void    *host_ptr;        /* host regions: CPU address; else NULL */
    void    *device_ptr;      /* address GPU kernels use; NULL for placement-only pools */
} kvp_region_info;

/* Describe region `region`.  Errors: INVALID. */
int kv_pool_region_info(const kvp_pool *pool, uint32_t region, kvp_region_info *out);

/* Synchronous copy of bytes [offset, offset+bytes) of a region into host memory
 * (diagnostics and tests).  Errors: INVALID, HIP. */
int kv_pool_region_read(kvp_pool *pool, uint32_t region, uint64_t offset, uint64_t bytes,
                        void *host_dst);

/* The library's target counts (Eq. 2 with the remainder rule) for n blocks
 * over n_regions bandwidths; host only.  Errors: INVALID. */
int kv_pool_counts(const uint64_t *bandwidths, uint32_t n_regions, uint64_t n, uint64_t *counts_out);

/* ---- measured bandwidths (pool organizer, Sec. 4.1.2) ---- */

#define KVP_MEASURE_SHARED_LINK 1u  /* divide host regions' rate by their count */
#define KVP_MEASURE_FILES_TOGETHER 2u /* read all file regions at once, as a retrieve does */
#define KVP_MEASURE_SHARED_HBM  4u  /* divide staging regions' rate by their count */

/*
 * Measure each region's read rate into HBM, the b_i of Eq. 1: the region's
 * class kernel shape streams min(probe_bytes, capacity) bytes of the region
 * into a scratch buffer (allocated for the call); an HBM staging region
 * min(max(probe_bytes, 1 GiB), capacity), since the GPU's last-level cache
 * holds the writes of a shorter copy and it would measure above the sustained
 * rate.  Best of 3 timed runs after a warm-up, in MB/s (>= 1).  Host regions are measured one at a time; all of
 * them reach the GPU over the same host link, so KVP_MEASURE_SHARED_LINK
 * divides their figure by the number of host regions.  Staging regions are
 * measured one at a time too; all of them are the one GPU's HBM, and
 * KVP_MEASURE_SHARED_HBM divides their figure by their number (Eq. 1 then
 * balances the host link against the whole HBM; on a 128K-token request that
 * placed about 165 blocks on the host regions instead of 42 and retrieved in
 * 6.26-6.35 ms against 6.17-6.23, so create does not use it).  A file region is read
 * the way a retrieve reads it: its worker thread reads its file into the
 * pool's pinned ring (min(probe_bytes, its share of the ring) bytes, best of 3
 * after a warm-up; a file the pool created is measured on a probe file
 * written beside it first, a block device is read in place from its start).
 * Without KVP_MEASURE_FILES_TOGETHER one region at a time, with it all file
 * regions at once, each credited with its probe bytes over the time until the
 * last of them finished (best of 3), so that regions sharing one device get
 * rates that add up to what they deliver together.  Region contents are read, not
 * changed.  Waits for the probes.
 *   probe_bytes   in [64 KiB, 64 GiB].
 *   mbps_out[n_regions]   caller-owned.
 * Errors: INVALID (placement-only pool, bad flags or size), NOMEM, HIP.
 */
int kv_pool_measure_bandwidth(kvp_pool *pool, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps_out);

/*
 * Replace the bandwidth weights b_i (Eq. 1) used by later kv_pool_place and
 * kv_pool_extend calls; existing placements keep their locations.
 *   bandwidths[n_regions]  positive integers.  Errors: INVALID.
 */
int kv_pool_set_bandwidths(kvp_pool *pool, const uint64_t *bandwidths);

/* ---- launch configuration and timing ---- */

#define KVP_CLASS_HOST     0u   /* work on host regions (zero-copy kernel) */
#define KVP_CLASS_STAGING  1u   /* work on staging regions (HBM kernel) */
#define KVP_OP_RETRIEVE    0u
#define KVP_OP_STORE       1u

#define KVP_LAUNCH_NT_LOAD   1u  /* non-temporal loads */
#define KVP_LAUNCH_NT_STORE  2u  /* non-temporal stores */
#define KVP_LAUNCH_LDS       4u  /* pool_layout 1: stage each chunk through LDS */
#define KVP_LAUNCH_SPLIT2    8u  /* pool_layout 0: copy each chunk as two half-chunk units
                                    (probe: 256 x 4-vector tiles instead of 256 x 8) */
#define KVP_LAUNCH_XCD      16u  /* renumber workgroups so that each of the 8 XCDs takes
                                    contiguous units (grids that are multiples of 8) */
#define KVP_LAUNCH_SDMA     32u  /* host class only: copy-engine transport (below) */
#define KVP_LAUNCH_CHUNK_MAJOR 64u /* order units chunk by chunk over all blocks (the units in
                                    flight then write neighbouring slots of one layer buffer)
                                    instead of block by block */
#define KVP_LAUNCH_UPLOAD  128u  /* on either class of an op: no small-call launch (below) */
#define KVP_LAUNCH_TILE    256u  /* workgroup-owned tiles: a workgroup moves one moved chunk of 8
                                    consecutive work items at a time, so its writes run over
                                    neighbouring slots of one per-layer buffer (instead of taking
                                    units g, g+G, ... of the whole launch) */

/* Set the grid (workgroups of 256 threads; 0 = library default) and flags
 * of one (class, op) kernel; flags replace the current ones.  Defaults: host
 * class 12 workgroups (token-major pool: 16, 20 for the store); staging class
 * 2^20, i.e. one unit per workgroup up to that many (the launch caps a grid at
 * the call's unit count), with KVP_LAUNCH_NT_LOAD | KVP_LAUNCH_NT_STORE, plus
 * KVP_LAUNCH_SPLIT2 for pool_layout 0 and KVP_LAUNCH_CHUNK_MAJOR for its
 * retrieve; KVP_LAUNCH_NT_STORE for the host-class store; KVP_LAUNCH_LDS for
 * pool_layout 1 except the host-class store.  With the default host-class
 * retrieve grid, a retrieve enqueued while a host-class store kernel of this
 * pool has not finished takes 48 workgroups: with traffic both ways the
 * link's reads need more in flight (measured on MI355X, a 128K-token
 * LLaMA-shaped store and retrieve at once: 264.6 instead of 320 ms), while
 * alone, or beside HBM-bound kernels, 12 do as well or better.  An explicit
 * grid is always used as given.
 *
 * KVP_LAUNCH_SDMA (host class, either op) replaces the zero-copy kernel by
 * the GPU's copy engines: a call's host-class blocks, grouped per region into
 * runs at consecutive offsets (one run per region for a placed request, whose
 * blocks share one range, Sec. 4.1.3), cross the host link as hipMemcpy
 * copies (2-D with the block as pitch when only a layer range moves) on the
 * pool's internal stream into a ring of 2 HBM slots of max(1 GiB, block
 * bytes) each (kv_pool_set_copy_ring); the staging-class kernel (its grid and flags) moves each
 * filled slot to or from the engine cache on `stream`, where the
 * staging-class blocks are then moved too.  The copy engines hold no compute
 * units while the bytes cross the link, so kernels running beside a retrieve
 * keep the whole GPU; the price is one HBM write and read of the host bytes.
 * For the store, whether the device-to-host copies stay on the copy engines
 * is the HIP runtime's choice: ROCm 7.2's runtime keeps them there, while the
 * 7.0 runtime that PyTorch 2.10 ships runs them as a copy kernel of its own
 * on 256 workgroups (as fast as the 12-workgroup store kernel, but holding
 * more compute units); the no-CU copy kind does not change that.
 * The ring is allocated when the flag is first set (NOMEM if it
 * does not fit) and kept until kv_pool_destroy; the grid and other flags of
 * the host class are unused while it is set.  Results are identical to the
 * kernel's.
 *
 * Small calls: when a store or retrieve moves no bytes through the
 * copy-engine ring, is not timed, and its work list -- 2 * (layers moved)
 * engine pointers plus two 8-byte words per present block -- fits in 384
 * words (3 KiB), that list travels
 * in the kernel arguments and both classes run in ONE launch: workgroups up
 * to each class's grid (capped at its units), the copy form of the host
 * class's flags (of the staging class's when no host-class block is moved),
 * without KVP_LAUNCH_XCD and KVP_LAUNCH_CHUNK_MAJOR.  This saves the
 * work-list upload and the wait between two launches (tens of microseconds
 * on MI355X); for a full 32-layer range it covers up to 160 blocks.
 * KVP_LAUNCH_UPLOAD on either class of the op turns it off (one launch per
 * class after an upload, as for larger calls).  Results are identical.
 * Errors: INVALID (unknown flags; KVP_LAUNCH_SDMA on the staging class or on
 * a placement-only pool), NOMEM, HIP. */
int kv_pool_set_launch(kvp_pool *pool, uint32_t cls, uint32_t op, uint32_t grid, uint32_t flags);

/* Bytes per slot of the copy-engine transport's 2-slot HBM ring (default
 * 1 GiB); a slot always holds at least one block, so smaller requests are
 * raised to the block size.  Each slot costs one hand-over between the copy
 * stream and `stream` (tens to hundreds of microseconds on MI355X), so larger
 * slots trade HBM for fewer hand-overs: a 128K-token LLaMA-shaped retrieve
 * measured 204.6 ms with 1 GiB slots and 210-226 ms with 256 MiB ones.  An existing ring is freed after the
 * work on it finishes and, if any host-class op uses KVP_LAUNCH_SDMA,
 * reallocated at the new size right away.
 *   slot_bytes   multiple of 4096 in [64 KiB, 64 GiB].
 * Errors: INVALID (bad size, placement-only pool), NOMEM, HIP. */
int kv_pool_set_copy_ring(kvp_pool *pool, uint64_t slot_bytes);

/* Bytes per slot of the file regions' 2-slot pinned ring (a multiple of 4096
 * in [64 KiB, 64 GiB]; raised to one block).  The ring is freed after the work
 * on it and allocated again at the new size.  If that allocation fails
 * (NOMEM), the pool has no ring: stores and retrieves with file entries, and
 * kv_pool_measure_bandwidth on a pool with file regions, return NOMEM until a
 * later call here succeeds; other transfers are unaffected.  Errors: INVALID
 * (bad size, or the pool has no file region), NOMEM, HIP. */
int kv_pool_set_file_ring(kvp_pool *pool, uint64_t slot_bytes);

typedef struct {
    float    host_ms;         /* duration of the host-class kernel, -1 if none ran; with
                                 KVP_LAUNCH_SDMA, from the first copy or kernel of the
                                 host class to its last */
    float    staging_ms;      /* duration of the staging-class kernel, -1 if none ran */
    uint32_t host_blocks;     /* blocks read from / written to host regions */
    uint32_t staging_blocks;  /* blocks read from / written to staging regions */
} kvp_timing;

/* Enable (1) or disable (0) HIP-event timing of the kernels store/retrieve
 * launch; either way the recorded history is cleared.  Timed calls take one
 * launch per class (never the small-call launch), so each class has a
 * duration of its own.  Timing events are
 * recorded on the stream each kernel runs on (the caller's stream for the
 * host class, the pool's internal stream for the staging class unless the
 * call's staging bytes are few enough to run it on the caller's; with
 * KVP_LAUNCH_SDMA both classes time on the caller's stream, except a
 * retrieve's host-class start, recorded before its first copy).
 * Errors: INVALID. */
int kv_pool_set_timing(kvp_pool *pool, int enable);

/* Durations of the kernels of the last timed store or retrieve; waits for
 * them to finish.  Errors: INVALID (timing off or nothing timed), HIP. */
int kv_pool_last_timing(kvp_pool *pool, kvp_timing *out);

typedef struct {
    uint32_t calls;           /* timed store / retrieve calls summarised */
    uint32_t host_calls;      /* of which launched a host-class kernel */
    uint32_t staging_calls;   /* of which launched a staging-class kernel */
    uint32_t reserved;
    float    host_ms_sum, host_ms_min, host_ms_max;          /* -1 when no such kernel ran */
    float    staging_ms_sum, staging_ms_min, staging_ms_max;
} kvp_timing_summary;

/* Kernel durations of every store / retrieve timed since timing was enabled
 * or since the previous summary (at most the last 4096 calls), then clears
 * that history; waits for the kernels.  Lets a caller time calls issued back
 * to back without synchronising between them.  Errors: INVALID (timing off),
 * HIP. */
int kv_pool_timing_summary(kvp_pool *pool, kvp_timing_summary *out);

/* ---- bandwidth probes (the measured peaks that bound the two kernels) ---- */

/* Streaming copy kernel: bytes from src to dst (device-visible addresses,
 * 16-byte aligned, bytes a multiple of 16), `grid` workgroups of 256
 * threads (0 = default), KVP_LAUNCH_NT_* and KVP_LAUNCH_SPLIT2 flags, on
 * `stream` of the current device.  Errors: INVALID, HIP. */
int kv_probe_copy_kernel(void *dst, const void *src, uint64_t bytes, uint32_t grid,
                         uint32_t flags, void *stream);

/* hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, stream): the copy
 * engines' rate over the same buffers.  Errors: HIP. */
int kv_probe_memcpy(void *dst, const void *src, uint64_t bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KVPOOL_H */

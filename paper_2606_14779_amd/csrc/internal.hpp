// Internal types of the KV-pool library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <map>
#include <memory>
#include <mutex>
#include <deque>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "kvpool.h"

namespace kvp {

// ---------------------------------------------------------------- errors

struct Error {
    int code;
    std::string msg;
};

[[noreturn]] void fail(int code, const std::string &msg);
void check_hip(hipError_t e, const char *what);   // on failure: clears the last error, throws HIP
void clear_hip_error();                            // take a failed call's code off the thread

constexpr uint64_t kSector = 4096;   // allocation granule of every region (the LBA-range rule's sector)

inline uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Make `dev` the calling thread's device for the scope, then restore.
class DeviceScope {
public:
    explicit DeviceScope(int dev)
    {
        if (dev < 0) return;
        check_hip(hipGetDevice(&old_), "hipGetDevice");
        if (old_ != dev) check_hip(hipSetDevice(dev), "hipSetDevice");
        else old_ = -1;
    }
    ~DeviceScope()
    {
        if (old_ >= 0) (void)hipSetDevice(old_);
    }

private:
    int old_ = -1;
};


// ---------------------------------------------------------------- placement (Sec. 4.1.2-4.1.3)

// Eq. (2) target counts with the remainder rule.  Throws INVALID on bad input.
void target_counts(const uint64_t *bandwidth, uint32_t n_dev, uint64_t n_blocks, uint64_t *counts);

// Algorithm 1 partition: region of every block, striped by largest deficit.
void stripe(const std::vector<uint64_t> &counts, uint32_t n_blocks, std::vector<uint32_t> &region_of);

// Address-ordered first-fit allocator of byte ranges with coalescing on free.
class RangeAllocator {
public:
    explicit RangeAllocator(uint64_t capacity = 0);
    bool first_fit(uint64_t len, uint64_t *start) const;
    // All-or-nothing; allocates nothing (cannot fail) when start begins a free range,
    // as every range that first_fit finds does.
    void take(uint64_t start, uint64_t len);
    // Makes the next k calls of give() allocation-free.  May throw (out of
    // host memory), leaving the free ranges as they were.
    void reserve_gives(size_t k);
    // Cannot fail within the reserved count.
    void give(uint64_t start, uint64_t len);
    uint64_t largest() const;

private:
    using Free = std::map<uint64_t, uint64_t>;
    Free free_;                             // start -> length
    std::vector<Free::node_type> spare_;    // unlinked nodes for give()
};

// ---------------------------------------------------------------- GLT (Sec. 4.1.1)

struct GltEntry {
    uint64_t request;
    uint32_t block;
    uint32_t region;    // device_idx
    uint32_t type;      // KVP_REGION_HOST (MEM) / KVP_REGION_STAGING (SSD stand-in)
    uint32_t gen;
    uint64_t offset;    // location
};

// Open-addressing hash table keyed by (request, block).  reserve() makes room
// for that many further entries and is all-or-nothing; inserts within the
// reserved room allocate nothing, so they cannot fail.
class Glt {
public:
    Glt();
    void reserve(size_t extra);
    void insert(const GltEntry &e);
    const GltEntry *find(uint64_t request, uint32_t block) const;
    bool erase(uint64_t request, uint32_t block);
    size_t size() const { return count_; }

private:
    static uint64_t hash(uint64_t request, uint32_t block);
    void place(const GltEntry &e);
    std::vector<GltEntry> slots_;
    std::vector<uint8_t> used_;
    size_t count_ = 0;
};

// ---------------------------------------------------------------- pool state

struct RequestRec;

struct Allocation {       // one contiguous range of one request in one region
    RequestRec *owner;
    uint32_t region;
    uint32_t gen;
    uint64_t base;
    uint64_t blocks;      // blocks of the request stored in this range
    uint64_t len;         // bytes reserved (sector-rounded)
};

struct RequestRec {
    uint64_t id;
    uint32_t n_blocks;              // over all offload sets (place, then each extend)
    uint32_t gen;
    std::deque<Allocation> ranges;  // one per (offload set, region); stable addresses
    hipEvent_t stored = nullptr;   // recorded after each store touching the request
    hipEvent_t busy = nullptr;     // recorded after each store / retrieve touching it; each record
                                   // covers the one before it, so it waits for every earlier call
    bool stored_rec = false;
    bool busy_rec = false;
    hipStream_t busy_stream = nullptr;   // stream of the last busy record
    uint64_t call_mark = 0;         // the last store / retrieve call that listed it (pool lock held)
};

struct Region {
    kvp_region_desc desc{};
    uint64_t bandwidth = 0;
    uint64_t capacity = 0;
    void *host = nullptr;
    void *dev = nullptr;
    int numa_actual = -1;
    uint32_t flags_used = 0;
    RangeAllocator alloc;
    std::map<uint64_t, Allocation *> live;   // base -> allocation
    // file regions: the open file or block device, and its worker thread
    int fd = -1;
    bool file_owned = false;                 // created by the pool: removed at destroy
    std::string file_path;
    uint32_t worker = 0;
};

// ---------------------------------------------------------------- file regions (fileio.cpp)

struct IoGroup {                 // a set of reads or writes waited for together
    std::mutex mu;
    std::condition_variable cv;
    uint32_t pending = 0;
    int err = 0;                 // first failure's errno, with its message
    std::string what;
    std::chrono::steady_clock::time_point done_at;   // when pending last fell to 0
};

struct IoJob {
    int fd = -1;
    bool write = false;
    uint64_t off = 0;            // in the file, sector aligned
    uint64_t len = 0;            // sector multiple
    char *buf = nullptr;         // sector aligned
    IoGroup *group = nullptr;
};

// One worker thread per file region (the per-device workers of Sec. 4.1.3):
// each runs the reads and writes of its region in submission order.
class FileWorkers {
public:
    explicit FileWorkers(size_t n);
    ~FileWorkers();
    void submit(size_t worker, const IoJob &job);

private:
    struct Worker {
        std::thread th;
        std::mutex mu;
        std::condition_variable cv;
        std::deque<IoJob> q;
        bool stop = false;
    };
    static void run(Worker &w);
    void shutdown();
    std::vector<std::unique_ptr<Worker>> w_;
};

void io_wait(IoGroup &g);            // waits, then throws KVP_ERR_IO on a failure
void io_drain(IoGroup &g) noexcept;  // waits, forgets any failure

// One file read or write: `len` bytes at `file_off` of a region, to or from
// offset `slot_off` of a ring slot.
struct FileSpan {
    uint32_t region;
    uint64_t file_off;
    uint64_t len;
    uint64_t slot_off;
};

// The blocks moved through one ring slot: work items [first, first + n) and
// spans [span0, span0 + spans).
struct FileBatch {
    uint32_t ring;
    uint32_t first, n;
    size_t span0, spans;
};

struct FileGeometry {
    uint64_t base;         // device address of slot 0
    uint64_t slot_bytes;
    uint32_t slots;
    uint32_t next;         // ring slot of the first batch
    uint64_t block_bytes;
    uint64_t chunk_bytes;
};

void open_file_region(Region &r, const char *path);   // creates (or opens a block device); sets fd
void close_file_region(Region &r) noexcept;          // closes; removes a file the pool created
void file_region_read(const Region &r, uint64_t offset, uint64_t bytes, void *dst);
struct Pool;
// MB/s of each file region through the retrieve's own path (the region's
// worker, into the pool's pinned ring), one region at a time or all at once
// (together); entries of other regions are left as they are.
void measure_file_regions(Pool &p, uint64_t probe_bytes, bool together, uint64_t *mbps);

struct LaunchCfg {
    uint32_t grid;
    uint32_t flags;
    bool default_grid;   // the library chose the grid (it may then adapt it per call)
};

struct Slot {                    // one work-list buffer of the upload ring
    void *host = nullptr;        // pinned
    void *dev = nullptr;
    size_t cap = 0;
    hipEvent_t done = nullptr;   // recorded on the caller stream after the call's kernels
    bool pending = false;
};

struct TimedCall {                // one store / retrieve recorded while timing is on
    hipEvent_t t0[2] = {nullptr, nullptr};
    hipEvent_t t1[2] = {nullptr, nullptr};
    uint32_t blocks[2] = {0, 0};
    bool ran[2] = {false, false};
};

// Work-list scratch of kv_pool_retrieve_noalloc: one static device array per
// GPU (kernels.hip), shared by every pool and call on that GPU.  `dev` is the
// array's device address on that GPU (never the array's host-side name);
// `host` is a pinned buffer of the same size, allocated once with it, in
// which the host writes a call's list before the upload.  `staged` is
// recorded after a call's upload (the host buffer may then be rewritten),
// `free` after its kernels (the device array may then be overwritten).
// Nothing here is ever released: each GPU keeps them until the process ends,
// and no destructor makes a HIP call at exit.
constexpr uint64_t kScratchBytes = 1ull << 20;

struct ScratchDevice {
    std::mutex mu;          // serialises the calls that use the array, in enqueue order
    bool ready = false;
    void *dev = nullptr;
    void *host = nullptr;
    hipEvent_t staged = nullptr, free = nullptr;
    bool staged_rec = false, free_rec = false;
};

// Set up the scratch of `device` (the current device) on first use: the
// array's address by hipGetSymbolAddress, the pinned buffer and the events.
// Thread safe.  Throws HIP / NOMEM.
ScratchDevice &scratch_setup(int device);
// The scratch of a device whose set-up is done (INVALID otherwise); allocates nothing.
ScratchDevice &scratch_device(int device);

constexpr uint32_t kBounceSlots = 2;                 // copy-engine transport: ring slots
constexpr uint64_t kBounceSlotMin = 1ull << 30;      //   default bytes per slot (one block at least)

constexpr uint32_t kFileSlots = 2;                   // file regions: pinned ring slots
constexpr uint64_t kFileSlotMax = 256ull << 20;      //   default bytes per slot (one block at least)

struct Pool {
    int device = -1;
    bool placement_only = true;
    kvp_kv_spec spec{};
    uint64_t chunk_bytes = 0;
    uint64_t block_bytes = 0;
    std::vector<Region> regions;
    std::vector<uint64_t> bandwidth;
    std::unordered_map<uint64_t, std::unique_ptr<RequestRec>> requests;
    Glt glt;
    uint32_t next_gen = 1;
    uint64_t call_epoch = 0;        // numbers the store / retrieve calls
    mutable std::mutex mu;

    hipStream_t s_stage = nullptr;     // the staging-class kernel's stream (host class: caller's);
                                       // with KVP_LAUNCH_SDMA the host-link copies' stream instead
    hipEvent_t fork = nullptr, stage_done = nullptr;
    hipEvent_t uploaded = nullptr;     // a call's work list is in device memory (s_stage)
    // host link, per direction [op]: the last host-class kernel enqueued; the
    // next one (any stream) waits for it, so calls take the link in turn
    hipEvent_t link_done[2] = {nullptr, nullptr};
    bool link_rec[2] = {false, false};
    hipStream_t link_stream[2] = {nullptr, nullptr};   // stream of that kernel (same stream: no wait)
    std::vector<Slot> ring;
    uint32_t ring_next = 0;
    LaunchCfg launch[2][2];      // [class][op]

    // copy-engine transport of the host class (KVP_LAUNCH_SDMA): hipMemcpy on
    // s_stage between host regions and an HBM bounce ring, HBM kernel between
    // the ring and the engine cache; allocated when first enabled
    char *bounce = nullptr;
    uint64_t bounce_slot_bytes = 0;
    uint64_t bounce_slot_request = kBounceSlotMin;   // kv_pool_set_copy_ring
    hipEvent_t bounce_filled[kBounceSlots] = {};
    hipEvent_t bounce_free[kBounceSlots] = {};   // last reader / writer of the slot done
    bool bounce_free_rec[kBounceSlots] = {};
    uint32_t bounce_next = 0;

    // file regions: a worker per region, and a ring of pinned, GPU-mapped
    // slots between the files and the engine cache
    std::unique_ptr<FileWorkers> workers;
    char *file_ring = nullptr;         // host address of slot 0
    uint64_t file_ring_dev = 0;        // its device address
    uint64_t file_slot_bytes = 0;
    hipEvent_t file_free[kFileSlots] = {};   // the last kernel reading or filling the slot is done
    bool file_free_rec[kFileSlots] = {};
    IoGroup file_io[kFileSlots];       // the slot's reads or writes
    uint32_t file_next = 0;

    bool timing = false;
    std::vector<TimedCall> timed;      // calls recorded since timing was enabled or last summarised
    std::vector<hipEvent_t> spare;     // timing events ready for reuse
};

// ---------------------------------------------------------------- helpers shared by the pool sources

void free_slot(Slot &s);                                    // pool.cpp: one work-list buffer
void release_bounce(Pool &p);                               // pool.cpp: copy-engine ring, after its work
void ensure_bounce(Pool &p);                                // pool.cpp: copy-engine ring on first use
void measure_regions(Pool &p, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps);   // control.cpp
void alloc_file_ring(Pool &p, uint64_t slot_bytes);         // pool.cpp: the file regions' ring
void free_file_ring(Pool &p);                               // pool.cpp: after the work on it
void drain_timed(Pool &p, kvp_timing_summary *sum);        // transfer.cpp: wait, summarise, recycle

// ---------------------------------------------------------------- kernels (kernels.hip)

struct CopyItem {          // 16 bytes, one block of work
    uint64_t pool;         // device-visible address of the block in its region
    uint32_t slot;         // engine-cache slot
    uint32_t reserved;
};

struct CopyArgs {
    const CopyItem *items;     // device
    const uint64_t *cache;     // device, [chunks]: engine buffer of moved chunk k, i.e. the K (even
                               // chunk0 + k) or V (odd) buffer of layer (chunk0 + k) / 2
    uint32_t n_items;
    uint32_t chunks;           // chunks per item moved by this launch: 2 * (layers in range)
    uint32_t chunk0;           // first chunk: 2 * first layer
    uint32_t parts;            // units per chunk (1, or 2 with KVP_LAUNCH_SPLIT2 on plain chunks)
    uint32_t xcd_remap;        // 1: renumber workgroups so each XCD takes contiguous units
    uint32_t chunk_major;      // 1: units ordered chunk, item, part (else item, chunk, part)
    uint64_t chunk_bytes;      // C, multiple of 16
    uint32_t heads;            // token-major conversion: H
    uint32_t tokens;           //   bs
    uint32_t row_vec;          //   D*elem_bytes/16
    uint32_t layout;           // 0 head-major, 1 token-major
    uint32_t tile_items;       // > 0: workgroup-owned tiles of this many items x 1 moved chunk
};

// A call whose work list is small enough travels in the kernel arguments,
// and both classes run in one launch: workgroups [0, grid_host) take the
// host-class items [0, n_host), the others the staging-class items.  There is
// then no work-list upload and no second launch to wait for.
constexpr uint32_t kInlineWords = 384;   // 3 KiB: [chunks cache pointers][items, two words each]

struct SmallCallArgs {
    CopyArgs a;                // geometry; a.items and a.cache unused, a.n_items = all items
    uint32_t n_host;           // items [0, n_host) are host-class, the rest staging-class
    uint32_t grid_host;        // workgroups taking the host-class items (the rest: staging)
    uint64_t words[kInlineWords];
};
// passed by value as the kernel's only argument: it must fit the 4 KiB kernel-argument segment
static_assert(sizeof(SmallCallArgs) <= 4096, "small-call arguments exceed the kernel-argument segment");

// ---------------------------------------------------------------- copy-engine plan (bounce.cpp)

struct HostBlock {         // one host-class block of a call
    uint32_t region;
    uint64_t offset;       // in the region
    uint32_t slot;         // engine-cache slot
};

// One host-link copy: `blocks` blocks of one region at consecutive offsets,
// the moved part of each (`width` bytes) packed back to back in a ring slot.
struct LinkRun {
    uint32_t region;
    uint64_t offset;       // of the first block in the region
    uint32_t blocks;
    uint64_t slot_offset;  // where the first block's part sits in the ring slot
};

// The blocks that go through one ring slot: work items [first, first + n)
// and runs [run0, run0 + runs).
struct Batch {
    uint32_t ring;
    uint32_t first, n;
    size_t run0, runs;
};

struct RingGeometry {
    uint64_t base;         // device address of slot 0
    uint64_t slot_bytes;   // >= block_bytes
    uint32_t slots;
    uint32_t next;         // ring slot of the first batch
    uint64_t block_bytes;
    uint64_t chunk_bytes;
};

// Pack a call's host-class blocks into ring slots: grouped by region
// (stable), cut into runs where offsets stop being consecutive or a slot
// fills.  Appends one work item per block, addressing the block's part in
// its slot less chunk0 chunks (the kernel adds (chunk0 + k) chunks).
void plan_bounce(const RingGeometry &g, std::vector<HostBlock> &blocks, uint64_t width, uint32_t chunk0,
                 std::vector<CopyItem> &items, std::vector<LinkRun> &runs, std::vector<Batch> &batches);

// Pack a call's file-class blocks into ring slots: grouped by region, in
// offset order within a region; the moved part of each block (`width` bytes
// from `skip` on) back to back in a slot, and neighbouring blocks of a region
// merged into one span when whole blocks move.  Appends one work item per
// block, addressing its part in the slot less chunk0 chunks.
void plan_file(const FileGeometry &g, std::vector<HostBlock> &blocks, uint64_t skip, uint64_t width, uint32_t chunk0,
               std::vector<CopyItem> &items, std::vector<FileSpan> &spans, std::vector<FileBatch> &batches);


// cls: KVP_CLASS_HOST / KVP_CLASS_STAGING / kClassRing (selects the kernel
// entry point: zero-copy host region, HBM staging region, copy-engine ring);
// gather: pool -> cache (retrieve); !gather: cache -> pool (store)
constexpr uint32_t kClassRing = 2;
constexpr uint32_t kClassFile = 4;   // a file regions' ring slot (pinned host memory)
hipError_t launch_chunk_copy(const CopyArgs &a, uint32_t cls, bool gather, uint32_t grid, uint32_t flags,
                             hipStream_t s);
// One launch of both classes for a call whose table and items are already in
// f.words (f.a.chunks pointers, then f.a.n_items items); the copy form comes
// from `flags`, the workgroups of each class from its grid, capped at its units.
hipError_t launch_small_call(SmallCallArgs &f, bool gather, uint32_t grid_host, uint32_t grid_staging,
                             uint32_t flags, hipStream_t s);
hipError_t launch_probe_copy(void *dst, const void *src, uint64_t bytes, uint32_t grid,
                             uint32_t flags, hipStream_t s);
uint32_t default_grid(uint32_t cls, uint32_t op, const kvp_kv_spec &spec);
uint32_t default_flags(uint32_t cls, uint32_t op, const kvp_kv_spec &spec);

}  // namespace kvp

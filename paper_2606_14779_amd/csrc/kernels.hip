// Data-movement kernels of the KV pool, for gfx950 (MI355X).
//
// Nothing here is a contraction, so there is no MFMA: every kernel is a bit
// copy of 16-byte vectors.  One unit of work is one (block, layer, K/V)
// chunk of C bytes, or half of one (KVP_LAUNCH_SPLIT2, plain chunks only).
// A 256-thread workgroup (four 64-lane wavefronts) copies a whole unit per
// step; each lane holds up to UNROLL 16-byte loads in flight before it
// stores, so a workgroup keeps 256*UNROLL*16 bytes in flight (32 KiB at
// UNROLL = 8, one LLaMA-shaped chunk).  Loads and stores of a wavefront cover
// 1 KiB of contiguous memory, which the memory system merges into full
// 128-byte lines.
//
// The grid is persistent: workgroup g takes units g, g+G, g+2G, ...  With K
// moved chunks per block (2L for all layers, fewer for a layer range), unit
// u is part u % parts of moved chunk (u / parts) % K of work item
// u / (K*parts), so neighbouring workgroups read neighbouring pieces of the
// same pool block (the pool side streams through memory in address order).  There is no data
// reuse; an optional renumbering that gives each of the 8 XCDs contiguous
// units (KVP_LAUNCH_XCD) measured no better than the round-robin default, and
// so did the optional chunk-major order (KVP_LAUNCH_CHUNK_MAJOR), in which the
// units in flight write neighbouring slots of one per-layer engine buffer.
// The work list and the engine pointer table are read with scalar loads, and
// the next unit's entries are fetched while the current unit is copied.
//
// Five entry points share the body, so that traces and counters tell them
// apart: host_region_copy (zero-copy reads or writes of pinned host regions
// over the host link), staging_region_copy (HBM staging regions),
// ring_slot_copy (a copy-engine ring slot in HBM, whose host-link leg is a
// hipMemcpy), file_slot_copy (a file regions' ring slot in pinned host
// memory, filled or emptied by file reads and writes), and small_call_copy
// (both region classes of a call whose work list fits in the kernel
// arguments, in one launch with no upload).
//
// Three copy forms:
//   - head-major pool chunks: the chunk is [H][bs][D] on both sides; a plain
//     contiguous copy (this moves the layer axis from inside the block to
//     the per-layer engine buffers).
//   - token-major pool chunks, direct: every 16-byte vector of a [bs][H][D]
//     chunk maps to one vector of the [H][bs][D] chunk; both sides move in
//     runs of D*elem_bytes bytes.
//   - token-major pool chunks, LDS-staged: the chunk is read contiguously
//     into LDS, then written contiguously in the other order, so both global
//     sides are fully contiguous per workgroup.

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "internal.hpp"

namespace kvp {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
// Every buffer the kernels touch is global memory (HBM or mapped host
// memory); saying so lets the compiler emit global_* instead of flat_*
// accesses, which do not occupy the LDS counter.
typedef __attribute__((address_space(1))) v4u gv4u;

constexpr uint32_t kThreads = 256;
constexpr uint32_t kXcds = 8;     // MI355X: 8 accelerator complex dies, 32 CUs each
constexpr uint64_t kMaxLdsChunk = 64 * 1024;
constexpr uint32_t kTileItems = 8;  // KVP_LAUNCH_TILE: work items per workgroup-owned tile

template <bool NT>
__device__ __forceinline__ v4u load16(const v4u *p)
{
    const gv4u *g = (const gv4u *)p;
    if constexpr (NT)
        return __builtin_nontemporal_load(g);
    else
        return *g;
}

template <bool NT>
__device__ __forceinline__ void store16(v4u *p, v4u v)
{
    gv4u *g = (gv4u *)p;
    if constexpr (NT)
        __builtin_nontemporal_store(v, g);
    else
        *g = v;
}

// Loads of a batch must not sit under per-lane branches: the compiler then
// waits for each load before issuing the next, leaving one 16-byte load in
// flight per lane.  Out-of-range lanes therefore load a clamped (valid)
// index and only their stores are predicated.
__device__ __forceinline__ uint32_t clamp_index(uint32_t v, uint32_t nvec) { return v < nvec ? v : nvec - 1; }

// Workgroup-cooperative contiguous copy of nvec 16-byte vectors.
template <int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void wg_copy(const v4u *__restrict__ src, v4u *__restrict__ dst, uint32_t nvec)
{
    const uint32_t tid = threadIdx.x;
    uint32_t base = 0;
    for (; base + kThreads * UNROLL <= nvec; base += kThreads * UNROLL) {
        v4u r[UNROLL];
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) r[i] = load16<NTL>(src + base + i * kThreads + tid);
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) store16<NTS>(dst + base + i * kThreads + tid, r[i]);
    }
    if (base < nvec) {  // ragged tail: one batch, clamped loads, predicated stores
        v4u r[UNROLL];
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) r[i] = load16<NTL>(src + clamp_index(base + i * kThreads + tid, nvec));
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = base + i * kThreads + tid;
            if (v < nvec) store16<NTS>(dst + v, r[i]);
        }
    }
}

// Index maps between the two chunk orders, in 16-byte vectors; rv vectors
// make one head_dim row.  Head-major [H][bs][rv] index v <-> token-major
// [bs][H][rv] index.
__device__ __forceinline__ uint32_t hm_to_tm(uint32_t v, uint32_t heads, uint32_t tokens, uint32_t rv)
{
    const uint32_t row = v / rv, w = v - row * rv;
    const uint32_t h = row / tokens, t = row - h * tokens;
    return (t * heads + h) * rv + w;
}

__device__ __forceinline__ uint32_t tm_to_hm(uint32_t v, uint32_t heads, uint32_t tokens, uint32_t rv)
{
    const uint32_t row = v / rv, w = v - row * rv;
    const uint32_t t = row / heads, h = row - t * heads;
    return (h * tokens + t) * rv + w;
}

// Source index of destination vector v.  GATHER: destination head-major
// (cache), source token-major (pool); store: the reverse.
template <bool GATHER>
__device__ __forceinline__ uint32_t src_of(uint32_t v, uint32_t heads, uint32_t tokens, uint32_t rv)
{
    if constexpr (GATHER)
        return hm_to_tm(v, heads, tokens, rv);
    else
        return tm_to_hm(v, heads, tokens, rv);
}

// Direct token-major <-> head-major chunk conversion.  The lane index runs
// over the destination, so stores are contiguous; loads come in runs of rv
// vectors (one head_dim row).
template <bool GATHER, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void wg_convert(const v4u *__restrict__ src, v4u *__restrict__ dst, uint32_t nvec,
                                           uint32_t heads, uint32_t tokens, uint32_t rv)
{
    const uint32_t tid = threadIdx.x;
    for (uint32_t base = 0; base < nvec; base += kThreads * UNROLL) {
        v4u r[UNROLL];
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = clamp_index(base + i * kThreads + tid, nvec);
            r[i] = load16<NTL>(src + src_of<GATHER>(v, heads, tokens, rv));
        }
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = base + i * kThreads + tid;
            if (v < nvec) store16<NTS>(dst + v, r[i]);
        }
    }
}

// LDS-staged conversion: the chunk is read contiguously into LDS (UNROLL
// 16-byte loads in flight per lane, as in the plain copy), then written
// contiguously in the other order out of LDS.
template <bool GATHER, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void wg_convert_lds(const v4u *__restrict__ src, v4u *__restrict__ dst, uint32_t nvec,
                                               uint32_t heads, uint32_t tokens, uint32_t rv, v4u *lds)
{
    const uint32_t tid = threadIdx.x;
    for (uint32_t base = 0; base < nvec; base += kThreads * UNROLL) {
        v4u r[UNROLL];
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) r[i] = load16<NTL>(src + clamp_index(base + i * kThreads + tid, nvec));
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = base + i * kThreads + tid;
            if (v < nvec) lds[v] = r[i];
        }
    }
    __syncthreads();
    for (uint32_t base = 0; base < nvec; base += kThreads * UNROLL) {
        v4u r[UNROLL];
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = clamp_index(base + i * kThreads + tid, nvec);
            r[i] = lds[src_of<GATHER>(v, heads, tokens, rv)];
        }
#pragma unroll
        for (int i = 0; i < UNROLL; ++i) {
            const uint32_t v = base + i * kThreads + tid;
            if (v < nvec) store16<NTS>(dst + v, r[i]);
        }
    }
    __syncthreads();  // LDS is reused by the next chunk
}

enum Form { kPlain = 0, kConvert = 1, kConvertLds = 2 };

// The work list and the engine pointer table are written by the host before
// the launch and only read here; reading them through the constant address
// space lets the compiler use scalar loads (uniform per workgroup) instead
// of vector loads, and the next unit's entries are fetched while the current
// chunk is copied.
typedef __attribute__((address_space(4))) const CopyItem citem_t;
typedef __attribute__((address_space(4))) const uint64_t cptr_t;

struct Unit {
    uint64_t pool;   // device address of the chunk in its region
    uint64_t cache;  // device address of the chunk in the engine cache
};

// Unit u of a launch: item u / (chunks * parts), then chunk, then part of
// the chunk (parts > 1 only for plain chunks); or, chunk-major, chunk
// u / (items * parts), then item, then part, so that the units in flight
// write neighbouring slots of one per-layer buffer.  table[k] is the engine
// buffer of moved chunk k; the pool block holds chunk chunk0 + k.
__device__ __forceinline__ Unit unit_at(const CopyArgs &a, citem_t *items, cptr_t *table, uint32_t u)
{
    uint32_t item, k, p;
    if (a.chunk_major) {
        const uint32_t per_chunk = a.n_items * a.parts;
        k = u / per_chunk;
        const uint32_t r = u - k * per_chunk;
        item = r / a.parts;
        p = r - item * a.parts;
    } else {
        const uint32_t per_item = a.chunks * a.parts;
        item = u / per_item;
        const uint32_t r = u - item * per_item;
        k = r / a.parts;
        p = r - k * a.parts;
    }
    const uint32_t c = a.chunk0 + k;
    const uint64_t part = static_cast<uint64_t>(p) * (a.chunk_bytes / a.parts);
    const uint64_t pool = items[item].pool;
    const uint64_t slot = items[item].slot;
    return Unit{pool + static_cast<uint64_t>(c) * a.chunk_bytes + part, table[k] + slot * a.chunk_bytes + part};
}

// Workgroup g of the G that share the launch's a.n_items items takes units
// g, g + G, g + 2G, ...
template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void chunk_copy_body(const CopyArgs &a, citem_t *items, cptr_t *table, uint32_t g,
                                                uint32_t G)
{
    extern __shared__ v4u lds[];
    const uint32_t units = a.n_items * a.chunks * a.parts;
    const uint32_t nvec = static_cast<uint32_t>((a.chunk_bytes / a.parts) >> 4);
    uint32_t u = g;
    if (u >= units) return;
    Unit cur = unit_at(a, items, table, u);
    for (;;) {
        const uint32_t nu = u + G;
        const bool more = nu < units;
        const Unit next = more ? unit_at(a, items, table, nu) : cur;   // fetched while this chunk is copied
        const v4u *src = reinterpret_cast<const v4u *>(GATHER ? cur.pool : cur.cache);
        v4u *dst = reinterpret_cast<v4u *>(GATHER ? cur.cache : cur.pool);
        if constexpr (FORM == kPlain)
            wg_copy<UNROLL, NTL, NTS>(src, dst, nvec);
        else if constexpr (FORM == kConvert)
            wg_convert<GATHER, UNROLL, NTL, NTS>(src, dst, nvec, a.heads, a.tokens, a.row_vec);
        else
            wg_convert_lds<GATHER, UNROLL, NTL, NTS>(src, dst, nvec, a.heads, a.tokens, a.row_vec, lds);
        if (!more) break;
        u = nu;
        cur = next;
    }
}

// Workgroup-owned tiles (KVP_LAUNCH_TILE): tile t is moved chunk t % K of
// the a.tile_items consecutive work items from (t / K) * a.tile_items on;
// workgroup g takes tiles g, g+G, ... and copies each itself, item by item
// (the parts of a chunk in turn).  Its writes then run over neighbouring
// slots of one per-layer engine buffer, and its reads over the same chunk
// of neighbouring pool blocks.
template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void chunk_copy_tiles(const CopyArgs &a, citem_t *items, cptr_t *table, uint32_t g,
                                                 uint32_t G)
{
    extern __shared__ v4u lds[];
    const uint32_t K = a.chunks, TB = kTileItems;   // a.tile_items is kTileItems when set
    const uint32_t tiles = (a.n_items + TB - 1) / TB * K;
    const uint64_t part_bytes = a.chunk_bytes / a.parts;
    const uint32_t nvec = static_cast<uint32_t>(part_bytes >> 4);
    for (uint32_t t = g; t < tiles; t += G) {
        const uint32_t grp = t / K, k = t - grp * K;
        const uint32_t i0 = grp * TB;
        const uint32_t ni = a.n_items - i0 < TB ? a.n_items - i0 : TB;
        const uint64_t cache = table[k];
        const uint64_t coff = static_cast<uint64_t>(a.chunk0 + k) * a.chunk_bytes;
        // the tile's work items, all fetched (scalar loads) before its first copy;
        // indices past the last item are clamped to it and never copied
        uint64_t pool_of[kTileItems], slot_of[kTileItems];
#pragma unroll
        for (uint32_t j = 0; j < kTileItems; ++j) {
            const uint32_t i = i0 + (j < ni ? j : ni - 1);
            pool_of[j] = items[i].pool + coff;
            slot_of[j] = cache + static_cast<uint64_t>(items[i].slot) * a.chunk_bytes;
        }
#pragma unroll
        for (uint32_t j = 0; j < kTileItems; ++j) {
            if (j >= ni) break;
            const uint64_t pool = pool_of[j], slot = slot_of[j];
            for (uint32_t p = 0; p < a.parts; ++p) {
                const uint64_t off = p * part_bytes;
                const v4u *src = reinterpret_cast<const v4u *>(GATHER ? pool + off : slot + off);
                v4u *dst = reinterpret_cast<v4u *>(GATHER ? slot + off : pool + off);
                if constexpr (FORM == kPlain)
                    wg_copy<UNROLL, NTL, NTS>(src, dst, nvec);
                else if constexpr (FORM == kConvert)
                    wg_convert<GATHER, UNROLL, NTL, NTS>(src, dst, nvec, a.heads, a.tokens, a.row_vec);
                else
                    wg_convert_lds<GATHER, UNROLL, NTL, NTS>(src, dst, nvec, a.heads, a.tokens, a.row_vec, lds);
            }
        }
    }
}

// A launch of one class: the work list and table in device memory, every
// workgroup on its items.
template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void class_body(const CopyArgs &a)
{
    uint32_t g = blockIdx.x;
    if (a.xcd_remap) {
        // workgroups are dealt to the 8 XCDs round-robin; renumber them so that
        // each XCD takes one contiguous run of units per pass over the grid
        const uint32_t per = gridDim.x / kXcds;          // grid is a multiple of 8 here
        g = (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
    }
    if (a.tile_items)
        chunk_copy_tiles<GATHER, FORM, UNROLL, NTL, NTS>(a, (citem_t *)a.items, (cptr_t *)a.cache, g, gridDim.x);
    else
        chunk_copy_body<GATHER, FORM, UNROLL, NTL, NTS>(a, (citem_t *)a.items, (cptr_t *)a.cache, g, gridDim.x);
}

// One entry point per kind of source, so that traces and counters tell the
// zero-copy (host link) kernel, the HBM staging kernel and the kernel that
// empties / fills a copy-engine ring slot apart.  The body is the same.
template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void host_region_copy(CopyArgs a)
{
    class_body<GATHER, FORM, UNROLL, NTL, NTS>(a);
}

template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void staging_region_copy(CopyArgs a)
{
    class_body<GATHER, FORM, UNROLL, NTL, NTS>(a);
}

template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void ring_slot_copy(CopyArgs a)
{
    class_body<GATHER, FORM, UNROLL, NTL, NTS>(a);
}

template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void file_slot_copy(CopyArgs a)
{
    class_body<GATHER, FORM, UNROLL, NTL, NTS>(a);
}

// Both classes of a small call in one launch, the table and the items read
// from the kernel arguments (scalar loads, as from the work list).  The
// class split is uniform per workgroup.
template <bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void small_call_copy(SmallCallArgs f)
{
    // f is the kernel's only explicit argument, so it sits at offset 0 of the
    // kernel-argument segment; the table and the items are addressed there
    // (constant address space, scalar loads), never through a copy of f.
    typedef __attribute__((address_space(4))) const char cchar_t;
    cchar_t *words = (cchar_t *)__builtin_amdgcn_kernarg_segment_ptr() + offsetof(SmallCallArgs, words);
    cptr_t *table = (cptr_t *)words;
    citem_t *items = (citem_t *)(words + static_cast<uint64_t>(f.a.chunks) * sizeof(uint64_t));
    CopyArgs a = f.a;
    const bool host = blockIdx.x < f.grid_host;
    a.n_items = host ? f.n_host : f.a.n_items - f.n_host;
    chunk_copy_body<GATHER, FORM, UNROLL, NTL, NTS>(a, host ? items : items + f.n_host, table,
                                                    host ? blockIdx.x : blockIdx.x - f.grid_host,
                                                    host ? f.grid_host : gridDim.x - f.grid_host);
}

// Contiguous streaming copy over tiles of 256*UNROLL vectors (bandwidth probe).
template <int UNROLL, bool NTL, bool NTS>
__global__ __launch_bounds__(kThreads) void probe_copy_kernel(const v4u *__restrict__ src, v4u *__restrict__ dst,
                                                              uint64_t nvec)
{
    const uint64_t tile = static_cast<uint64_t>(kThreads) * UNROLL;
    const uint64_t tiles = (nvec + tile - 1) / tile;
    for (uint64_t t = blockIdx.x; t < tiles; t += gridDim.x) {
        const uint64_t base = t * tile;
        const uint64_t left = nvec - base;
        wg_copy<UNROLL, NTL, NTS>(src + base, dst + base, static_cast<uint32_t>(left < tile ? left : tile));
    }
}

// ---------------------------------------------------------------- static work-list scratch

// The work list of kv_pool_retrieve_noalloc lives here instead of in memory
// the library allocates.  Host code never passes this name to a kernel or a
// copy: on the host it is only a stand-in for the symbol, and its device
// address (one per GPU) comes from hipGetSymbolAddress in scratch_setup.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
ScratchDevice g_scratch[kMaxScratchDevices];
std::mutex g_scratch_setup;
}  // namespace

ScratchDevice &scratch_setup(int device)
{
    if (device < 0 || device >= kMaxScratchDevices)
        fail(KVP_ERR_INVALID, "device " + std::to_string(device) + " outside the scratch table");
    ScratchDevice &sd = g_scratch[device];
    std::lock_guard<std::mutex> lock(g_scratch_setup);
    if (sd.ready) return sd;
    void *dev = nullptr;
    check_hip(hipGetSymbolAddress(&dev, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!dev || (reinterpret_cast<uintptr_t>(dev) & 255))
        fail(KVP_ERR_HIP, "scratch symbol has no 256-byte aligned device address");
    void *host = nullptr;
    if (hipHostMalloc(&host, kScratchBytes, hipHostMallocDefault) != hipSuccess || !host) {
        clear_hip_error();
        fail(KVP_ERR_NOMEM, "pinned staging buffer of the static scratch");
    }
    hipEvent_t ev[2] = {nullptr, nullptr};
    for (auto &e : ev) {
        const hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (r != hipSuccess) {
            for (auto &x : ev)
                if (x) (void)hipEventDestroy(x);
            (void)hipHostFree(host);
            check_hip(r, "hipEventCreate");
        }
    }
    sd.dev = dev;
    sd.host = host;
    sd.staged = ev[0];
    sd.free = ev[1];
    sd.ready = true;
    return sd;
}

ScratchDevice &scratch_device(int device)
{
    if (device < 0 || device >= kMaxScratchDevices || !g_scratch[device].ready)
        fail(KVP_ERR_INVALID, "static scratch of device " + std::to_string(device) + " is not set up");
    return g_scratch[device];
}

// ---------------------------------------------------------------- host-side dispatch

constexpr uint32_t kClassSmall = 3;   // dispatch only: small_call_copy

__device__ __host__ inline const CopyArgs &geometry(const CopyArgs &a) { return a; }
__device__ __host__ inline const CopyArgs &geometry(const SmallCallArgs &f) { return f.a; }

template <uint32_t CLS, bool GATHER, int FORM, int UNROLL, bool NTL, bool NTS, class A>
static void launch_one(const A &a, dim3 g, size_t lds, hipStream_t s)
{
    if constexpr (CLS == kClassSmall)
        hipLaunchKernelGGL((small_call_copy<GATHER, FORM, UNROLL, NTL, NTS>), g, dim3(kThreads), lds, s, a);
    else if constexpr (CLS == KVP_CLASS_HOST)
        hipLaunchKernelGGL((host_region_copy<GATHER, FORM, UNROLL, NTL, NTS>), g, dim3(kThreads), lds, s, a);
    else if constexpr (CLS == KVP_CLASS_STAGING)
        hipLaunchKernelGGL((staging_region_copy<GATHER, FORM, UNROLL, NTL, NTS>), g, dim3(kThreads), lds, s, a);
    else if constexpr (CLS == kClassFile)
        hipLaunchKernelGGL((file_slot_copy<GATHER, FORM, UNROLL, NTL, NTS>), g, dim3(kThreads), lds, s, a);
    else
        hipLaunchKernelGGL((ring_slot_copy<GATHER, FORM, UNROLL, NTL, NTS>), g, dim3(kThreads), lds, s, a);
}

template <uint32_t CLS, bool GATHER, int FORM, int UNROLL, class A>
static hipError_t launch_form(const A &a, uint32_t grid, uint32_t flags, size_t lds, hipStream_t s)
{
    const bool ntl = flags & KVP_LAUNCH_NT_LOAD, nts = flags & KVP_LAUNCH_NT_STORE;
    const dim3 g(grid);
    if (ntl && nts)
        launch_one<CLS, GATHER, FORM, UNROLL, true, true>(a, g, lds, s);
    else if (ntl)
        launch_one<CLS, GATHER, FORM, UNROLL, true, false>(a, g, lds, s);
    else if (nts)
        launch_one<CLS, GATHER, FORM, UNROLL, false, true>(a, g, lds, s);
    else
        launch_one<CLS, GATHER, FORM, UNROLL, false, false>(a, g, lds, s);
    return hipGetLastError();
}

template <uint32_t CLS, bool GATHER, int FORM, class A>
static hipError_t launch_unroll(const A &a, uint32_t grid, uint32_t flags, size_t lds, hipStream_t s)
{
    // enough 16-byte loads in flight per lane to cover the whole unit, up to 8
    const CopyArgs &geo = geometry(a);
    const uint64_t per_lane = (geo.chunk_bytes / geo.parts / 16 + kThreads - 1) / kThreads;
    if (per_lane >= 8) return launch_form<CLS, GATHER, FORM, 8>(a, grid, flags, lds, s);
    if (per_lane >= 4) return launch_form<CLS, GATHER, FORM, 4>(a, grid, flags, lds, s);
    if (per_lane >= 2) return launch_form<CLS, GATHER, FORM, 2>(a, grid, flags, lds, s);
    return launch_form<CLS, GATHER, FORM, 1>(a, grid, flags, lds, s);
}

template <uint32_t CLS, bool GATHER, class A>
static hipError_t launch_dir(const A &a, uint32_t grid, uint32_t flags, hipStream_t s)
{
    const CopyArgs &geo = geometry(a);
    if (geo.layout == 0) return launch_unroll<CLS, GATHER, kPlain>(a, grid, flags, 0, s);
    if ((flags & KVP_LAUNCH_LDS) && geo.chunk_bytes <= kMaxLdsChunk)
        return launch_unroll<CLS, GATHER, kConvertLds>(a, grid, flags, geo.chunk_bytes, s);
    return launch_unroll<CLS, GATHER, kConvert>(a, grid, flags, 0, s);
}

hipError_t launch_chunk_copy(const CopyArgs &args, uint32_t cls, bool gather, uint32_t grid, uint32_t flags,
                             hipStream_t s)
{
    if (args.n_items == 0) return hipSuccess;
    CopyArgs a = args;
    // halves of a plain chunk are independent contiguous copies
    a.parts = (a.layout == 0 && (flags & KVP_LAUNCH_SPLIT2) && a.chunk_bytes % 32 == 0) ? 2u : 1u;
    const uint64_t units = static_cast<uint64_t>(a.n_items) * a.chunks * a.parts;
    if (grid > units) grid = static_cast<uint32_t>(units);
    if (grid == 0) grid = 1;
    // the XCD renumbering is a permutation of [0, grid) only for multiples of 8
    a.xcd_remap = (flags & KVP_LAUNCH_XCD) && grid % kXcds == 0 ? 1u : 0u;
    a.chunk_major = (flags & KVP_LAUNCH_CHUNK_MAJOR) ? 1u : 0u;
    a.tile_items = (flags & KVP_LAUNCH_TILE) ? kTileItems : 0u;
    if (a.tile_items) {   // a grid of at most one workgroup per tile
        const uint64_t tiles = (static_cast<uint64_t>(a.n_items) + kTileItems - 1) / kTileItems * a.chunks;
        if (grid > tiles) grid = static_cast<uint32_t>(tiles);
        a.xcd_remap = (flags & KVP_LAUNCH_XCD) && grid % kXcds == 0 ? 1u : 0u;
    }
    if (cls == KVP_CLASS_HOST)
        return gather ? launch_dir<KVP_CLASS_HOST, true>(a, grid, flags, s)
                      : launch_dir<KVP_CLASS_HOST, false>(a, grid, flags, s);
    if (cls == KVP_CLASS_STAGING)
        return gather ? launch_dir<KVP_CLASS_STAGING, true>(a, grid, flags, s)
                      : launch_dir<KVP_CLASS_STAGING, false>(a, grid, flags, s);
    if (cls == kClassFile)
        return gather ? launch_dir<kClassFile, true>(a, grid, flags, s) : launch_dir<kClassFile, false>(a, grid, flags, s);
    return gather ? launch_dir<kClassRing, true>(a, grid, flags, s) : launch_dir<kClassRing, false>(a, grid, flags, s);
}

hipError_t launch_small_call(SmallCallArgs &f, bool gather, uint32_t grid_host, uint32_t grid_staging,
                             uint32_t flags, hipStream_t s)
{
    CopyArgs &a = f.a;
    if (a.n_items == 0) return hipSuccess;
    a.parts = (a.layout == 0 && (flags & KVP_LAUNCH_SPLIT2) && a.chunk_bytes % 32 == 0) ? 2u : 1u;
    a.xcd_remap = 0;
    a.chunk_major = 0;
    a.tile_items = 0;
    auto cap = [&](uint32_t grid, uint32_t n) {
        const uint64_t units = static_cast<uint64_t>(n) * a.chunks * a.parts;
        if (n == 0) return 0u;
        return grid == 0 ? 1u : static_cast<uint32_t>(grid < units ? grid : units);
    };
    f.grid_host = cap(grid_host, f.n_host);
    const uint32_t grid = f.grid_host + cap(grid_staging, a.n_items - f.n_host);
    return gather ? launch_dir<kClassSmall, true>(f, grid, flags, s) : launch_dir<kClassSmall, false>(f, grid, flags, s);
}

hipError_t launch_probe_copy(void *dst, const void *src, uint64_t bytes, uint32_t grid, uint32_t flags,
                             hipStream_t s)
{
    const uint64_t nvec = bytes / 16;
    if (nvec == 0) return hipSuccess;
    const bool split = flags & KVP_LAUNCH_SPLIT2;
    const uint64_t tiles = (nvec + kThreads * (split ? 4 : 8) - 1) / (kThreads * (split ? 4 : 8));
    if (grid == 0) grid = 2048;
    if (grid > tiles) grid = static_cast<uint32_t>(tiles);
    const bool ntl = flags & KVP_LAUNCH_NT_LOAD, nts = flags & KVP_LAUNCH_NT_STORE;
    const v4u *sp = static_cast<const v4u *>(src);
    v4u *dp = static_cast<v4u *>(dst);
    dim3 g(grid), b(kThreads);
    if (split) {
        if (ntl && nts)
            hipLaunchKernelGGL((probe_copy_kernel<4, true, true>), g, b, 0, s, sp, dp, nvec);
        else if (ntl)
            hipLaunchKernelGGL((probe_copy_kernel<4, true, false>), g, b, 0, s, sp, dp, nvec);
        else if (nts)
            hipLaunchKernelGGL((probe_copy_kernel<4, false, true>), g, b, 0, s, sp, dp, nvec);
        else
            hipLaunchKernelGGL((probe_copy_kernel<4, false, false>), g, b, 0, s, sp, dp, nvec);
        return hipGetLastError();
    }
    if (ntl && nts)
        hipLaunchKernelGGL((probe_copy_kernel<8, true, true>), g, b, 0, s, sp, dp, nvec);
    else if (ntl)
        hipLaunchKernelGGL((probe_copy_kernel<8, true, false>), g, b, 0, s, sp, dp, nvec);
    else if (nts)
        hipLaunchKernelGGL((probe_copy_kernel<8, false, true>), g, b, 0, s, sp, dp, nvec);
    else
        hipLaunchKernelGGL((probe_copy_kernel<8, false, false>), g, b, 0, s, sp, dp, nvec);
    return hipGetLastError();
}

}  // namespace kvp

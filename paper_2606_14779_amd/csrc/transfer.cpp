// Store / retrieve engine of the KV pool.
//
// Retrieval follows Sec. 4.3 of the paper: look every block up, group the
// blocks by pool device, and read all devices in parallel.  Here the groups
// are the two region classes -- pinned host regions, read by a zero-copy
// kernel over the host link (or by the copy engines through an HBM ring), and
// HBM staging regions, read by an HBM gather kernel.  "In parallel" means the
// staging kernel is forked onto the pool's internal stream while the host
// kernel runs on the caller's stream, and the two are joined again on the
// caller's stream, so the caller sees one stream-ordered operation.  The store
// (Alg. 1, offload) is the same path in the other direction.  The per-call
// work list (the engine-buffer pointers of the moved chunks, then one 16-byte
// item per block) travels in the kernel arguments of a single launch when it
// is small enough; otherwise it is written to a pinned buffer and uploaded
// with one asynchronous copy.  Those buffers come from a ring guarded by
// events, so a call only blocks when the ring wraps onto work that is still
// running.

#include <algorithm>

#include <unordered_map>

#include "internal.hpp"

namespace kvp {

namespace {

constexpr size_t kSlotMin = 64 * 1024;   // smallest work-list buffer
// Staging-class bytes below which the HBM kernel runs on the caller's stream
// ahead of the host-class kernel instead of being forked: forking costs about
// 25 us of host time per call, more than such a kernel takes (32 MiB read and
// written at ~2.5 TB/s copied: ~13 us).
constexpr uint64_t kForkMinBytes = 32ull << 20;
// Host-class retrieve workgroups while a host-class store of this pool is in
// flight.  Under two-way traffic the reads need more in flight: a 128K-token
// LLaMA-shaped store and retrieve at once took 264.6 ms with 48 against
// 320 ms with the 12 that a lone retrieve wants (which, beside HBM-bound
// work, loses with more).
constexpr uint32_t kDuplexReadGrid = 48;

// The live allocation holding the block at map entry e, or an error.
const Allocation *resolve(const Pool &p, const kvp_loc &e, uint32_t b, const Allocation *hint)
{
    const uint32_t N = static_cast<uint32_t>(p.regions.size());
    if (e.region >= N)
        fail(KVP_ERR_INVALID, "map entry " + std::to_string(b) + ": region " + std::to_string(e.region) +
                                  " out of range");
    const Region &r = p.regions[e.region];
    if (e.offset % 16 != 0 || e.offset > r.capacity || r.capacity - e.offset < p.block_bytes)
        fail(KVP_ERR_INVALID, "map entry " + std::to_string(b) + ": offset outside region");
    const Allocation *a = hint;
    if (!(a && a->region == e.region && e.offset >= a->base && e.offset < a->base + a->blocks * p.block_bytes)) {
        auto it = r.live.upper_bound(e.offset);
        if (it == r.live.begin()) fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": no live placement there");
        a = std::prev(it)->second;
        if (e.offset >= a->base + a->blocks * p.block_bytes)
            fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": no live placement there");
    }
    if ((e.offset - a->base) % p.block_bytes != 0 || a->gen != e.gen)
        fail(KVP_ERR_STALE, "map entry " + std::to_string(b) + ": stale generation or block boundary");
    return a;
}

constexpr size_t kMaxTimedCalls = 4096;

hipEvent_t timing_event(Pool &p)
{
    if (!p.spare.empty()) {
        hipEvent_t e = p.spare.back();
        p.spare.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    check_hip(hipEventCreate(&e), "hipEventCreate");
    return e;
}

Slot &acquire_slot(Pool &p, size_t bytes)
{
    Slot &s = p.ring[p.ring_next];
    p.ring_next = (p.ring_next + 1) % static_cast<uint32_t>(p.ring.size());
    if (s.pending) {
        check_hip(hipEventSynchronize(s.done), "hipEventSynchronize");
        s.pending = false;
    }
    if (s.cap < bytes) {
        free_slot(s);
        const size_t cap = round_up(std::max(bytes, kSlotMin), kSlotMin);
        void *h = nullptr, *d = nullptr;
        if (hipHostMalloc(&h, cap, hipHostMallocDefault) != hipSuccess || !h) {
            clear_hip_error();
            fail(KVP_ERR_NOMEM, "work-list pinned buffer");
        }
        if (hipMalloc(&d, cap) != hipSuccess || !d) {
            clear_hip_error();
            (void)hipHostFree(h);
            fail(KVP_ERR_NOMEM, "work-list device buffer");
        }
        s.host = h;
        s.dev = d;
        s.cap = cap;
    }
    return s;
}

// The file regions' blocks of a call, batch by batch through the pinned ring
// (see fileio.cpp): a retrieve reads a batch's spans by the regions' workers,
// then moves the slot to the engine cache by a kernel on stream `sf`; a store
// fills the slot by a kernel, waits for it, and has the workers write the
// spans while the next batch's kernel runs.  A slot is refilled only after
// its previous kernel and its previous reads or writes are done.  On return
// every read or write is done; on a failure the workers are drained first.
void run_file_batches(Pool &p, bool gather, const std::vector<FileBatch> &batches,
                      const std::vector<FileSpan> &spans, const CopyArgs &a, const LaunchCfg &lc, hipStream_t sf)
{
    auto submit = [&](const FileBatch &bt, bool write) {
        char *slot = p.file_ring + static_cast<uint64_t>(bt.ring) * p.file_slot_bytes;
        for (size_t i = bt.span0; i < bt.span0 + bt.spans; ++i) {
            const FileSpan &sp = spans[i];
            const Region &r = p.regions[sp.region];
            p.workers->submit(r.worker, IoJob{r.fd, write, sp.file_off, sp.len, slot + sp.slot_off, &p.file_io[bt.ring]});
        }
    };
    auto kernel = [&](const FileBatch &bt) {
        CopyArgs k = a;
        k.items = a.items + bt.first;
        k.n_items = bt.n;
        check_hip(launch_chunk_copy(k, kClassFile, gather, lc.grid, lc.flags, sf), "kernel launch");
        check_hip(hipEventRecord(p.file_free[bt.ring], sf), "hipEventRecord");
        p.file_free_rec[bt.ring] = true;
    };
    // the slot is free: its reads or writes and its kernel are done
    auto slot_free = [&](const FileBatch &bt) {
        io_wait(p.file_io[bt.ring]);
        if (p.file_free_rec[bt.ring]) check_hip(hipEventSynchronize(p.file_free[bt.ring]), "hipEventSynchronize");
    };
    try {
        if (gather) {
            // read ahead: the next batch's reads are queued behind this one's (into the
            // other slot) before this one is waited for, so each worker moves on as soon
            // as its own part of a batch is read
            if (!batches.empty()) {
                slot_free(batches[0]);
                submit(batches[0], false);
            }
            for (size_t i = 0; i < batches.size(); ++i) {
                if (i + 1 < batches.size()) {
                    slot_free(batches[i + 1]);
                    submit(batches[i + 1], false);
                }
                io_wait(p.file_io[batches[i].ring]);
                kernel(batches[i]);
            }
        } else {
            for (const FileBatch &bt : batches) {
                slot_free(bt);
                kernel(bt);
                check_hip(hipEventSynchronize(p.file_free[bt.ring]), "hipEventSynchronize");
                submit(bt, true);
            }
        }
        for (auto &g : p.file_io) io_wait(g);
    } catch (...) {
        for (auto &g : p.file_io) io_drain(g);
        p.file_next = static_cast<uint32_t>((p.file_next + batches.size()) % kFileSlots);
        throw;
    }
    p.file_next = static_cast<uint32_t>((p.file_next + batches.size()) % kFileSlots);
}

}  // namespace

// Wait for every recorded call, optionally summarise it, and recycle its events.
void drain_timed(Pool &p, kvp_timing_summary *sum)
{
    kvp_timing_summary s{};
    s.host_ms_min = s.staging_ms_min = -1.f;
    s.host_ms_max = s.staging_ms_max = -1.f;
    for (auto &tc : p.timed) {
        ++s.calls;
        for (int c = 0; c < 2; ++c) {
            if (!tc.ran[c]) continue;
            check_hip(hipEventSynchronize(tc.t1[c]), "hipEventSynchronize");
            float ms = 0.f;
            check_hip(hipEventElapsedTime(&ms, tc.t0[c], tc.t1[c]), "hipEventElapsedTime");
            float &mn = c == 0 ? s.host_ms_min : s.staging_ms_min;
            float &mx = c == 0 ? s.host_ms_max : s.staging_ms_max;
            (c == 0 ? s.host_ms_sum : s.staging_ms_sum) += ms;
            (c == 0 ? s.host_calls : s.staging_calls) += 1;
            mn = mn < 0.f ? ms : std::min(mn, ms);
            mx = std::max(mx, ms);
        }
    }
    for (auto &tc : p.timed)
        for (int c = 0; c < 2; ++c) {
            if (tc.t0[c]) p.spare.push_back(tc.t0[c]);
            if (tc.t1[c]) p.spare.push_back(tc.t1[c]);
        }
    p.timed.clear();
    if (sum) *sum = s;
}

// noalloc (retrieve only): the work list goes through the device's static
// scratch instead of the upload ring, and the host class always takes the
// zero-copy kernel (the copy-engine ring is memory of its own); no small-call
// launch and no timing, so that the call makes no allocation and creates no
// HIP object.
void pool_transfer(Pool &p, const kvp_loc *map, uint32_t n_blocks, const int32_t *table, uint32_t num_slots,
                   uint32_t layer_begin, uint32_t layer_end, void *const *k_layers, void *const *v_layers,
                   void *stream_ptr, bool gather, bool noalloc)
{
    if (p.placement_only) fail(KVP_ERR_INVALID, "placement-only pool has no memory to copy");
    if (n_blocks && (!map || !table)) fail(KVP_ERR_INVALID, "null map or block table");
    const uint32_t L = p.spec.num_layers;
    if (layer_begin >= layer_end || layer_end > L)
        fail(KVP_ERR_INVALID, "layer range [" + std::to_string(layer_begin) + ", " + std::to_string(layer_end) +
                                  ") not inside [0, " + std::to_string(L) + ")");
    if (!k_layers || !v_layers) fail(KVP_ERR_INVALID, "null layer pointer array");
    for (uint32_t l = layer_begin; l < layer_end; ++l) {
        const uintptr_t k = reinterpret_cast<uintptr_t>(k_layers[l]), v = reinterpret_cast<uintptr_t>(v_layers[l]);
        if (!k || !v || (k & 15) || (v & 15))
            fail(KVP_ERR_INVALID, "layer " + std::to_string(l) + ": null or unaligned cache pointer");
    }
    // a kernel's units (blocks x 2L chunks x at most 2 parts) and its workgroup stride (at most 2^20)
    // are summed in 32 bits: at most 2^31 units keeps that sum from wrapping
    if (static_cast<uint64_t>(n_blocks) * 4 * L > (1ull << 31)) fail(KVP_ERR_INVALID, "request too large");

    std::lock_guard<std::mutex> lock(p.mu);
    DeviceScope dev(p.device);
    const uint32_t op = gather ? KVP_OP_RETRIEVE : KVP_OP_STORE;
    if (noalloc && !gather) fail(KVP_ERR_INVALID, "the static-scratch path is a retrieve");
    const bool sdma = !noalloc && (p.launch[KVP_CLASS_HOST][op].flags & KVP_LAUNCH_SDMA) != 0;
    if (sdma && !p.bounce)   // only after a kv_pool_set_copy_ring that could not allocate
        fail(KVP_ERR_NOMEM, "copy-engine ring not allocated: set a smaller ring or clear KVP_LAUNCH_SDMA");

    // GLT-resolved locations, grouped by region class (Sec. 4.3)
    std::vector<CopyItem> items[2];
    std::vector<HostBlock> host_blocks;   // copy-engine transport: placed in ring slots below
    std::vector<HostBlock> file_blocks;   // file regions: placed in the file ring's slots below
    std::vector<RequestRec *> touched;
    const uint64_t epoch = ++p.call_epoch;
    // No two present entries may write the same place: a destination slot on
    // retrieve, a pool block on store.  One pass over bitmaps -- of the
    // destination slots, or of the blocks of each allocation a store touches
    // (the block index within its allocation is exact after resolve) -- with
    // sorted slots only for a retrieve into far more slots than it moves.
    std::vector<uint64_t> seen;
    const bool slot_bits = gather && num_slots <= std::max<uint64_t>(64ull * n_blocks, 1ull << 16);
    if (slot_bits) seen.assign((num_slots + 63) / 64, 0);
    std::vector<uint32_t> wide_slots;
    std::unordered_map<const Allocation *, uint64_t> alloc_word;   // store: first bitmap word of an allocation
    std::vector<uint64_t> region_word(p.regions.size(), 0);        // store: that of each region's hint
    bool dup = false;
    uint64_t dup_slot = 0;
    auto mark = [&](uint64_t bit) {
        uint64_t &w = seen[bit >> 6];
        const uint64_t m = 1ull << (bit & 63);
        if ((w & m) && !dup) {
            dup = true;
            dup_slot = bit;
        }
        w |= m;
    };
    // one hint per region: a request's blocks in a region share one range,
    // while consecutive blocks of a striped map alternate between regions
    std::vector<const Allocation *> hints(p.regions.size(), nullptr);
    for (uint32_t b = 0; b < n_blocks; ++b) {
        const kvp_loc &e = map[b];
        if (e.region == KVP_ABSENT) continue;
        const Allocation *hint = resolve(p, e, b, e.region < hints.size() ? hints[e.region] : nullptr);
        const bool new_hint = hint != hints[e.region];
        hints[e.region] = hint;
        const int32_t slot = table[b];
        if (slot < 0 || static_cast<uint32_t>(slot) >= num_slots)
            fail(KVP_ERR_INVALID, "block table entry " + std::to_string(b) + " = " + std::to_string(slot) +
                                      " outside [0, " + std::to_string(num_slots) + ")");
        if (slot_bits) {
            mark(static_cast<uint64_t>(slot));
        } else if (gather) {
            wide_slots.push_back(static_cast<uint32_t>(slot));
        } else {
            if (new_hint) {
                auto it = alloc_word.find(hint);
                if (it == alloc_word.end()) {
                    it = alloc_word.emplace(hint, seen.size()).first;
                    seen.resize(seen.size() + (hint->blocks + 63) / 64, 0);
                }
                region_word[e.region] = it->second;
            }
            mark(region_word[e.region] * 64 + (e.offset - hint->base) / p.block_bytes);
        }
        if (new_hint && hint->owner->call_mark != epoch) {   // each request listed once
            hint->owner->call_mark = epoch;
            touched.push_back(hint->owner);
        }
        const Region &r = p.regions[e.region];
        if (r.desc.type == KVP_REGION_FILE) {
            if (noalloc)
                fail(KVP_ERR_INVALID, "map entry " + std::to_string(b) + ": the allocation-free call reads no file region");
            file_blocks.push_back(HostBlock{e.region, e.offset, static_cast<uint32_t>(slot)});
        } else {
            const uint32_t cls = r.desc.type == KVP_REGION_HOST ? KVP_CLASS_HOST : KVP_CLASS_STAGING;
            if (cls == KVP_CLASS_HOST && sdma)
                host_blocks.push_back(HostBlock{e.region, e.offset, static_cast<uint32_t>(slot)});
            else
                items[cls].push_back(
                    CopyItem{reinterpret_cast<uint64_t>(r.dev) + e.offset, static_cast<uint32_t>(slot), 0u});
        }
    }
    if (!wide_slots.empty()) {
        std::sort(wide_slots.begin(), wide_slots.end());
        auto d = std::adjacent_find(wide_slots.begin(), wide_slots.end());
        if (d != wide_slots.end()) {
            dup = true;
            dup_slot = *d;
        }
    }
    if (dup)
        fail(KVP_ERR_INVALID, gather ? "destination slot " + std::to_string(dup_slot) + " named twice"
                                     : std::string("two map entries name the same pool block"));
    const uint64_t width = 2ull * (layer_end - layer_begin) * p.chunk_bytes;   // bytes moved per block
    const uint64_t skip = 2ull * layer_begin * p.chunk_bytes;
    std::vector<LinkRun> runs;
    std::vector<Batch> batches;
    if (!host_blocks.empty()) {
        const RingGeometry g{reinterpret_cast<uint64_t>(p.bounce), p.bounce_slot_bytes, kBounceSlots, p.bounce_next,
                             p.block_bytes, p.chunk_bytes};
        plan_bounce(g, host_blocks, width, 2 * layer_begin, items[KVP_CLASS_HOST], runs, batches);
    }

    std::vector<CopyItem> file_items;
    std::vector<FileSpan> spans;
    std::vector<FileBatch> file_batches;
    if (!file_blocks.empty()) {
        if (!p.file_ring || p.file_slot_bytes < p.block_bytes)   // only after a kv_pool_set_file_ring that could not allocate
            fail(KVP_ERR_NOMEM, "file-region ring not allocated: set a smaller one with kv_pool_set_file_ring");
        const FileGeometry fg{p.file_ring_dev, p.file_slot_bytes, kFileSlots, p.file_next, p.block_bytes,
                              p.chunk_bytes};
        plan_file(fg, file_blocks, skip, width, 2 * layer_begin, file_items, spans, file_batches);
    }

    const size_t n_items = items[0].size() + items[1].size() + file_items.size();
    const size_t ptr_bytes = round_up(static_cast<size_t>(2 * (layer_end - layer_begin)) * sizeof(uint64_t), 16);
    const size_t list_bytes = ptr_bytes + n_items * sizeof(CopyItem);
    if (noalloc && list_bytes > kScratchBytes)
        fail(KVP_ERR_INVALID, "work list of " + std::to_string(list_bytes) + " bytes (" + std::to_string(n_items) +
                                  " blocks) exceeds the static scratch of " + std::to_string(kScratchBytes) + " bytes");
    if (p.timing && !noalloc) {
        if (p.timed.size() >= kMaxTimedCalls) drain_timed(p, nullptr);   // bound the history
        TimedCall tc;
        for (int c = 0; c < 2; ++c) {
            tc.blocks[c] = static_cast<uint32_t>(items[c].size());
            if (!items[c].empty()) {
                tc.t0[c] = timing_event(p);
                tc.t1[c] = timing_event(p);
            }
        }
        p.timed.push_back(tc);
    }
    if (n_items == 0) return;

    hipStream_t s = static_cast<hipStream_t>(stream_ptr);
    // ordering with earlier work on the same requests from any stream:
    // retrieve after store (read after write), store after store/retrieve
    for (RequestRec *rec : touched) {
        if (gather && rec->stored_rec) check_hip(hipStreamWaitEvent(s, rec->stored, 0), "hipStreamWaitEvent");
        if (!gather && rec->busy_rec) check_hip(hipStreamWaitEvent(s, rec->busy, 0), "hipStreamWaitEvent");
    }
    // busy must cover every call still touching the request, not only this
    // one: two retrieves of a request may run on different streams at once,
    // and release, destroy and a later store wait on busy alone.  So when
    // the previous record was on another stream, the caller's stream first
    // waits for it (after this call's kernels, so only later work on the
    // stream is held back), and the new record covers both.
    auto mark_requests = [&] {
        for (RequestRec *rec : touched) {
            if (rec->busy_rec && rec->busy_stream != s)
                check_hip(hipStreamWaitEvent(s, rec->busy, 0), "hipStreamWaitEvent");
            check_hip(hipEventRecord(rec->busy, s), "hipEventRecord");
            rec->busy_rec = true;
            rec->busy_stream = s;
            if (!gather) {
                check_hip(hipEventRecord(rec->stored, s), "hipEventRecord");
                rec->stored_rec = true;
            }
        }
    };
    // one host-class kernel on the link at a time, in enqueue order: two of
    // them would only share its bandwidth and both end late
    auto take_link = [&] {
        if (p.link_rec[op] && p.link_stream[op] != s)
            check_hip(hipStreamWaitEvent(s, p.link_done[op], 0), "hipStreamWaitEvent");
    };
    auto hand_back_link = [&] {
        check_hip(hipEventRecord(p.link_done[op], s), "hipEventRecord");
        p.link_rec[op] = true;
        p.link_stream[op] = s;
    };

    const uint32_t chunks = 2 * (layer_end - layer_begin);
    CopyArgs geo = {};
    geo.chunks = chunks;
    geo.chunk0 = 2 * layer_begin;
    geo.parts = 1;
    geo.chunk_bytes = p.chunk_bytes;
    geo.heads = p.spec.num_kv_heads;
    geo.tokens = p.spec.block_size;
    geo.row_vec = static_cast<uint32_t>(static_cast<uint64_t>(p.spec.head_dim) * p.spec.elem_bytes / 16);
    geo.layout = p.spec.pool_layout;
    auto fill_table = [&](uint64_t *t) {   // engine buffer of moved chunk k
        for (uint32_t k = 0; k < chunks; ++k) {
            const uint32_t l = layer_begin + k / 2;
            t[k] = reinterpret_cast<uint64_t>(k % 2 ? v_layers[l] : k_layers[l]);
        }
    };

    // the internal stream takes work only for enough staging bytes or for ring batches
    const bool fork_staging = batches.empty() && items[KVP_CLASS_STAGING].size() * width >= kForkMinBytes;
    const LaunchCfg &ls = p.launch[KVP_CLASS_STAGING][op];
    LaunchCfg lh = p.launch[KVP_CLASS_HOST][op];
    const bool host = !items[KVP_CLASS_HOST].empty();
    if (gather && host && lh.default_grid && p.link_rec[KVP_OP_STORE] && lh.grid < kDuplexReadGrid &&
        hipPeekAtLastError() == hipSuccess) {   // never clear an error the caller has yet to read
        // a store's host-class kernel not yet finished: the link carries traffic both ways
        const hipError_t q = hipEventQuery(p.link_done[KVP_OP_STORE]);
        if (q == hipErrorNotReady) {
            (void)hipGetLastError();   // "not ready" is the answer, not an error to leave behind
            lh.grid = kDuplexReadGrid;
        } else {
            check_hip(q, "hipEventQuery");
        }
    }
    if (!noalloc && batches.empty() && file_batches.empty() && !p.timing &&
        !((lh.flags | ls.flags) & KVP_LAUNCH_UPLOAD) &&
        chunks + 2 * n_items <= kInlineWords) {
        // Small call: table and items in the kernel arguments, both classes in
        // one launch in the host class's copy form (the link-bound part; the
        // form does not change what is written)
        SmallCallArgs f = {};
        f.a = geo;
        f.a.n_items = static_cast<uint32_t>(n_items);
        f.n_host = static_cast<uint32_t>(items[KVP_CLASS_HOST].size());
        fill_table(f.words);
        auto *list = reinterpret_cast<CopyItem *>(f.words + chunks);
        std::copy(items[0].begin(), items[0].end(), list);
        std::copy(items[1].begin(), items[1].end(), list + items[0].size());
        if (host) take_link();
        check_hip(launch_small_call(f, gather, lh.grid, ls.grid, host ? lh.flags : ls.flags, s), "kernel launch");
        if (host) hand_back_link();
        mark_requests();
        return;
    }

    // work list: [chunks cache pointers][host items][staging items][file items], in a
    // ring slot of the pool, or in the device's static scratch (noalloc)
    const size_t bytes = list_bytes;
    Slot *slot = nullptr;
    ScratchDevice *sd = nullptr;
    std::unique_lock<std::mutex> scratch_lock;
    void *host_list = nullptr, *dev_base = nullptr;
    if (noalloc) {
        sd = &scratch_device(p.device);   // set up when the pool was created
        scratch_lock = std::unique_lock<std::mutex>(sd->mu);
        // the pinned buffer is rewritten only after the previous upload from it
        if (sd->staged_rec) check_hip(hipEventSynchronize(sd->staged), "hipEventSynchronize");
        host_list = sd->host;
        dev_base = sd->dev;
    } else {
        slot = &acquire_slot(p, bytes);
        host_list = slot->host;
        dev_base = slot->dev;
    }
    fill_table(static_cast<uint64_t *>(host_list));
    auto *list = reinterpret_cast<CopyItem *>(static_cast<char *>(host_list) + ptr_bytes);
    std::copy(items[0].begin(), items[0].end(), list);
    std::copy(items[1].begin(), items[1].end(), list + items[0].size());
    std::copy(file_items.begin(), file_items.end(), list + items[0].size() + items[1].size());

    // With earlier work still running on the caller's stream (calls issued
    // back to back, e.g. one per layer), the upload goes on the pool's stream:
    // it is done while the previous call's host-link kernel still runs, where
    // in line it would leave the link idle between the two kernels (74 us per
    // layer call, against 36.5 us).  On an idle caller stream it stays in
    // line, which costs less host time (9.5 against 26 us per call: the wait
    // on a pending event from another stream is what costs).  The slot is free
    // on the device: it was reclaimed only after the last call that read it.
    bool ahead = false;
    if (!noalloc && hipPeekAtLastError() == hipSuccess) {   // never clear an error the caller has yet to read
        const hipError_t q = hipStreamQuery(s);
        if (q == hipErrorNotReady) {
            (void)hipGetLastError();   // "not ready" is the answer, not an error to leave behind
            ahead = true;
        } else {
            check_hip(q, "hipStreamQuery");
        }
    }
    if (noalloc) {
        // the array is overwritten only after the previous call's kernels
        // (from any pool, on any stream) have read it
        if (sd->free_rec) check_hip(hipStreamWaitEvent(s, sd->free, 0), "hipStreamWaitEvent");
        check_hip(hipMemcpyAsync(dev_base, host_list, bytes, hipMemcpyHostToDevice, s), "hipMemcpyAsync");
        check_hip(hipEventRecord(sd->staged, s), "hipEventRecord");
        sd->staged_rec = true;
    } else {
        check_hip(hipMemcpyAsync(dev_base, host_list, bytes, hipMemcpyHostToDevice, ahead ? p.s_stage : s),
                  "hipMemcpyAsync");
        slot->pending = true;  // from here on the slot is in use even if a launch fails
    }
    // After a failure once the work list is on its way (a file read or write
    // that fails, a launch or copy the runtime refuses), whatever was enqueued
    // still runs and reads the work list.  So the caller's stream joins the
    // pool's stream, and the work list's and the requests' completion events
    // are recorded after all of it before the error is returned: a later call
    // cannot rewrite the list under those kernels, and release waits for them.
    // Nothing here throws, so the first error is the one reported.
    auto settle = [&]() noexcept {
        (void)hipEventRecord(p.stage_done, p.s_stage);
        (void)hipStreamWaitEvent(s, p.stage_done, 0);
        if (noalloc) {
            if (hipEventRecord(sd->free, s) == hipSuccess) sd->free_rec = true;
        } else {
            (void)hipEventRecord(slot->done, s);
        }
        for (RequestRec *rec : touched) {
            if (rec->busy_rec && rec->busy_stream != s) (void)hipStreamWaitEvent(s, rec->busy, 0);
            if (hipEventRecord(rec->busy, s) == hipSuccess) {
                rec->busy_rec = true;
                rec->busy_stream = s;
            }
            if (!gather && hipEventRecord(rec->stored, s) == hipSuccess) rec->stored_rec = true;
        }
        clear_hip_error();
    };
    auto enqueue = [&] {
        if (ahead) {
            check_hip(hipEventRecord(p.uploaded, p.s_stage), "hipEventRecord");
            check_hip(hipStreamWaitEvent(s, p.uploaded, 0), "hipStreamWaitEvent");
        }
        if (fork_staging || !batches.empty() || !file_batches.empty())
            check_hip(hipEventRecord(p.fork, s), "hipEventRecord");

        const CopyItem *dev_list = reinterpret_cast<const CopyItem *>(static_cast<char *>(dev_base) + ptr_bytes);
        // Staging class forked onto the internal stream first, then the host
        // class on the caller's stream itself; the caller's stream then waits for
        // the staging kernel.  One extra stream keeps the pool within the few
        // hardware queues a process gets, so caller streams (e.g. compute
        // overlapping a layerwise retrieve) are not serialised behind it.
        size_t first = 0;
        CopyArgs args[2] = {geo, geo};
        for (uint32_t c = 0; c < 2; ++c) {
            args[c].items = dev_list + first;
            args[c].cache = static_cast<const uint64_t *>(dev_base);
            args[c].n_items = static_cast<uint32_t>(items[c].size());
            first += items[c].size();
        }
        TimedCall *tc = p.timing && !noalloc ? &p.timed.back() : nullptr;
        auto launch = [&](uint32_t c, hipStream_t st) {
            const LaunchCfg &lc = c == KVP_CLASS_HOST ? lh : p.launch[c][op];
            if (tc) check_hip(hipEventRecord(tc->t0[c], st), "hipEventRecord");
            check_hip(launch_chunk_copy(args[c], c, gather, lc.grid, lc.flags, st), "kernel launch");
            if (tc) {
                check_hip(hipEventRecord(tc->t1[c], st), "hipEventRecord");
                tc->ran[c] = true;
            }
        };
        const bool staging = !items[KVP_CLASS_STAGING].empty();
        if (batches.empty()) {
            if (fork_staging) {
                check_hip(hipStreamWaitEvent(p.s_stage, p.fork, 0), "hipStreamWaitEvent");
                launch(KVP_CLASS_STAGING, p.s_stage);
                check_hip(hipEventRecord(p.stage_done, p.s_stage), "hipEventRecord");
            } else if (staging) {
                launch(KVP_CLASS_STAGING, s);   // small: in order on the caller's stream
            }
            if (host) {
                take_link();
                launch(KVP_CLASS_HOST, s);
                hand_back_link();
            }
            if (fork_staging) check_hip(hipStreamWaitEvent(s, p.stage_done, 0), "hipStreamWaitEvent");
        } else {
            // Copy-engine transport: the host-link copies take the internal
            // stream (no stream beyond the kernel path's two) and every kernel
            // runs on the caller's stream -- the staging class first, then one
            // ring-slot kernel per batch.  A slot is refilled only after its
            // previous contents were consumed (by any call, either op).
            if (staging) launch(KVP_CLASS_STAGING, s);
            const LaunchCfg &lc = p.launch[KVP_CLASS_STAGING][op];
            const hipMemcpyKind kind = gather ? hipMemcpyHostToDevice : hipMemcpyDeviceToHost;
            hipStream_t sc = p.s_stage;
            auto link_copies = [&](const Batch &bt) {
                char *ring = p.bounce + static_cast<uint64_t>(bt.ring) * p.bounce_slot_bytes;
                for (size_t i = bt.run0; i < bt.run0 + bt.runs; ++i) {
                    const LinkRun &run = runs[i];
                    char *hmem = static_cast<char *>(p.regions[run.region].host) + run.offset + skip;
                    char *dev = ring + run.slot_offset;
                    void *dst = gather ? static_cast<void *>(dev) : static_cast<void *>(hmem);
                    const void *src = gather ? static_cast<const void *>(hmem) : static_cast<const void *>(dev);
                    if (width == p.block_bytes)
                        check_hip(hipMemcpyAsync(dst, src, run.blocks * width, kind, sc), "hipMemcpyAsync");
                    else
                        check_hip(hipMemcpy2DAsync(dst, gather ? width : p.block_bytes, src, gather ? p.block_bytes : width,
                                                   width, run.blocks, kind, sc),
                                  "hipMemcpy2DAsync");
                }
            };
            auto ring_kernel = [&](const Batch &bt) {
                CopyArgs a = args[KVP_CLASS_HOST];
                a.items = dev_list + bt.first;
                a.n_items = bt.n;
                check_hip(launch_chunk_copy(a, kClassRing, gather, lc.grid, lc.flags, s), "kernel launch");
            };
            if (gather) {
                check_hip(hipStreamWaitEvent(sc, p.fork, 0), "hipStreamWaitEvent");
                if (tc) check_hip(hipEventRecord(tc->t0[KVP_CLASS_HOST], sc), "hipEventRecord");
                for (const Batch &bt : batches) {
                    if (p.bounce_free_rec[bt.ring])
                        check_hip(hipStreamWaitEvent(sc, p.bounce_free[bt.ring], 0), "hipStreamWaitEvent");
                    link_copies(bt);
                    check_hip(hipEventRecord(p.bounce_filled[bt.ring], sc), "hipEventRecord");
                    check_hip(hipStreamWaitEvent(s, p.bounce_filled[bt.ring], 0), "hipStreamWaitEvent");
                    ring_kernel(bt);
                    check_hip(hipEventRecord(p.bounce_free[bt.ring], s), "hipEventRecord");
                    p.bounce_free_rec[bt.ring] = true;
                }
            } else {
                if (tc) check_hip(hipEventRecord(tc->t0[KVP_CLASS_HOST], s), "hipEventRecord");
                for (const Batch &bt : batches) {
                    if (p.bounce_free_rec[bt.ring])
                        check_hip(hipStreamWaitEvent(s, p.bounce_free[bt.ring], 0), "hipStreamWaitEvent");
                    ring_kernel(bt);
                    check_hip(hipEventRecord(p.bounce_filled[bt.ring], s), "hipEventRecord");
                    check_hip(hipStreamWaitEvent(sc, p.bounce_filled[bt.ring], 0), "hipStreamWaitEvent");
                    link_copies(bt);
                    check_hip(hipEventRecord(p.bounce_free[bt.ring], sc), "hipEventRecord");
                    p.bounce_free_rec[bt.ring] = true;
                }
                check_hip(hipEventRecord(p.stage_done, sc), "hipEventRecord");
                check_hip(hipStreamWaitEvent(s, p.stage_done, 0), "hipStreamWaitEvent");
            }
            p.bounce_next = static_cast<uint32_t>((p.bounce_next + batches.size()) % kBounceSlots);
            if (tc) {
                check_hip(hipEventRecord(tc->t1[KVP_CLASS_HOST], s), "hipEventRecord");
                tc->ran[KVP_CLASS_HOST] = true;
            }
        }
        if (!file_batches.empty()) {
            // file-region kernels on the pool's stream, beside the host-class
            // kernel on the caller's, then joined back into the caller's stream
            if (!fork_staging && batches.empty()) check_hip(hipStreamWaitEvent(p.s_stage, p.fork, 0), "hipStreamWaitEvent");
            CopyArgs fa = geo;
            fa.items = dev_list + items[0].size() + items[1].size();
            fa.cache = static_cast<const uint64_t *>(dev_base);
            LaunchCfg lf = p.launch[KVP_CLASS_HOST][op];
            lf.flags &= ~(KVP_LAUNCH_SDMA | KVP_LAUNCH_UPLOAD);
            run_file_batches(p, gather, file_batches, spans, fa, lf, p.s_stage);
            check_hip(hipEventRecord(p.stage_done, p.s_stage), "hipEventRecord");
            check_hip(hipStreamWaitEvent(s, p.stage_done, 0), "hipStreamWaitEvent");
        }
    };
    try {
        enqueue();
    } catch (...) {
        settle();
        throw;
    }
    if (noalloc) {
        check_hip(hipEventRecord(sd->free, s), "hipEventRecord");
        sd->free_rec = true;
    } else {
        check_hip(hipEventRecord(slot->done, s), "hipEventRecord");
    }
    mark_requests();
}

}  // namespace kvp

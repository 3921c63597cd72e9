// Copy-engine transport plan: which host-link copies fill which ring slot,
// and the work items that move each slot to or from the engine cache.
//
// A placed request's blocks in one region occupy one contiguous range
// (Sec. 4.1.3, the LBA-range rule), so after grouping by region the blocks of
// a call form long runs at consecutive offsets: one copy per region per slot.

#include <algorithm>

#include "internal.hpp"

namespace kvp {

void plan_bounce(const RingGeometry &g, std::vector<HostBlock> &blocks, uint64_t width, uint32_t chunk0,
                 std::vector<CopyItem> &items, std::vector<LinkRun> &runs, std::vector<Batch> &batches)
{
    if (width == 0 || width > g.block_bytes || g.slot_bytes < g.block_bytes || g.slots == 0)
        fail(KVP_ERR_INVALID, "copy ring geometry");
    std::stable_sort(blocks.begin(), blocks.end(),
                     [](const HostBlock &x, const HostBlock &y) { return x.region < y.region; });
    const uint64_t per_slot = g.slot_bytes / width;   // >= 1
    const uint64_t rebase = static_cast<uint64_t>(chunk0) * g.chunk_bytes;
    uint64_t used = per_slot;   // forces a first batch
    for (const HostBlock &hb : blocks) {
        if (used == per_slot) {
            const uint32_t ring = static_cast<uint32_t>((g.next + batches.size()) % g.slots);
            batches.push_back(Batch{ring, static_cast<uint32_t>(items.size()), 0u, runs.size(), 0});
            used = 0;
        }
        Batch &bt = batches.back();
        LinkRun *last = bt.runs ? &runs.back() : nullptr;
        if (last && last->region == hb.region && last->offset + last->blocks * g.block_bytes == hb.offset) {
            ++last->blocks;
        } else {
            runs.push_back(LinkRun{hb.region, hb.offset, 1u, used * width});
            ++bt.runs;
        }
        const uint64_t at = g.base + bt.ring * g.slot_bytes + used * width;
        items.push_back(CopyItem{at - rebase, hb.slot, 0u});   // unsigned wrap is exact
        ++bt.n;
        ++used;
    }
}

}  // namespace kvp

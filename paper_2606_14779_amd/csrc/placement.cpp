// Placement of a request's blocks over the pool regions.
//
// Pool organizer (Sec. 4.1.2, Eq. 1): region i receives the fraction
// p_i = b_i / sum_j b_j of the blocks.  Bandwidth-aware allocator (Sec. 4.1.3,
// Eq. 2, Algorithm 1): region i's target count is floor(p_i * n) plus at most
// one leftover block; leftovers go to the regions with the largest p_i, equal
// p_i broken by the lower index.  The blocks are then handed out one by one
// in the request's own (layer-then-token) order; the algorithm only requires
// that the chosen region still has room, and this library picks the region
// that is furthest behind its proportional share, so every request is
// striped over all regions.
// KV-passthrough (Sec. 4.2) gives each (request, region) one contiguous
// range of ceil(c_i * KV_size / sector) sectors; the same rule is used for
// host regions, with a 4096-byte sector.

#include <algorithm>
#include <numeric>

#include "internal.hpp"

namespace kvp {

void target_counts(const uint64_t *bandwidth, uint32_t n_dev, uint64_t n_blocks, uint64_t *counts)
{
    if (n_dev == 0) fail(KVP_ERR_INVALID, "no regions");
    unsigned __int128 sum_b = 0;
    for (uint32_t i = 0; i < n_dev; ++i) {
        if (bandwidth[i] == 0) fail(KVP_ERR_INVALID, "bandwidth of region " + std::to_string(i) + " is 0");
        sum_b += bandwidth[i];
    }
    std::vector<uint32_t> rank(n_dev);   // allocated before counts is written: a failure leaves it as it was
    // floor(p_i * n) = floor(b_i * n / sum b), exact in 128-bit integers
    uint64_t floors = 0;
    for (uint32_t i = 0; i < n_dev; ++i) {
        counts[i] = static_cast<uint64_t>((static_cast<unsigned __int128>(bandwidth[i]) * n_blocks) / sum_b);
        floors += counts[i];
    }
    // sum of the fractional parts is below n_dev, so fewer than n_dev leftovers
    const uint64_t leftover = n_blocks - floors;
    std::iota(rank.begin(), rank.end(), 0u);
    std::stable_sort(rank.begin(), rank.end(),
                     [&](uint32_t a, uint32_t b) { return bandwidth[a] > bandwidth[b]; });
    for (uint64_t k = 0; k < leftover; ++k) counts[rank[k]] += 1;
}

void stripe(const std::vector<uint64_t> &counts, uint32_t n_blocks, std::vector<uint32_t> &region_of)
{
    // Region i is "behind" at block j by (j+1)*c_i/n - a_i blocks; compare
    // n times that value, (j+1)*c_i - n*a_i, to stay in integers.
    const size_t n_dev = counts.size();
    std::vector<uint64_t> given(n_dev, 0);
    region_of.resize(n_blocks);
    for (uint32_t j = 0; j < n_blocks; ++j) {
        size_t pick = n_dev;
        __int128 lead = 0;
        for (size_t i = 0; i < n_dev; ++i) {
            if (given[i] == counts[i]) continue;
            const __int128 behind = static_cast<__int128>(j + 1) * counts[i] -
                                    static_cast<__int128>(n_blocks) * given[i];
            if (pick == n_dev || behind > lead) {
                pick = i;
                lead = behind;
            }
        }
        region_of[j] = static_cast<uint32_t>(pick);
        ++given[pick];
    }
}

RangeAllocator::RangeAllocator(uint64_t capacity)
{
    if (capacity) free_.emplace(0, capacity);
}

bool RangeAllocator::first_fit(uint64_t len, uint64_t *start) const
{
    for (const auto &kv : free_) {
        if (kv.second >= len) {
            *start = kv.first;
            return true;
        }
    }
    return false;
}

void RangeAllocator::take(uint64_t start, uint64_t len)
{
    auto it = free_.upper_bound(start);
    --it;  // the free range containing start (first_fit guarantees it exists)
    const uint64_t fs = it->first, fl = it->second;
    const uint64_t tail = fs + fl - start - len;
    if (start == fs) {
        if (tail == 0) {
            if (spare_.size() < spare_.capacity())
                spare_.push_back(free_.extract(it));   // kept for a later give()
            else
                free_.erase(it);
            return;
        }
        auto node = free_.extract(it);   // re-keyed in place: no allocation
        node.key() = start + len;
        node.mapped() = tail;
        free_.insert(std::move(node));
        return;
    }
    if (tail) free_.emplace(start + len, tail);   // the only step that can fail, taken first
    it->second = start - fs;
}

void RangeAllocator::reserve_gives(size_t k)
{
    if (spare_.size() >= k) return;
    spare_.reserve(k);
    Free scratch;   // nodes are made by inserting and unlinking them
    while (spare_.size() < k) {
        scratch.emplace(0, 0);
        spare_.push_back(scratch.extract(scratch.begin()));
    }
}

void RangeAllocator::give(uint64_t start, uint64_t len)
{
    auto next = free_.lower_bound(start);
    if (next != free_.end() && start + len == next->first) {   // merge with the range after
        auto node = free_.extract(next);
        node.key() = start;
        node.mapped() += len;
        next = free_.insert(std::move(node)).position;
        if (next != free_.begin()) {                           // and with the one before
            auto prev = std::prev(next);
            if (prev->first + prev->second == start) {
                prev->second += next->second;
                free_.erase(next);
            }
        }
        return;
    }
    if (next != free_.begin()) {
        auto prev = std::prev(next);
        if (prev->first + prev->second == start) {
            prev->second += len;
            return;
        }
    }
    if (spare_.empty()) {
        free_.emplace(start, len);
        return;
    }
    auto node = std::move(spare_.back());
    spare_.pop_back();
    node.key() = start;
    node.mapped() = len;
    free_.insert(std::move(node));
}

uint64_t RangeAllocator::largest() const
{
    uint64_t m = 0;
    for (const auto &kv : free_) m = std::max(m, kv.second);
    return m;
}

}  // namespace kvp

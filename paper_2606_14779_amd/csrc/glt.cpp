// Global lookup table (Sec. 4.1.1, Table "Fields of the GLT"): one entry per
// offloaded block with its key, device index, device type and location.
// The key is a hash of the block identifier (request, block index); the full
// identifier is stored too, so two blocks whose hashes collide never alias.
// Linear probing with backward-shift deletion; kept at load factor 1/2 or below.

#include "internal.hpp"

namespace kvp {

static inline uint64_t mix64(uint64_t x)
{
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

Glt::Glt() : slots_(1024), used_(1024, 0) {}

uint64_t Glt::hash(uint64_t request, uint32_t block)
{
    return mix64(request ^ mix64(0x4B56ull << 32 | block));
}

// Probe from the entry's home slot to its own or the first empty slot.
void Glt::place(const GltEntry &e)
{
    const size_t mask = slots_.size() - 1;
    size_t i = hash(e.request, e.block) & mask;
    while (used_[i]) {
        if (slots_[i].request == e.request && slots_[i].block == e.block) {
            slots_[i] = e;
            return;
        }
        i = (i + 1) & mask;
    }
    slots_[i] = e;
    used_[i] = 1;
    ++count_;
}

void Glt::reserve(size_t extra)
{
    size_t cap = slots_.size();
    while ((count_ + extra) * 2 > cap) cap *= 2;
    if (cap == slots_.size()) return;
    Glt bigger;                      // built aside, swapped in only when complete
    bigger.slots_.assign(cap, GltEntry{});
    bigger.used_.assign(cap, 0);
    for (size_t i = 0; i < slots_.size(); ++i)
        if (used_[i]) bigger.place(slots_[i]);
    slots_.swap(bigger.slots_);
    used_.swap(bigger.used_);
}

void Glt::insert(const GltEntry &e)
{
    reserve(1);
    place(e);
}

const GltEntry *Glt::find(uint64_t request, uint32_t block) const
{
    const size_t mask = slots_.size() - 1;
    size_t i = hash(request, block) & mask;
    while (used_[i]) {
        if (slots_[i].request == request && slots_[i].block == block) return &slots_[i];
        i = (i + 1) & mask;
    }
    return nullptr;
}

bool Glt::erase(uint64_t request, uint32_t block)
{
    const size_t mask = slots_.size() - 1;
    size_t i = hash(request, block) & mask;
    while (used_[i] && !(slots_[i].request == request && slots_[i].block == block)) i = (i + 1) & mask;
    if (!used_[i]) return false;
    // backward-shift: pull later members of the probe run into the hole
    size_t hole = i, j = i;
    for (;;) {
        j = (j + 1) & mask;
        if (!used_[j]) break;
        const size_t home = hash(slots_[j].request, slots_[j].block) & mask;
        // j may move to hole iff home is not cyclically in (hole, j]
        const bool in_range = hole <= j ? (home > hole && home <= j) : (home > hole || home <= j);
        if (!in_range) {
            slots_[hole] = slots_[j];
            hole = j;
        }
    }
    used_[hole] = 0;
    --count_;
    return true;
}

}  // namespace kvp

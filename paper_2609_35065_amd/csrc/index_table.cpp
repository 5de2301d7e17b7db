// index_table.cpp -- host table of the staged-chunk index (plain C++).

#include "index_table.h"

#include <algorithm>

#include "tempokv.h"

namespace tkv {

bool IndexTable::init(int64_t max_entries_, int64_t reserve_changes) {
    if (max_entries_ <= 0 || max_entries_ > (int64_t(1) << 28) || reserve_changes < 0) return false;
    max_entries = max_entries_;
    log2cap = 6;
    while ((int64_t(1) << log2cap) < 2 * max_entries) ++log2cap;
    cap = int64_t(1) << log2cap;
    live = tombs = 0;
    rebuilt = true;
    entries.assign((size_t)cap, IndexEntry{0, -1, kEmpty});
    spare_.assign((size_t)cap, IndexEntry{0, -1, kEmpty});
    dirty_.clear();
    dirty_.reserve((size_t)reserve_changes);
    return true;
}

int64_t IndexTable::probe(uint64_t key, int64_t *free_pos) const {
    const uint64_t mask = (uint64_t)cap - 1;
    uint64_t pos = index_home(key, log2cap);
    int64_t first_free = -1;
    for (int64_t n = 0; n < cap; ++n) {
        const IndexEntry &e = entries[pos];
        if (e.state == kEmpty) {
            if (first_free < 0) first_free = (int64_t)pos;
            break;
        }
        if (e.state == kTomb) {
            if (first_free < 0) first_free = (int64_t)pos;
        } else if (e.key == key) {
            if (free_pos) *free_pos = first_free;
            return (int64_t)pos;
        }
        pos = (pos + 1) & mask;
    }
    if (free_pos) *free_pos = first_free;
    return -1;
}

// Rebuild without tombstones once live keys and tombstones fill three
// quarters of the table, in the spare buffer reserved by init.
void IndexTable::rehash_if_crowded() {
    if ((live + tombs) * 4 <= cap * 3) return;
    rebuilt = true;
    dirty_.clear();
    spare_.swap(entries);
    std::fill(entries.begin(), entries.end(), IndexEntry{0, -1, kEmpty});
    tombs = 0;
    const uint64_t mask = (uint64_t)cap - 1;
    for (const IndexEntry &e : spare_) {
        if (e.state != kLive) continue;
        uint64_t pos = index_home(e.key, log2cap);
        while (entries[pos].state != kEmpty) pos = (pos + 1) & mask;
        entries[pos] = e;
    }
}

int IndexTable::insert(const uint64_t *keys, const int32_t *slots, int32_t n) {
    for (int32_t i = 0; i < n; ++i) {
        int64_t free_pos = -1;
        const int64_t at = probe(keys[i], &free_pos);
        if (at >= 0) {
            entries[at].slot = slots[i];
            dirty_.push_back(at);
            continue;
        }
        if (live >= max_entries || free_pos < 0) return KV_ENOSPC;
        if (entries[free_pos].state == kTomb) --tombs;
        entries[free_pos] = IndexEntry{keys[i], slots[i], kLive};
        dirty_.push_back(free_pos);
        ++live;
        rehash_if_crowded();
    }
    return KV_OK;
}

void IndexTable::erase(const uint64_t *keys, int32_t n) {
    for (int32_t i = 0; i < n; ++i) {
        const int64_t at = probe(keys[i], nullptr);
        if (at < 0) continue;
        entries[at].state = kTomb;
        entries[at].slot = -1;
        dirty_.push_back(at);
        --live;
        ++tombs;
    }
    rehash_if_crowded();
}

int32_t IndexTable::find(uint64_t key) const {
    const int64_t at = probe(key, nullptr);
    return at >= 0 ? entries[at].slot : -1;
}

const std::vector<int64_t> &IndexTable::changes() {
    std::sort(dirty_.begin(), dirty_.end());
    dirty_.erase(std::unique(dirty_.begin(), dirty_.end()), dirty_.end());
    return dirty_;
}

}  // namespace tkv

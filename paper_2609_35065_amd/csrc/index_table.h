// index_table.h -- the staged-chunk index's host table: key -> staging slot,
// open addressing with linear probing from a Fibonacci-hashed home position
// and tombstones for erased keys.  Plain C++ (no HIP header): index.hip
// mirrors the table to the device, and the table can also be built and tested
// on its own.
#pragma once

#include <stdint.h>

#include <vector>

namespace tkv {

// One table entry: 16 bytes, the layout of the device mirror too (read by one
// dwordx4 load in the lookup kernel's probe loop).
struct alignas(16) IndexEntry {
    uint64_t key;
    int32_t slot;
    int32_t state;   // kEmpty, kLive or kTomb
};
constexpr int32_t kEmpty = 0;
constexpr int32_t kLive = 1;
constexpr int32_t kTomb = 2;

// Home position of a key in a table of 2^log2cap entries (Fibonacci hashing:
// the high bits of key * 2^64/phi), so that any key set, including small or
// sequential keys, spreads over the table.  constexpr, so the lookup kernel
// calls the same function on the device.
constexpr uint64_t index_home(uint64_t key, int log2cap) {
    return (key * 0x9E3779B97F4A7C15ull) >> (64 - log2cap);
}

class IndexTable {
  public:
    // Size the table for up to max_entries live keys (2^k >= 2 * max_entries
    // positions, at least 64) and reserve every buffer a mutation needs, so
    // that inserts, erases and rebuilds allocate no memory afterwards.
    // Returns false for max_entries outside [1, 2^28].
    bool init(int64_t max_entries, int64_t reserve_changes);

    // Position of `key`, or -1; *free_pos (if given) receives the first
    // reusable position met on the probe path (tombstone or empty), or -1.
    int64_t probe(uint64_t key, int64_t *free_pos) const;

    // Insert or update n pairs.  Returns KV_OK, or KV_ENOSPC at the first key
    // that would exceed max_entries live keys (the pairs before it stay).
    int insert(const uint64_t *keys, const int32_t *slots, int32_t n);

    // Remove n keys; absent keys are ignored.
    void erase(const uint64_t *keys, int32_t n);

    // Slot of a key, or -1.
    int32_t find(uint64_t key) const;

    // Sorted, de-duplicated positions changed since the last clear_changes().
    const std::vector<int64_t> &changes();
    void clear_changes() { dirty_.clear(); }

    int64_t max_entries = 0;
    int log2cap = 0;
    int64_t cap = 0;
    int64_t live = 0;
    int64_t tombs = 0;
    bool rebuilt = true;               // the whole table changed (new, or rehashed) since the last upload
    std::vector<IndexEntry> entries;   // the table, cap positions

  private:
    void rehash_if_crowded();
    std::vector<IndexEntry> spare_;    // same size as entries: a rebuild fills it, then swaps
    std::vector<int64_t> dirty_;       // positions changed since the last clear_changes()
};

}  // namespace tkv

// Randomised check of the index's host table (paper_2609_35065_amd/csrc/
// index_table.cpp) against std::unordered_map, built with the address and
// undefined-behaviour sanitizers by tests/test_sanitizers.py.  It also
// replays the table's change lists onto a mirror, as the device upload does,
// and checks that the mirror always equals the table.
#include <stdio.h>
#include <string.h>

#include <random>
#include <unordered_map>
#include <vector>

#include "index_table.h"
#include "tempokv.h"

#define CHECK(c)                                                     \
    do {                                                             \
        if (!(c)) {                                                  \
            fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
            return 1;                                                \
        }                                                            \
    } while (0)

static int run(uint64_t seed, int64_t max_entries, int rounds) {
    std::mt19937_64 rng(seed);
    tkv::IndexTable t;
    CHECK(t.init(max_entries, 4096));
    std::unordered_map<uint64_t, int32_t> ref;
    std::vector<tkv::IndexEntry> mirror;
    // keys from a small universe so that inserts update, erases hit, and tombstones pile up
    std::vector<uint64_t> universe(3 * (size_t)max_entries);
    for (auto &k : universe) k = rng();
    universe[0] = 0;   // the key 0 is a key like any other
    for (int round = 0; round < rounds; ++round) {
        const int op = (int)(rng() % 3);
        const int32_t n = (int32_t)(rng() % (uint64_t)(max_entries / 2 + 2));
        std::vector<uint64_t> keys(n);
        std::vector<int32_t> slots(n);
        for (int32_t i = 0; i < n; ++i) {
            keys[i] = universe[rng() % universe.size()];
            slots[i] = (int32_t)(rng() % 100000);
        }
        if (op < 2) {
            const int rc = t.insert(keys.data(), slots.data(), n);
            for (int32_t i = 0; i < n; ++i) {
                auto it = ref.find(keys[i]);
                if (it == ref.end() && (int64_t)ref.size() >= max_entries) {
                    CHECK(rc == KV_ENOSPC);   // stops at the first key that does not fit
                    break;
                }
                ref[keys[i]] = slots[i];
                if (i == n - 1) CHECK(rc == KV_OK);
            }
        } else {
            t.erase(keys.data(), n);
            for (uint64_t k : keys) ref.erase(k);
        }
        CHECK(t.live == (int64_t)ref.size());
        CHECK((t.live + t.tombs) * 4 <= t.cap * 3);
        for (uint64_t k : universe) {
            auto it = ref.find(k);
            CHECK(t.find(k) == (it == ref.end() ? -1 : it->second));
        }
        // the upload: the whole image after a rebuild, else the changed positions
        if (t.rebuilt) {
            mirror = t.entries;
        } else {
            for (int64_t p : t.changes()) {
                CHECK(p >= 0 && p < t.cap);
                mirror[(size_t)p] = t.entries[(size_t)p];
            }
        }
        t.rebuilt = false;
        t.clear_changes();
        CHECK(mirror.size() == t.entries.size());
        CHECK(memcmp(mirror.data(), t.entries.data(), mirror.size() * sizeof(tkv::IndexEntry)) == 0);
    }
    return 0;
}

int main() {
    tkv::IndexTable bad;
    if (bad.init(0, 0) || bad.init(int64_t(1) << 29, 0)) {
        fprintf(stderr, "init accepted an invalid size\n");
        return 1;
    }
    const int64_t sizes[] = {1, 2, 7, 32, 100, 1000};
    for (int64_t m : sizes)
        for (uint64_t seed = 1; seed <= 4; ++seed)
            if (run(seed * 7919 + (uint64_t)m, m, 300)) return 1;
    printf("index table check ok\n");
    return 0;
}

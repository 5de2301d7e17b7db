/* Host form of the workload generator's KV content formula (input
 * generation only; no part of the method under test).  Word i of a buffer:
 *   chi = fmix32(hi32(i) + k2);  v = fmix32(fmix32(lo32(i) ^ k1) ^ chi)
 *   finite: v &= 0xBFFFBFFF
 * fmix32 is the 32-bit MurmurHash3 finalizer (Appleby, public domain). */
#include <stdint.h>

static inline uint32_t fmix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x85EBCA6Bu;
    x ^= x >> 13;
    x *= 0xC2B2AE35u;
    x ^= x >> 16;
    return x;
}

void kvfill_words(uint32_t k1, uint32_t k2, uint64_t start, uint64_t count, int finite, uint32_t *out)
{
    const uint32_t mask = finite ? 0xBFFFBFFFu : 0xFFFFFFFFu;
    uint64_t pos = 0;
    while (pos < count) {
        uint64_t idx0 = start + pos;
        uint64_t room = (1ull << 32) - (idx0 & 0xFFFFFFFFull);
        uint64_t n = count - pos < room ? count - pos : room;
        uint32_t chi = fmix32((uint32_t)(idx0 >> 32) + k2);
        uint32_t lo0 = (uint32_t)idx0;
        uint32_t *o = out + pos;
        for (uint64_t i = 0; i < n; i++)
            o[i] = fmix32(fmix32((lo0 + (uint32_t)i) ^ k1) ^ chi) & mask;
        pos += n;
    }
}

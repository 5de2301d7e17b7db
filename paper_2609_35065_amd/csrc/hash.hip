// hash.hip -- chained prefix hash and prefix lookup kernels for CDNA4 (gfx950).
//
// Hash.  h_{-1} = seed, h_b = M(h_{b-1} ^ d_b ^ G), d_b = sum_j M(word(j, tok))
// over the 16 tokens of block b, M = SplitMix64's finalizer.  The digests are
// independent and computed one block per lane; the chain is sequential and
// runs on one lane per request, fed from LDS.  One 256-lane workgroup per
// request walks its blocks in tiles of 256.
//
// Lookup.  One wave per request probes up to 64 chunk keys at once in the
// device open-addressing table and turns the 64 hit flags into the length of
// the leading run of hits with one ballot and a count of trailing ones.

#include "internal.h"

namespace tkv {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int kHashThreads = 256;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(kHashThreads) void hash_kernel(const int32_t *__restrict__ tokens,
                                                          const int64_t *__restrict__ tok_off,
                                                          uint64_t seed, const int64_t *__restrict__ blk_off,
                                                          uint64_t *__restrict__ out) {
    __shared__ uint64_t dig[kHashThreads];
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t t0 = tok_off[r];
    const int64_t n = tok_off[r + 1] - t0;
    int64_t nb = n > 0 ? n / 16 : 0;
    const int64_t o0 = blk_off[r];
    const int64_t span = blk_off[r + 1] - o0;
    if (span < nb) nb = span > 0 ? span : 0;

    uint64_t h = seed;
    for (int64_t tile = 0; tile < nb; tile += kHashThreads) {
        const int64_t b = tile + tid;
        if (b < nb) {
            const int32_t *tp = tokens + t0 + b * 16;
            uint64_t d = 0;
#pragma unroll
            for (int j = 0; j < 16; ++j)
                d += mix64((uint64_t)(uint32_t)tp[j] + ((uint64_t)(j + 1) << 32));
            dig[tid] = d;
        }
        __syncthreads();
        if (tid == 0) {
            const int64_t cnt = nb - tile < kHashThreads ? nb - tile : kHashThreads;
            for (int64_t k = 0; k < cnt; ++k) {
                h = mix64(h ^ dig[k] ^ kGamma);
                out[o0 + tile + k] = h;
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(64) void lookup_kernel(const IndexEntry *__restrict__ table, int log2cap,
                                                    const uint64_t *__restrict__ bh,
                                                    const int64_t *__restrict__ blk_off, int32_t bpc,
                                                    const int64_t *__restrict__ chunk_off,
                                                    int32_t *__restrict__ chunk_slot,
                                                    int32_t *__restrict__ hit_chunks) {
    const int r = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t b0 = blk_off[r];
    int64_t nb = blk_off[r + 1] - b0;
    if (nb < 0) nb = 0;
    int64_t nc = nb / bpc;
    const int64_t c0 = chunk_off[r];
    const int64_t cspan = chunk_off[r + 1] - c0;
    if (cspan < nc) nc = cspan > 0 ? cspan : 0;
    const uint64_t mask = (uint64_t(1) << log2cap) - 1;

    int32_t hits = 0;
    bool alive = true;
    for (int64_t base = 0; base < nc; base += 64) {
        const int64_t j = base + lane;
        int32_t slot = -1;
        if (j < nc) {
            const uint64_t key = bh[b0 + (j + 1) * bpc - 1];
            uint64_t pos = index_home(key, log2cap);
            for (uint64_t probe = 0; probe <= mask; ++probe) {   // bounded: a full table ends the walk
                const IndexEntry e = table[pos];
                if (e.state == kEmpty) break;
                if (e.state == kLive && e.key == key) {
                    slot = e.slot;
                    break;
                }
                pos = (pos + 1) & mask;
            }
            chunk_slot[c0 + j] = slot;
        }
        const uint64_t present = __ballot(j < nc && slot >= 0);
        if (alive) {
            const uint64_t missing = ~present;
            const int run = missing ? __builtin_ctzll(missing) : 64;
            hits += run;
            alive = (run == 64);
        }
    }
    if (lane == 0) hit_chunks[r] = hits;
}

}  // namespace

hipError_t launch_hash(const int32_t *tokens, const int64_t *tok_off, int32_t num_reqs, uint64_t seed,
                       const int64_t *blk_off, uint64_t *out, hipStream_t stream) {
    if (num_reqs <= 0) return hipSuccess;
    (void)hipGetLastError();
    hipLaunchKernelGGL(hash_kernel, dim3(num_reqs), dim3(kHashThreads), 0, stream, tokens, tok_off, seed,
                       blk_off, out);
    return hipGetLastError();
}

hipError_t launch_lookup(const IndexEntry *table, int log2cap, const uint64_t *block_hash,
                         const int64_t *blk_off, int32_t num_reqs, int32_t bpc, const int64_t *chunk_off,
                         int32_t *chunk_slot, int32_t *hit_chunks, hipStream_t stream) {
    if (num_reqs <= 0) return hipSuccess;
    (void)hipGetLastError();
    hipLaunchKernelGGL(lookup_kernel, dim3(num_reqs), dim3(64), 0, stream, table, log2cap, block_hash, blk_off,
                       bpc, chunk_off, chunk_slot, hit_chunks);
    return hipGetLastError();
}

}  // namespace tkv

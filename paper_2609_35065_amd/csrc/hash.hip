// hash.hip -- chained prefix hash and prefix lookup kernels for CDNA4 (gfx950).
//
// Hash.  h_{-1} = seed, h_b = M(h_{b-1} ^ d_b ^ G), d_b = sum_j M(word(j, tok))
// over the 16 tokens of block b, M = SplitMix64's finalizer.  The digests are
// independent and computed one block per lane; the chain is sequential, so
// its latency sets the rate: it runs on the scalar ALU of one wave per
// request (a step is ~20 scalar instructions: two xor-shift-multiply rounds
// on 32-bit halves), while the workgroup's other waves digest the next tile.
//
// Lookup.  One wave per request probes up to 64 chunk keys at once in the
// device open-addressing table and turns the 64 hit flags into the length of
// the leading run of hits with one ballot and a count of trailing ones.

#include "internal.h"

namespace tkv {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int kWave = 64;
constexpr int kHashThreads = 256;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}

// Lane K of `old` takes the wave-uniform value `val` (v_writelane_b32 with
// an inline-constant lane number); the other lanes keep theirs.
template <int K>
__device__ __forceinline__ uint32_t writelane(uint32_t old, uint32_t val) {
    asm("v_writelane_b32 %0, %1, %2" : "+v"(old) : "s"(val), "n"(K));
    return old;
}

// Steps K..K+7 of the chain over a full group of 64 blocks, unrolled so that
// every lane number is an immediate.  The eight digests are read into scalar
// registers before the eight dependent steps, keeping v_readlane latency off
// the chain.
template <int K>
struct ChainGroup {
    static __device__ __forceinline__ void run(uint64_t &h, uint64_t d, uint32_t &lo, uint32_t &hi) {
        uint64_t dk[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) dk[j] = readlane64(d, K + j);
        __builtin_amdgcn_sched_barrier(0);   // keep the reads ahead of the steps
        uint64_t hk[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            h = mix64(h ^ dk[j]);
            hk[j] = h;
        }
        Park<K, 0>::run(hk, lo, hi);
        ChainGroup<K + 8>::run(h, d, lo, hi);
    }
    template <int B, int J>
    struct Park {
        static __device__ __forceinline__ void run(const uint64_t *hk, uint32_t &lo, uint32_t &hi) {
            lo = writelane<B + J>(lo, (uint32_t)hk[J]);
            hi = writelane<B + J>(hi, (uint32_t)(hk[J] >> 32));
            Park<B, J + 1>::run(hk, lo, hi);
        }
    };
    template <int B>
    struct Park<B, 8> {
        static __device__ __forceinline__ void run(const uint64_t *, uint32_t &, uint32_t &) {}
    };
};
template <>
struct ChainGroup<64> {
    static __device__ __forceinline__ void run(uint64_t &, uint64_t, uint32_t &, uint32_t &) {}
};

__device__ __forceinline__ uint64_t block_digest(const int32_t *tp) {
    uint64_t d = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) d += mix64((uint64_t)(uint32_t)tp[j] + ((uint64_t)(j + 1) << 32));
    return d ^ kGamma;   // the chain's constant, folded in here, off the chain
}

// One 256-lane workgroup per request, blocks in tiles of 256.  The digests
// of a tile are independent: all four waves compute the first tile into LDS;
// afterwards wave 0 runs the chain over tile t while waves 1-3 digest tile
// t+1 into the other LDS buffer.  The chain runs with wave-uniform values, so
// it executes on the scalar ALU: for each group of 64 blocks, lane k holds
// digest k, v_readlane moves it to scalar registers, and v_writelane parks
// h_k in lane k, which then stores the group's 64 hashes in one write.
__global__ __launch_bounds__(kHashThreads) void hash_kernel(const int32_t *__restrict__ tokens,
                                                           const int64_t *__restrict__ tok_off, uint64_t seed,
                                                           const int64_t *__restrict__ blk_off,
                                                           uint64_t *__restrict__ out) {
    __shared__ uint64_t dig[2][kHashThreads];
    const int r = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // wave-uniform by construction
    const int lane = tid % kWave;
    const int64_t t0 = tok_off[r];
    const int64_t n = tok_off[r + 1] - t0;
    int64_t nb = n > 0 ? n / 16 : 0;
    const int64_t o0 = blk_off[r];
    const int64_t span = blk_off[r + 1] - o0;
    if (span < nb) nb = span > 0 ? span : 0;
    const int64_t ntiles = (nb + kHashThreads - 1) / kHashThreads;
    const int32_t *tk = tokens + t0;

    if (tid < nb) dig[0][tid] = block_digest(tk + (int64_t)tid * 16);
    __syncthreads();
    uint64_t h = seed;   // live in wave 0 only
    for (int64_t t = 0; t < ntiles; ++t) {
        const int64_t tb = t * kHashThreads;
        if (wave == 0) {
            const uint64_t *dt = dig[t & 1];
            const int64_t left = nb - tb < kHashThreads ? nb - tb : kHashThreads;
            for (int64_t g = 0; g < left; g += kWave) {
                const uint64_t d = dt[g + lane];
                uint32_t mine_lo = 0, mine_hi = 0;
                if (left - g >= kWave) {
                    ChainGroup<0>::run(h, d, mine_lo, mine_hi);
                } else {                               // ragged last group
                    const int cnt = (int)(left - g);
                    uint64_t mine = 0;
                    for (int k = 0; k < cnt; ++k) {
                        h = mix64(h ^ readlane64(d, k));
                        if (lane == k) mine = h;
                    }
                    mine_lo = (uint32_t)mine;
                    mine_hi = (uint32_t)(mine >> 32);
                }
                if (g + lane < left) out[o0 + tb + g + lane] = ((uint64_t)mine_hi << 32) | mine_lo;
            }
        } else if (t + 1 < ntiles) {
            const int64_t nt = tb + kHashThreads;
            for (int i = tid - kWave; i < kHashThreads; i += kHashThreads - kWave)
                if (nt + i < nb) dig[(t + 1) & 1][i] = block_digest(tk + (nt + i) * 16);
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
    hipLaunchKernelGGL(hash_kernel, dim3(num_reqs), dim3(kHashThreads), 0, stream, tokens, tok_off, seed, blk_off,
                       out);
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

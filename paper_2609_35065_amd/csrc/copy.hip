// copy.hip -- retrieve scatter and store gather between staged chunks and
// paged KV blocks, for CDNA4 (gfx950).
//
// The unit of work is one segment: the B tokens of one layer's K or V plane
// that make up one paged block, B*H*D*e contiguous bytes on both sides
// (32 KiB for block 16 x 8 heads x 128 dims x 2 bytes).  One workgroup of
// 256 lanes moves one segment with 16-byte vector loads and stores: each
// wave instruction covers 1 KiB of contiguous bytes, and every lane issues
// all its loads for the segment before its first store, so a 32 KiB segment
// has 8 loads of 16 bytes in flight per lane.
//
// Segment order.  Workgroup g handles job q = g mod num_jobs of the segment
// position (layer, plane, block-in-chunk) = g / num_jobs.  Consecutive
// workgroups therefore copy the same segment position for consecutive jobs:
// jobs that share a staged chunk (many requests reusing one prefix) re-read
// the same 32 KiB within a short window, where L2 or the Infinity Cache
// serves it, and at any moment the paged writes fall inside one layer plane
// instead of the whole pool, which keeps the page-translation working set
// small.
//
// Retrieve reads staging with ordinary (cached) loads because chunks are
// shared between jobs, and writes the paged blocks with non-temporal stores
// because nothing re-reads them in this kernel.  Store reads the paged blocks
// non-temporally (each is read once) and writes staging non-temporally.

#include "internal.h"

namespace tkv {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;                    // 16-byte vectors per lane per pass
constexpr int64_t kPassVecs = (int64_t)kThreads * kUnroll;

template <bool kSrcCached>
__device__ __forceinline__ v4u load16(const v4u *p) {
    if constexpr (kSrcCached) return *p;
    else return __builtin_nontemporal_load(p);
}

// Copy `bytes` (a multiple of 16) from src to dst with the whole workgroup.
template <bool kSrcCached>
__device__ __forceinline__ void copy_segment(v4u *__restrict__ dst, const v4u *__restrict__ src,
                                             int64_t bytes, int tid) {
    const int64_t n = bytes >> 4;
    int64_t base = 0;
    for (; base + kPassVecs <= n; base += kPassVecs) {
        v4u r[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) r[k] = load16<kSrcCached>(src + base + k * kThreads + tid);
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) __builtin_nontemporal_store(r[k], dst + base + k * kThreads + tid);
    }
    if (base < n) {   // ragged tail: segments that are not a multiple of 32 KiB
        v4u r[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int64_t v = base + k * kThreads + tid;
            if (v < n) r[k] = load16<kSrcCached>(src + v);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int64_t v = base + k * kThreads + tid;
            if (v < n) __builtin_nontemporal_store(r[k], dst + v);
        }
    }
}

template <bool kRetrieve>
__global__ __launch_bounds__(kThreads) void kv_copy_kernel(CopyParams p) {
    const int tid = threadIdx.x;
    for (int64_t g = blockIdx.x; g < p.total_segs; g += gridDim.x) {
        const int64_t q = g % p.num_jobs;
        int64_t t = g / p.num_jobs;
        const int32_t i = (int32_t)(t % p.nseg);
        t /= p.nseg;
        const int32_t kv = (int32_t)(t & 1);
        const int32_t l = (int32_t)(t >> 1);

        const kv_job jb = p.jobs[q];
        if (jb.slot < 0 || jb.slot >= p.num_slots || jb.req < 0 || jb.req >= p.num_reqs || jb.chunk < 0 ||
            (int64_t)(jb.chunk + 1) * p.nseg > p.bt_stride)
            continue;
        const int32_t blk = p.bt[(int64_t)jb.req * p.bt_stride + (int64_t)jb.chunk * p.nseg + i];
        if (blk < 0 || blk >= p.num_blocks) continue;

        char *stg = p.staging + (int64_t)jb.slot * p.slot_bytes + (((int64_t)l * 2 + kv) * p.nseg + i) * p.seg_bytes;
        char *pg = p.layers[l] + kv * p.kv_stride + (int64_t)blk * p.block_stride;
        if constexpr (kRetrieve)
            copy_segment<true>(reinterpret_cast<v4u *>(pg), reinterpret_cast<const v4u *>(stg), p.seg_bytes, tid);
        else
            copy_segment<false>(reinterpret_cast<v4u *>(stg), reinterpret_cast<const v4u *>(pg), p.seg_bytes, tid);
    }
}

}  // namespace

hipError_t launch_copy(const CopyParams &p, bool retrieve, hipStream_t stream) {
    if (p.total_segs <= 0) return hipSuccess;
    const int64_t kMaxGrid = int64_t(1) << 30;
    const unsigned grid = (unsigned)(p.total_segs < kMaxGrid ? p.total_segs : kMaxGrid);
    (void)hipGetLastError();   // clear an error left by an unrelated earlier call
    if (retrieve)
        hipLaunchKernelGGL(kv_copy_kernel<true>, dim3(grid), dim3(kThreads), 0, stream, p);
    else
        hipLaunchKernelGGL(kv_copy_kernel<false>, dim3(grid), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace tkv

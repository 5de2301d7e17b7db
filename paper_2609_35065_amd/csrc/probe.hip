// probe.hip -- a measurement reference for the retrieve, not part of the path.
//
// kv_probe_mixed_traffic moves the retrieve's algorithmic bytes -- every
// segment of the distinct staged chunks read once, every destination segment
// written once -- in one launch, with no data passing from the reads to the
// writes: 256-lane workgroups, each one segment, readers spread evenly among
// writers in dispatch order (writers in (layer, plane)-major, then job, then
// segment order; readers likewise over the distinct slots).  Writes store a
// caller-given filler word non-temporally; reads are non-temporal and their
// values are kept alive by an empty asm, so the compiler cannot drop them.
// A retrieve that runs as fast as this launch loses nothing to its own
// structure (waiting on loads, re-reads through L2, block-id loads): what is
// left is the memory system's cost of interleaving these reads and writes.

#include "internal.h"

namespace tkv {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) v4i *const_job_ptr;
typedef const __attribute__((address_space(4))) int32_t *const_i32_ptr;

constexpr int kThreads = 256;

__device__ __forceinline__ bool probe_job_ok(const CopyParams &p, const v4i jb) {
    return jb.x >= 0 && jb.x < p.num_slots && jb.y >= 0 && jb.y < p.num_reqs && jb.z >= 0 &&
           ((int64_t)jb.z + 1) * p.nseg <= p.bt_stride;
}

// Blocks 0 .. nw+nr-1; block b is a reader when floor((b+1)*nr/n) exceeds
// floor(b*nr/n), so exactly nr readers are spread evenly over the n blocks.
__global__ __launch_bounds__(kThreads) void mixed_traffic_kernel(CopyParams p, const int32_t *slots, int32_t nslots,
                                                                 int64_t nw, int64_t nr, uint32_t fill) {
    const int tid = threadIdx.x;
    const int64_t n = nw + nr;
    const int64_t nv = p.seg_bytes >> 4;   // 16-byte vectors per segment
    v4u acc = {0, 0, 0, 0};
    for (int64_t b = blockIdx.x; b < n; b += gridDim.x) {
        const int64_t before = b * nr / n;
        if ((b + 1) * nr / n > before) {
            const int64_t per_pl = (int64_t)nslots * p.nseg;
            const int64_t pl = before / per_pl;
            const int64_t rem = before % per_pl;
            const int32_t slot = slots[rem / p.nseg];
            const int64_t s = rem % p.nseg;
            if (slot < 0 || slot >= p.num_slots) continue;
            const v4u *src = reinterpret_cast<const v4u *>(p.staging + (int64_t)slot * p.slot_bytes +
                                                           (pl * p.nseg + s) * p.seg_bytes);
#pragma unroll 8
            for (int64_t v = tid; v < nv; v += kThreads) acc ^= __builtin_nontemporal_load(src + v);
        } else {
            const int64_t wi = b - before;
            const int64_t per_pl = (int64_t)p.num_jobs * p.nseg;
            const int64_t pl = wi / per_pl;
            const int64_t rem = wi % per_pl;
            const v4i jb = ((const_job_ptr)p.jobs)[rem / p.nseg];
            if (!probe_job_ok(p, jb)) continue;
            const int32_t blk =
                ((const_i32_ptr)p.bt)[(int64_t)jb.y * p.bt_stride + (int64_t)jb.z * p.nseg + rem % p.nseg];
            if (blk < 0 || blk >= p.num_blocks) continue;
            v4u *dst = reinterpret_cast<v4u *>(p.layers[pl >> 1] + (pl & 1) * p.kv_stride +
                                               (int64_t)blk * p.block_stride);
            const v4u val = {fill, fill, fill, fill};
#pragma unroll 8
            for (int64_t v = tid; v < nv; v += kThreads) __builtin_nontemporal_store(val, dst + v);
        }
    }
    asm volatile("" : : "v"(acc.x), "v"(acc.y), "v"(acc.z), "v"(acc.w));
}

}  // namespace
}  // namespace tkv

extern "C" int kv_probe_mixed_traffic(const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                                      const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs,
                                      const kv_job *d_jobs, int32_t num_jobs, const int32_t *d_slots,
                                      int32_t num_read_slots, uint32_t fill, void *stream) {
    tkv::CopyParams p;
    const int rc = tkv::make_copy_params(p, layout, d_staging, (const void *const *)h_layer_ptrs, d_block_tables,
                                         bt_stride, num_reqs, d_jobs, num_jobs);
    if (rc != KV_OK) return rc;
    if (num_read_slots < 0 || (num_read_slots > 0 && !d_slots)) return KV_EINVAL;
    const int64_t planes = (int64_t)p.L * 2 * p.nseg;
    const int64_t nw = (int64_t)num_jobs * planes;
    const int64_t nr = (int64_t)num_read_slots * planes;
    const int64_t n = nw + nr;
    if (n == 0) return KV_OK;
    if (n >= (int64_t(1) << 31)) return KV_EINVAL;   // keeps b * nr inside 64 bits in the kernel
    (void)hipGetLastError();
    const unsigned grid = (unsigned)(n < (int64_t(1) << 30) ? n : (int64_t(1) << 30));
    hipLaunchKernelGGL(tkv::mixed_traffic_kernel, dim3(grid), dim3(tkv::kThreads), 0, (hipStream_t)stream, p, d_slots,
                       num_read_slots, nw, nr, fill);
    return hipGetLastError() == hipSuccess ? KV_OK : KV_EHIP;
}

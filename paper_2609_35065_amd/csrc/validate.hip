// validate.hip -- the job-batch check of kv_validate_jobs on the device, for
// job lists that are already in device memory (no copy back to the host).
//
// Within one copy launch the only writes that can race are two jobs naming
// one destination: a paged block in the scatter (a job writes the same block
// id in both planes of every layer), a staging slot in the gather.  Every
// (job, segment) is checked by one lane; a valid destination is marked in a
// caller-provided array with an atomic OR, and a lane that finds its mark
// already set has found a duplicate.  Range errors decide over duplicates, as
// in the host check, so the outcome does not depend on the order of the jobs.

#include "internal.h"

namespace tkv {
namespace {

constexpr int kThreads = 256;
constexpr int64_t kMaxBlocks = int64_t(1) << 16;

struct ValidateParams {
    const kv_job *jobs;
    const int32_t *bt;
    int32_t *flags;   // [0]: a range error, [1]: a duplicate destination
    int32_t *marks;   // one word per block (scatter) or slot (gather)
    int64_t num_jobs;
    int64_t num_blocks;
    int64_t num_slots;
    int32_t bt_stride;
    int32_t num_reqs;
    int32_t nseg;
    int32_t is_store;
};

// Zero n words: the flags and the marks (a kernel rather than a memset, so
// that the call can be recorded in a graph).
__global__ __launch_bounds__(kThreads) void validate_clear_kernel(int32_t *words, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
        words[i] = 0;
}

__global__ __launch_bounds__(kThreads) void validate_mark_kernel(ValidateParams p) {
    const int64_t total = p.num_jobs * p.nseg;
    for (int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x; t < total; t += (int64_t)gridDim.x * kThreads) {
        const int64_t q = t / p.nseg;
        const int32_t i = (int32_t)(t % p.nseg);
        const kv_job jb = p.jobs[q];
        if (jb.reserved != 0 || jb.slot < 0 || jb.slot >= p.num_slots || jb.req < 0 || jb.req >= p.num_reqs ||
            jb.chunk < 0 || ((int64_t)jb.chunk + 1) * p.nseg > p.bt_stride) {
            p.flags[0] = 1;
            continue;
        }
        const int32_t blk = p.bt[(int64_t)jb.req * p.bt_stride + (int64_t)jb.chunk * p.nseg + i];
        if (blk < 0 || blk >= p.num_blocks) {
            p.flags[0] = 1;
            continue;
        }
        // the gather's destination is the job's slot: marked once per job, by its segment-0 lane
        const int64_t dest = p.is_store ? (i == 0 ? jb.slot : -1) : blk;
        if (dest >= 0 && (atomicOr(&p.marks[dest], 1) & 1)) p.flags[1] = 1;
    }
}

__global__ __launch_bounds__(64) void validate_status_kernel(const int32_t *flags, int32_t *status) {
    if (threadIdx.x == 0) *status = flags[0] ? KV_ERANGE : (flags[1] ? KV_EDUP : KV_OK);
}

unsigned blocks_for(int64_t items) {
    const int64_t b = (items + kThreads - 1) / kThreads;
    return (unsigned)(b < 1 ? 1 : (b < kMaxBlocks ? b : kMaxBlocks));
}

}  // namespace
}  // namespace tkv

extern "C" {

int kv_validate_jobs_device(const kv_layout *layout, const int32_t *d_block_tables, int32_t bt_stride,
                            int32_t num_reqs, const kv_job *d_jobs, int32_t num_jobs, int is_store,
                            int32_t *d_marks, int32_t *d_status, void *stream) {
    const int rc = tkv::check_layout(layout);
    if (rc != KV_OK) return rc;
    if (num_jobs < 0 || num_reqs < 0 || bt_stride <= 0 || !d_marks || !d_status) return KV_EINVAL;
    if (num_jobs > 0 && (!d_block_tables || !d_jobs)) return KV_EINVAL;
    if (((uintptr_t)d_jobs & 15u) || ((uintptr_t)d_marks & 3u) || ((uintptr_t)d_status & 3u) ||
        ((uintptr_t)d_block_tables & 3u))
        return KV_EALIGN;
    tkv::ValidateParams p;
    p.jobs = d_jobs;
    p.bt = d_block_tables;
    p.flags = d_marks;
    p.marks = d_marks + 2;
    p.num_jobs = num_jobs;
    p.num_blocks = layout->num_blocks;
    p.num_slots = layout->num_slots;
    p.bt_stride = bt_stride;
    p.num_reqs = num_reqs;
    p.nseg = layout->chunk_tokens / layout->block_size;
    p.is_store = is_store ? 1 : 0;
    const int64_t words = 2 + (is_store ? layout->num_slots : layout->num_blocks);
    hipStream_t s = (hipStream_t)stream;
    (void)hipGetLastError();
    hipLaunchKernelGGL(tkv::validate_clear_kernel, dim3(tkv::blocks_for(words)), dim3(tkv::kThreads), 0, s, d_marks,
                       words);
    if (num_jobs > 0)
        hipLaunchKernelGGL(tkv::validate_mark_kernel, dim3(tkv::blocks_for((int64_t)num_jobs * p.nseg)),
                           dim3(tkv::kThreads), 0, s, p);
    hipLaunchKernelGGL(tkv::validate_status_kernel, dim3(1), dim3(64), 0, s, (const int32_t *)d_marks, d_status);
    return hipGetLastError() == hipSuccess ? KV_OK : KV_EHIP;
}

}  // extern "C"

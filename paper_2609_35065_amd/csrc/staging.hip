// staging.hip -- staging chunks from a lower tier in pinned host memory into
// the HBM staging buffer (the fast tier), and the stage-ready-gated retrieve
// that overlaps those copies with the scatter.
//
// The copies go to the DMA engines (hipMemcpyAsync), leaving the compute
// units to the scatter.  The scatter of a batch of jobs waits, on the compute
// stream, for an event recorded on the copy stream after the batch's chunks
// were copied: an event is the batch's stage-ready flag, so retrieval begins
// only once the matched KV is in the fast tier, while the copy of the next
// batch proceeds.

#include <algorithm>
#include <new>
#include <vector>

#include "internal.h"

struct kv_pipeline {
    int device = 0;
    std::vector<hipEvent_t> ev;
};

namespace {

int64_t slot_bytes_of(const kv_layout *lo) {
    return (int64_t)lo->block_size * lo->kv_heads * lo->head_dim * lo->elem_bytes * (lo->chunk_tokens / lo->block_size) *
           2 * lo->num_layers;
}

// DMA copies of the given slots between two buffers of the same slot layout,
// one per run of consecutive slot ids.
int copy_slots(const kv_layout *lo, char *dst, const char *src, const int32_t *slots, int32_t n, hipMemcpyKind kind,
               hipStream_t stream) {
    const int64_t sb = slot_bytes_of(lo);
    int32_t i = 0;
    while (i < n) {
        int32_t j = i + 1;
        while (j < n && slots[j] == slots[j - 1] + 1) ++j;
        const int64_t off = (int64_t)slots[i] * sb;
        if (hipMemcpyAsync(dst + off, src + off, (size_t)((j - i) * sb), kind, stream) != hipSuccess) return KV_EHIP;
        i = j;
    }
    return KV_OK;
}

int check_slots(const kv_layout *lo, const void *a, const void *b, const int32_t *slots, int32_t n) {
    const int rc = tkv::check_layout(lo);
    if (rc != KV_OK) return rc;
    if (n < 0 || (n > 0 && (!a || !b || !slots))) return KV_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        if (slots[i] < 0 || slots[i] >= lo->num_slots) return KV_ERANGE;
    return KV_OK;
}

}  // namespace

extern "C" {

int kv_stage_in(const kv_layout *layout, const void *h_lower_tier, void *d_staging, const int32_t *h_slots,
                int32_t n, void *stream) {
    const int rc = check_slots(layout, h_lower_tier, d_staging, h_slots, n);
    if (rc != KV_OK) return rc;
    return copy_slots(layout, (char *)d_staging, (const char *)h_lower_tier, h_slots, n, hipMemcpyHostToDevice,
                      (hipStream_t)stream);
}

int kv_stage_out(const kv_layout *layout, const void *d_staging, void *h_lower_tier, const int32_t *h_slots,
                 int32_t n, void *stream) {
    const int rc = check_slots(layout, h_lower_tier, d_staging, h_slots, n);
    if (rc != KV_OK) return rc;
    return copy_slots(layout, (char *)h_lower_tier, (const char *)d_staging, h_slots, n, hipMemcpyDeviceToHost,
                      (hipStream_t)stream);
}

int kv_pipeline_create(int32_t max_batches, kv_pipeline **out) {
    if (!out || max_batches <= 0 || max_batches > 65536) return KV_EINVAL;
    *out = nullptr;
    kv_pipeline *pl = new (std::nothrow) kv_pipeline();
    if (!pl) return KV_EINVAL;
    if (hipGetDevice(&pl->device) != hipSuccess) {
        delete pl;
        return KV_EHIP;
    }
    pl->ev.assign(max_batches, nullptr);
    for (auto &e : pl->ev)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
            kv_pipeline_destroy(pl);
            return KV_EHIP;
        }
    *out = pl;
    return KV_OK;
}

int kv_pipeline_destroy(kv_pipeline *pl) {
    if (!pl) return KV_EINVAL;
    for (hipEvent_t e : pl->ev)
        if (e) {
            (void)hipEventSynchronize(e);
            (void)hipEventDestroy(e);
        }
    delete pl;
    return KV_OK;
}

int kv_retrieve_pipelined(kv_pipeline *pl, const kv_layout *layout, const void *h_lower_tier, void *d_staging,
                          void *const *h_layer_ptrs, const int32_t *d_block_tables, int32_t bt_stride,
                          int32_t num_reqs, const kv_job *h_jobs, const kv_job *d_jobs, int32_t num_jobs,
                          int32_t slots_per_batch, void *copy_stream, void *stream) {
    if (!pl || slots_per_batch <= 0) return KV_EINVAL;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return KV_EHIP;
    if (dev != pl->device) return KV_EINVAL;
    tkv::CopyParams p;
    int rc = tkv::make_copy_params(p, layout, d_staging, (const void *const *)h_layer_ptrs, d_block_tables, bt_stride,
                                   num_reqs, d_jobs, num_jobs);
    if (rc != KV_OK) return rc;
    if (num_jobs == 0) return KV_OK;
    if (!h_jobs || !h_lower_tier) return KV_EINVAL;
    // distinct slot runs (the jobs are grouped by slot); every slot must exist
    int64_t runs = 0;
    for (int32_t q = 0; q < num_jobs; ++q) {
        if (h_jobs[q].slot < 0 || h_jobs[q].slot >= layout->num_slots) return KV_ERANGE;
        if (q == 0 || h_jobs[q].slot != h_jobs[q - 1].slot) ++runs;
    }
    const int64_t nev = (int64_t)pl->ev.size();
    const int64_t spb = std::max<int64_t>(slots_per_batch, (runs + nev - 1) / nev);
    std::vector<int32_t> slots;
    slots.reserve((size_t)std::min<int64_t>(spb, runs));
    int32_t q0 = 0;
    for (int64_t b = 0; q0 < num_jobs; ++b) {
        slots.clear();
        int32_t q1 = q0;
        while (q1 < num_jobs) {
            if (q1 == q0 || h_jobs[q1].slot != h_jobs[q1 - 1].slot) {
                if ((int64_t)slots.size() == spb) break;
                slots.push_back(h_jobs[q1].slot);
            }
            ++q1;
        }
        const int kind = kv_retrieve_plan(layout, h_jobs + q0, q1 - q0);
        std::sort(slots.begin(), slots.end());
        slots.erase(std::unique(slots.begin(), slots.end()), slots.end());
        rc = copy_slots(layout, (char *)d_staging, (const char *)h_lower_tier, slots.data(), (int32_t)slots.size(),
                        hipMemcpyHostToDevice, (hipStream_t)copy_stream);
        if (rc != KV_OK) return rc;
        if (hipEventRecord(pl->ev[b], (hipStream_t)copy_stream) != hipSuccess ||
            hipStreamWaitEvent((hipStream_t)stream, pl->ev[b], 0) != hipSuccess)
            return KV_EHIP;
        tkv::CopyParams pb = p;
        pb.jobs = d_jobs + q0;
        pb.num_jobs = q1 - q0;
        pb.total_segs = (int64_t)pb.num_jobs * p.L * 2 * p.nseg;
        const tkv::CopyKind ck = kind == KV_RETRIEVE_STREAM ? tkv::kRetrieveStream
                                 : kind == KV_RETRIEVE_PAIR ? tkv::kRetrievePair
                                                            : tkv::kRetrieve;
        if (tkv::launch_copy(pb, ck, (hipStream_t)stream) != hipSuccess) return KV_EHIP;
        q0 = q1;
    }
    return KV_OK;
}

}  // extern "C"

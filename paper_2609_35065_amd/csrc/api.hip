// api.hip -- the C ABI of the GPU calls: argument checks and launch set-up
// of the hash, lookup and copies.  The host-only calls are in host.cpp.

#include <string.h>

#include "internal.h"

namespace {

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

namespace tkv {

// Launch parameters of one copy call, after every argument check.
int make_copy_params(CopyParams &p, const kv_layout *lo, const void *staging, const void *const *layers,
                     const int32_t *bt, int32_t bt_stride, int32_t num_reqs, const kv_job *jobs,
                     int32_t num_jobs) {
    int rc = check_layout(lo);
    if (rc != KV_OK) return rc;
    if (num_jobs < 0 || num_reqs < 0 || bt_stride <= 0) return KV_EINVAL;
    if (!staging || !layers || !bt || (num_jobs > 0 && !jobs)) return KV_EINVAL;
    if (!aligned16(staging)) return KV_EALIGN;
    memset(&p, 0, sizeof(p));
    for (int l = 0; l < lo->num_layers; ++l) {
        if (!layers[l]) return KV_EINVAL;
        if (!aligned16(layers[l])) return KV_EALIGN;
        p.layers[l] = (char *)layers[l];
    }
    const int32_t nseg = lo->chunk_tokens / lo->block_size;
    p.staging = (char *)staging;
    p.bt = bt;
    p.jobs = jobs;
    p.seg_bytes = (int64_t)lo->block_size * lo->kv_heads * lo->head_dim * lo->elem_bytes;
    p.slot_bytes = p.seg_bytes * nseg * 2 * lo->num_layers;
    p.kv_stride = lo->paged_kv_stride;
    p.block_stride = lo->paged_block_stride;
    p.num_blocks = lo->num_blocks;
    p.num_slots = lo->num_slots;
    p.L = lo->num_layers;
    p.nseg = nseg;
    p.bt_stride = bt_stride;
    p.num_reqs = num_reqs;
    p.num_jobs = num_jobs;
    p.total_segs = (int64_t)num_jobs * lo->num_layers * 2 * nseg;
    return KV_OK;
}

}  // namespace tkv

using tkv::check_layout;
using tkv::make_copy_params;

extern "C" {

int kv_hash_prefix(const int32_t *d_tokens, const int64_t *d_tok_off, int32_t num_reqs, uint64_t seed,
                   const int64_t *d_blk_off, uint64_t *d_block_hash, void *stream) {
    if (num_reqs < 0) return KV_EINVAL;
    if (num_reqs == 0) return KV_OK;
    if (!d_tokens || !d_tok_off || !d_blk_off || !d_block_hash) return KV_EINVAL;
    return tkv::launch_hash(d_tokens, d_tok_off, num_reqs, seed, d_blk_off, d_block_hash, (hipStream_t)stream) ==
                   hipSuccess
               ? KV_OK
               : KV_EHIP;
}

int kv_lookup(const kv_index *idx, const uint64_t *d_block_hash, const int64_t *d_blk_off, int32_t num_reqs,
              int32_t blocks_per_chunk, const int64_t *d_chunk_off, int32_t *d_chunk_slot, int32_t *d_hit_chunks,
              void *stream) {
    if (!idx || num_reqs < 0 || blocks_per_chunk <= 0) return KV_EINVAL;
    if (num_reqs == 0) return KV_OK;
    if (!d_block_hash || !d_blk_off || !d_chunk_off || !d_chunk_slot || !d_hit_chunks) return KV_EINVAL;
    int log2cap = 0;
    const tkv::IndexEntry *table = tkv::index_device_table(idx, &log2cap);
    return tkv::launch_lookup(table, log2cap, d_block_hash, d_blk_off, num_reqs, blocks_per_chunk, d_chunk_off,
                              d_chunk_slot, d_hit_chunks, (hipStream_t)stream) == hipSuccess
               ? KV_OK
               : KV_EHIP;
}

int kv_retrieve_scatter(const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                        const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs, const kv_job *d_jobs,
                        int32_t num_jobs, void *stream) {
    tkv::CopyParams p;
    const int rc = make_copy_params(p, layout, d_staging, (const void *const *)h_layer_ptrs, d_block_tables,
                                    bt_stride, num_reqs, d_jobs, num_jobs);
    if (rc != KV_OK) return rc;
    return tkv::launch_copy(p, tkv::kRetrieve, (hipStream_t)stream) == hipSuccess ? KV_OK : KV_EHIP;
}

int kv_retrieve_scatter_as(int32_t kind, const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                           const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs, const kv_job *d_jobs,
                           int32_t num_jobs, void *stream) {
    tkv::CopyKind k;
    switch (kind) {
    case KV_RETRIEVE_UNIT: k = tkv::kRetrieve; break;
    case KV_RETRIEVE_PAIR: k = tkv::kRetrievePair; break;
    case KV_RETRIEVE_STREAM: k = tkv::kRetrieveStream; break;
    case KV_RETRIEVE_QUAD: k = tkv::kRetrieveQuad; break;
    default: return KV_EINVAL;
    }
    tkv::CopyParams p;
    const int rc = make_copy_params(p, layout, d_staging, (const void *const *)h_layer_ptrs, d_block_tables,
                                    bt_stride, num_reqs, d_jobs, num_jobs);
    if (rc != KV_OK) return rc;
    return tkv::launch_copy(p, k, (hipStream_t)stream) == hipSuccess ? KV_OK : KV_EHIP;
}

int kv_store_gather(const kv_layout *layout, void *d_staging, const void *const *h_layer_ptrs,
                    const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs, const kv_job *d_jobs,
                    int32_t num_jobs, void *stream) {
    tkv::CopyParams p;
    const int rc = make_copy_params(p, layout, d_staging, h_layer_ptrs, d_block_tables, bt_stride, num_reqs,
                                    d_jobs, num_jobs);
    if (rc != KV_OK) return rc;
    return tkv::launch_copy(p, tkv::kStore, (hipStream_t)stream) == hipSuccess ? KV_OK : KV_EHIP;
}

int kv_host_device_pointer(const void *h_ptr, void **d_ptr_out) {
    if (!h_ptr || !d_ptr_out) return KV_EINVAL;
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, const_cast<void *>(h_ptr), 0) != hipSuccess) {
        (void)hipGetLastError();
        return KV_EHIP;
    }
    *d_ptr_out = d;
    return KV_OK;
}

}  // extern "C"

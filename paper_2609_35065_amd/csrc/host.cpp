// host.cpp -- the host-only calls of the C ABI: layout checks, the retrieve
// planner, host job build, job validation and the commitment rule.  Plain
// C++ with no HIP header, so that it can also be built and tested on its own
// (for instance under the address and undefined-behaviour sanitizers).

#include <math.h>

#include <algorithm>
#include <unordered_set>
#include <vector>

#include "host.h"

namespace tkv {

// Layout checks shared by the copy directions and staging.
int check_layout(const kv_layout *lo) {
    if (!lo) return KV_EINVAL;
    if (lo->num_layers <= 0 || lo->num_layers > KV_MAX_LAYERS || lo->kv_heads <= 0 || lo->head_dim <= 0 ||
        lo->block_size <= 0 || lo->chunk_tokens <= 0 || lo->num_blocks <= 0 || lo->num_slots <= 0)
        return KV_EINVAL;
    if (lo->elem_bytes != 1 && lo->elem_bytes != 2 && lo->elem_bytes != 4) return KV_EINVAL;
    if (lo->chunk_tokens % lo->block_size != 0) return KV_EINVAL;
    const int64_t seg = (int64_t)lo->block_size * lo->kv_heads * lo->head_dim * lo->elem_bytes;
    if (seg > (int64_t(1) << 40)) return KV_EINVAL;
    if (lo->paged_kv_stride <= 0 || lo->paged_block_stride <= 0) return KV_EINVAL;
    if (lo->paged_block_stride < seg || lo->paged_kv_stride < seg) return KV_EINVAL;
    if (seg % 16 != 0 || lo->paged_kv_stride % 16 != 0 || lo->paged_block_stride % 16 != 0) return KV_EALIGN;
    // slot_bytes * num_slots must stay well inside int64
    const int64_t slot = seg * (lo->chunk_tokens / lo->block_size) * 2 * lo->num_layers;
    if (slot <= 0 || lo->num_slots > (int64_t(1) << 62) / slot) return KV_EINVAL;
    return KV_OK;
}

}  // namespace tkv

using tkv::check_layout;

extern "C" {

int kv_retrieve_plan(const kv_layout *layout, const kv_job *h_jobs, int32_t num_jobs) {
    const int rc = check_layout(layout);
    if (rc != KV_OK) return rc;
    if (num_jobs < 0 || (num_jobs > 0 && !h_jobs)) return KV_EINVAL;
    if (num_jobs == 0) return KV_RETRIEVE_UNIT;
    int64_t runs = 0, pairs_shared = 0;
    for (int32_t i = 0; i < num_jobs; ++i) {
        if (i == 0 || h_jobs[i].slot != h_jobs[i - 1].slot) ++runs;
        if ((i & 1) && h_jobs[i].slot == h_jobs[i - 1].slot) ++pairs_shared;
    }
    if (runs == num_jobs) {
        // no slot twice in a row; streaming needs every slot once
        std::unordered_set<int32_t> seen;
        seen.reserve((size_t)num_jobs * 2);
        bool distinct = true;
        for (int32_t i = 0; i < num_jobs && distinct; ++i) distinct = seen.insert(h_jobs[i].slot).second;
        if (distinct) return KV_RETRIEVE_STREAM;
    }
    // Pairs pay off when most pairs share their chunk and groups are small
    // (many groups in flight per XCD); measured at 32 KiB segments.
    const int64_t seg = (int64_t)layout->block_size * layout->kv_heads * layout->head_dim * layout->elem_bytes;
    if (seg == 32768 && 20 * pairs_shared >= 9 * (int64_t)num_jobs && num_jobs <= 16 * runs)
        return KV_RETRIEVE_PAIR;
    return KV_RETRIEVE_UNIT;
}

}  // extern "C"

namespace {

// Shared body of kv_build_jobs and kv_build_jobs_routed.  A request takes
// part when `requested` is null or requested[r] != 0; its matched chunks go to
// `ordinary` when decision[r] == KV_ORDINARY (and `ordinary` is given), else
// to `retrieve`.
int build_jobs(const int32_t *hit_chunks, const int32_t *chunk_slot, const uint64_t *block_hash,
               const int64_t *blk_off, const int64_t *chunk_off, int32_t num_reqs, int32_t bpc,
               const int32_t *free_slots, int32_t num_free, const uint8_t *requested, const int32_t *decision,
               kv_job *retrieve, int32_t *num_retrieve, kv_job *ordinary, int32_t *num_ordinary, kv_job *store,
               uint64_t *store_keys, int32_t *num_store, int32_t *dropped) {
    if (num_reqs < 0 || bpc <= 0 || num_free < 0) return KV_EINVAL;
    if (!num_retrieve || !num_store || !dropped) return KV_EINVAL;
    *num_retrieve = *num_store = *dropped = 0;
    if (num_ordinary) *num_ordinary = 0;
    if (num_reqs == 0) return KV_OK;
    if (!hit_chunks || !chunk_slot || !block_hash || !blk_off || !chunk_off || !retrieve || !store || !store_keys ||
        (num_free > 0 && !free_slots))
        return KV_EINVAL;
    for (int32_t r = 0; r < num_reqs; ++r) {
        const int64_t nb = blk_off[r + 1] - blk_off[r];
        const int64_t nc = chunk_off[r + 1] - chunk_off[r];
        if (nb < 0 || nc != nb / bpc || hit_chunks[r] < 0 || hit_chunks[r] > nc) return KV_EINVAL;
        if (decision && (!requested || requested[r]) && decision[r] != KV_COMMIT && decision[r] != KV_ORDINARY)
            return KV_EINVAL;
    }
    std::unordered_set<uint64_t> missing;   // distinct missing keys met so far
    int32_t nr = 0, no = 0, ns = 0, nd = 0;
    for (int32_t r = 0; r < num_reqs; ++r) {
        if (requested && !requested[r]) continue;
        const int64_t c0 = chunk_off[r];
        const int64_t nc = chunk_off[r + 1] - c0;
        const int32_t hit = hit_chunks[r];
        const bool ord = decision && decision[r] == KV_ORDINARY;
        for (int32_t j = 0; j < hit; ++j) {
            if (ord) ordinary[no++] = kv_job{chunk_slot[c0 + j], r, j, 0};
            else retrieve[nr++] = kv_job{chunk_slot[c0 + j], r, j, 0};
        }
        for (int64_t j = hit; j < nc; ++j) {
            if (chunk_slot[c0 + j] >= 0) continue;
            const uint64_t key = block_hash[blk_off[r] + (j + 1) * bpc - 1];
            if (!missing.insert(key).second) continue;
            if (ns >= num_free) {
                ++nd;
                continue;
            }
            store_keys[ns] = key;
            store[ns] = kv_job{free_slots[ns], r, (int32_t)j, 0};
            ++ns;
        }
    }
    *num_retrieve = nr;
    if (num_ordinary) *num_ordinary = no;
    *num_store = ns;
    *dropped = nd;
    return nd > 0 ? KV_ENOSPC : KV_OK;
}

}  // namespace

extern "C" {

int kv_build_jobs(const int32_t *h_hit_chunks, const int32_t *h_chunk_slot, const uint64_t *h_block_hash,
                  const int64_t *h_blk_off, const int64_t *h_chunk_off, int32_t num_reqs, int32_t blocks_per_chunk,
                  const int32_t *h_free_slots, int32_t num_free, kv_job *h_retrieve, int32_t *num_retrieve,
                  kv_job *h_store, uint64_t *h_store_keys, int32_t *num_store, int32_t *dropped) {
    return build_jobs(h_hit_chunks, h_chunk_slot, h_block_hash, h_blk_off, h_chunk_off, num_reqs, blocks_per_chunk,
                      h_free_slots, num_free, nullptr, nullptr, h_retrieve, num_retrieve, nullptr, nullptr, h_store,
                      h_store_keys, num_store, dropped);
}

int kv_chunk_keys(const uint64_t *h_block_hash, const int64_t *h_blk_off, int32_t num_reqs, int32_t blocks_per_chunk,
                  const int64_t *h_chunk_off, uint64_t *h_keys) {
    if (num_reqs < 0 || blocks_per_chunk <= 0) return KV_EINVAL;
    if (num_reqs == 0) return KV_OK;
    if (!h_block_hash || !h_blk_off || !h_chunk_off || !h_keys) return KV_EINVAL;
    for (int32_t r = 0; r < num_reqs; ++r) {
        const int64_t nb = h_blk_off[r + 1] - h_blk_off[r];
        const int64_t nc = h_chunk_off[r + 1] - h_chunk_off[r];
        if (nb < 0 || nc != nb / blocks_per_chunk) return KV_EINVAL;
        for (int64_t j = 0; j < nc; ++j)
            h_keys[h_chunk_off[r] + j] = h_block_hash[h_blk_off[r] + (j + 1) * blocks_per_chunk - 1];
    }
    return KV_OK;
}

int kv_decide_claims(int32_t num_reqs, const int32_t *h_hit_chunks, const int32_t *h_chunk_slot,
                     const int64_t *h_chunk_off, const double *h_ttu, const double *h_ttr,
                     const uint8_t *h_requested, uint64_t slot_bytes, uint64_t budget_bytes, int64_t num_slots,
                     uint8_t *h_protected, uint64_t *reserved_bytes, int32_t *h_decision) {
    if (num_reqs < 0 || num_slots <= 0 || !reserved_bytes) return KV_EINVAL;
    if (num_reqs == 0) return KV_OK;
    if (!h_hit_chunks || !h_chunk_slot || !h_chunk_off || !h_ttu || !h_ttr || !h_requested || !h_protected ||
        !h_decision)
        return KV_EINVAL;
    for (int32_t r = 0; r < num_reqs; ++r) {
        const int64_t nc = h_chunk_off[r + 1] - h_chunk_off[r];
        if (nc < 0 || h_hit_chunks[r] < 0 || h_hit_chunks[r] > nc) return KV_EINVAL;
        for (int32_t j = 0; j < h_hit_chunks[r]; ++j) {
            const int32_t s = h_chunk_slot[h_chunk_off[r] + j];
            if (s < 0 || s >= num_slots) return KV_ERANGE;
        }
    }
    // claims with a pending retrieval request first, then the others, each in request order
    std::vector<int32_t> order;
    order.reserve((size_t)num_reqs);
    for (int pass = 0; pass < 2; ++pass)
        for (int32_t r = 0; r < num_reqs; ++r)
            if ((h_requested[r] != 0) == (pass == 0)) order.push_back(r);
    std::unordered_set<int32_t> objs;
    for (int32_t r : order) {
        // the claim's KV objects: the distinct slots of its matched chunks
        objs.clear();
        uint64_t total = 0, fresh = 0;
        for (int32_t j = 0; j < h_hit_chunks[r]; ++j) {
            const int32_t s = h_chunk_slot[h_chunk_off[r] + j];
            if (!objs.insert(s).second) continue;
            total += slot_bytes;
            if (!h_protected[s]) fresh += slot_bytes;
        }
        const uint64_t free_bytes = budget_bytes > *reserved_bytes ? budget_bytes - *reserved_bytes : 0;
        const int d = kv_commit_should_stage(h_ttu[r], h_ttr[r], free_bytes, fresh, total, budget_bytes,
                                             h_requested[r] != 0);
        h_decision[r] = d;
        if (d == KV_COMMIT) {
            for (int32_t s : objs) h_protected[s] = 1;
            *reserved_bytes += fresh;
        }
    }
    return KV_OK;
}

int kv_build_jobs_routed(const int32_t *h_hit_chunks, const int32_t *h_chunk_slot, const uint64_t *h_block_hash,
                         const int64_t *h_blk_off, const int64_t *h_chunk_off, int32_t num_reqs,
                         int32_t blocks_per_chunk, const int32_t *h_free_slots, int32_t num_free,
                         const uint8_t *h_requested, const int32_t *h_decision, kv_job *h_retrieve,
                         int32_t *num_retrieve, kv_job *h_ordinary, int32_t *num_ordinary, kv_job *h_store,
                         uint64_t *h_store_keys, int32_t *num_store, int32_t *dropped) {
    if (num_reqs > 0 && (!h_requested || !h_decision || !h_ordinary)) return KV_EINVAL;
    if (!num_ordinary) return KV_EINVAL;
    return build_jobs(h_hit_chunks, h_chunk_slot, h_block_hash, h_blk_off, h_chunk_off, num_reqs, blocks_per_chunk,
                      h_free_slots, num_free, h_requested, h_decision, h_retrieve, num_retrieve, h_ordinary,
                      num_ordinary, h_store, h_store_keys, num_store, dropped);
}

int kv_group_jobs_by_slot(kv_job *h_jobs, int32_t num_jobs) {
    if (num_jobs < 0 || (num_jobs > 0 && !h_jobs)) return KV_EINVAL;
    std::stable_sort(h_jobs, h_jobs + num_jobs, [](const kv_job &a, const kv_job &b) { return a.slot < b.slot; });
    return KV_OK;
}

int kv_validate_jobs(const kv_layout *layout, const int32_t *h_block_tables, int32_t bt_stride, int32_t num_reqs,
                     const kv_job *h_jobs, int32_t num_jobs, int is_store) {
    int rc = check_layout(layout);
    if (rc != KV_OK) return rc;
    if (num_jobs < 0 || num_reqs < 0 || bt_stride <= 0) return KV_EINVAL;
    if (num_jobs == 0) return KV_OK;
    if (!h_block_tables || !h_jobs) return KV_EINVAL;
    const int32_t nseg = layout->chunk_tokens / layout->block_size;
    std::vector<uint8_t> seen(is_store ? (size_t)layout->num_slots : (size_t)layout->num_blocks, 0);
    for (int32_t q = 0; q < num_jobs; ++q) {
        const kv_job &jb = h_jobs[q];
        if (jb.reserved != 0 || jb.slot < 0 || jb.slot >= layout->num_slots || jb.req < 0 || jb.req >= num_reqs ||
            jb.chunk < 0 || ((int64_t)jb.chunk + 1) * nseg > bt_stride)
            return KV_ERANGE;
        for (int32_t i = 0; i < nseg; ++i) {
            const int32_t blk = h_block_tables[(int64_t)jb.req * bt_stride + (int64_t)jb.chunk * nseg + i];
            if (blk < 0 || blk >= layout->num_blocks) return KV_ERANGE;
        }
    }
    for (int32_t q = 0; q < num_jobs; ++q) {
        const kv_job &jb = h_jobs[q];
        if (is_store) {
            if (seen[jb.slot]++) return KV_EDUP;
        } else {
            for (int32_t i = 0; i < nseg; ++i) {
                const int32_t blk = h_block_tables[(int64_t)jb.req * bt_stride + (int64_t)jb.chunk * nseg + i];
                if (seen[blk]++) return KV_EDUP;
            }
        }
    }
    return KV_OK;
}

int kv_commit_should_stage(double ttu_s, double ttr_s, uint64_t free_protected_bytes, uint64_t claim_new_bytes,
                           uint64_t claim_total_bytes, uint64_t budget_bytes, int retrieval_requested) {
    if (isnan(ttu_s) || isnan(ttr_s) || claim_new_bytes > claim_total_bytes) return KV_EINVAL;
    const bool eligible = ttu_s <= ttr_s || retrieval_requested != 0;
    if (!eligible) return KV_DEFER;
    const bool fits = claim_total_bytes <= budget_bytes && claim_new_bytes <= free_protected_bytes;
    if (fits) return KV_COMMIT;
    return retrieval_requested ? KV_ORDINARY : KV_BLOCKED;
}

int kv_commit_should_stage_n(int32_t n, const double *h_ttu, const double *h_ttr, uint64_t free_protected_bytes,
                             const uint64_t *h_claim_new, const uint64_t *h_claim_total, uint64_t budget_bytes,
                             const uint8_t *h_requested, int32_t *h_out) {
    if (n < 0) return KV_EINVAL;
    if (n > 0 && (!h_ttu || !h_ttr || !h_claim_new || !h_claim_total || !h_requested || !h_out)) return KV_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        h_out[i] = kv_commit_should_stage(h_ttu[i], h_ttr[i], free_protected_bytes, h_claim_new[i], h_claim_total[i],
                                          budget_bytes, h_requested[i] != 0);
    return KV_OK;
}

const char *kv_strerror(int status) {
    switch (status) {
    case KV_OK: return "ok";
    case KV_EINVAL: return "invalid argument";
    case KV_EALIGN: return "pointer or stride not 16-byte aligned";
    case KV_ERANGE: return "slot, request, chunk or block id out of range";
    case KV_ENOSPC: return "no free staging slot or index full";
    case KV_EHIP: return "HIP runtime error";
    case KV_EDUP: return "duplicate destination within one batch";
    case KV_ELIMIT: return "request exceeds a fixed capacity of the allocation-free call";
    default: return "unknown status";
    }
}

const char *kv_version(void) { return "tempokv 0.1.0 gfx950"; }

}  // extern "C"

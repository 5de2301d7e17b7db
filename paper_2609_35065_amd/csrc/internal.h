// internal.h -- private declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "host.h"
#include "index_table.h"
#include "tempokv.h"

namespace tkv {

// Everything the copy kernels need, passed by value in the kernel-argument
// segment so that the per-layer base pointers are read with scalar loads and
// no device-side descriptor has to be allocated or uploaded.
struct CopyParams {
    char *staging;
    char *layers[KV_MAX_LAYERS];
    const int32_t *bt;
    const kv_job *jobs;
    int64_t slot_bytes;
    int64_t seg_bytes;
    int64_t kv_stride;
    int64_t block_stride;
    int64_t num_blocks;
    int64_t num_slots;
    int64_t total_segs;     // num_jobs * L * 2 * nseg
    int32_t L;
    int32_t nseg;           // C / B
    int32_t bt_stride;
    int32_t num_reqs;
    int32_t num_jobs;
};

// Which copy a launch performs.  The retrieve kinds move the same bytes:
// kRetrieve walks one (job, layer, plane) unit per workgroup, reading staged
// units through the caches; kRetrievePair walks pairs of jobs and reads a
// unit once for two jobs that share it; kRetrieveStream streams the staged
// units with non-temporal loads in the store's workgroup shape, for job lists
// that read each chunk once; kRetrieveQuad copies one segment of four
// consecutive jobs per 1024-lane workgroup.
enum CopyKind { kRetrieve, kRetrievePair, kRetrieveStream, kRetrieveQuad, kStore };

// Launchers (copy.hip, hash.hip).  Return hipSuccess or the launch error.
hipError_t launch_copy(const CopyParams &p, CopyKind kind, hipStream_t stream);
hipError_t launch_hash(const int32_t *tokens, const int64_t *tok_off, int32_t num_reqs, uint64_t seed,
                       const int64_t *blk_off, uint64_t *out, hipStream_t stream);
hipError_t launch_lookup(const IndexEntry *table, int log2cap, const uint64_t *block_hash,
                         const int64_t *blk_off, int32_t num_reqs, int32_t bpc, const int64_t *chunk_off,
                         int32_t *chunk_slot, int32_t *hit_chunks, hipStream_t stream);

// Launch parameters shared by the copy entry points (api.hip), after every
// argument check.  Returns KV_OK or a negative kv_status.
int make_copy_params(CopyParams &p, const kv_layout *lo, const void *staging, const void *const *layers,
                     const int32_t *bt, int32_t bt_stride, int32_t num_reqs, const kv_job *jobs, int32_t num_jobs);

// Device table of an index, for kv_lookup (index.hip).
const IndexEntry *index_device_table(const kv_index *idx, int *log2cap);

}  // namespace tkv

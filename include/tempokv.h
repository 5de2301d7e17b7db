/*
 * tempokv.h -- C ABI of the TempoKV staging hot path on MI355X (gfx950).
 *
 * TempoKV (Park, Kim, Kim; "TempoKV: Timely Staging of LLM KV Caches for
 * Memory-Semantic Flash") decides when to commit staging of reusable prefix
 * KV.  Underneath its staging layer sit a prefix lookup and a fast-tier-to-GPU
 * transfer that the paper reuses unchanged (Section 4, "Runtime and
 * controller integration").  This library is that data path, MI355X-native:
 *
 *   kv_hash_prefix        chained 64-bit hash of token ids over 16-token blocks
 *   kv_lookup             prefix match of chunk keys against a staged-chunk index
 *   kv_build_jobs         host job build: hits -> retrieve jobs, misses -> store jobs
 *   kv_retrieve_scatter   staged chunk [L,2,C,H,D] -> paged KV blocks (one launch;
 *                         kv_retrieve_plan / kv_retrieve_scatter_as pick a variant)
 *   kv_store_gather       paged KV blocks -> staged chunk (one launch)
 *   kv_commit_should_stage  the TTU/TTR commitment rule of Section 3.2 (host);
 *                         kv_decide_claims / kv_build_jobs_routed apply it to a
 *                         batch and route each claim; kv_ttr_* estimate TTR
 *   kv_stage_in / kv_retrieve_pipelined  lower tier -> HBM staging, and the
 *                         retrieve gated on those copies (stage-ready)
 *   kv_sim_run            claim/commitment controller in a discrete-event
 *                         simulation (Sections 3.1-3.3)
 *   kv_validate_jobs(_device)  race check of a job batch (duplicate
 *                         destinations, out-of-range ids), on host copies or
 *                         on the device
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Pointers named d_* are device-accessible (HBM, or mapped pinned host
 *    memory for the staging buffer); h_* are host memory.  The caller owns
 *    every buffer.  No call on the hot path allocates device or pinned host
 *    memory (kv_index_create allocates the index's device table and pinned
 *    snapshots, kv_pipeline_create its events; host-side calls use ordinary
 *    heap temporaries) or keeps a pointer after it returns.
 *  - GPU calls enqueue work on `stream` (a hipStream_t; NULL = the default
 *    stream) and return without synchronising.  Device faults surface at the
 *    caller's next synchronisation.
 *  - Return value: KV_OK (0) or a negative kv_status.  Argument errors are
 *    detected before anything is enqueued; KV_EHIP reports a failed launch.
 *  - Calls are reentrant; a kv_index must not be mutated concurrently.
 */
#ifndef TEMPOKV_H
#define TEMPOKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KV_HASH_BLOCK_TOKENS 16   /* tokens per hash block */
#define KV_MAX_LAYERS 128         /* layers one layout may name */

typedef enum kv_status {
    KV_OK = 0,
    KV_EINVAL = -1,  /* null pointer, negative count, inconsistent shape or offsets */
    KV_EALIGN = -2,  /* pointer or stride not 16-byte aligned */
    KV_ERANGE = -3,  /* slot, request, chunk or block id out of range (kv_validate_jobs) */
    KV_ENOSPC = -4,  /* no free staging slot for a miss, or the index is full */
    KV_EHIP = -5,    /* a HIP runtime call or kernel launch failed */
    KV_EDUP = -6,    /* two jobs of one batch write the same block (scatter) or slot (gather) */
    KV_ELIMIT = -7   /* request larger than a fixed capacity (kv_index_insert_static) */
} kv_status;

/* Shapes and strides of the two KV layouts.
 *   Staging slot s (one LMCache chunk of C tokens, Section 5 "Workload": only
 *   complete 256-token chunks are retained) is [L][2][C][H][D] elements of
 *   elem_bytes each, row-major, slot_bytes = L*2*C*H*D*elem_bytes apart.
 *   Paged KV (vLLM): one device pointer per layer; the B-token block `blk` of
 *   plane kv (0 = K, 1 = V) of layer l starts at
 *       layer_ptrs[l] + kv*paged_kv_stride + blk*paged_block_stride
 *   and holds [B][H][D] contiguous elements.  Per-layer [2][NB][B][H][D] is
 *   kv_stride = NB*B*H*D*e, block_stride = B*H*D*e; [NB][2][B][H][D] is
 *   kv_stride = B*H*D*e, block_stride = 2*B*H*D*e.
 * Requirements: all counts > 0; num_layers <= KV_MAX_LAYERS; elem_bytes in
 * {1, 2, 4} (the data is copied as opaque bits); chunk_tokens % block_size
 * == 0; B*H*D*elem_bytes and both strides multiples of 16. */
typedef struct kv_layout {
    int32_t num_layers;        /* L */
    int32_t kv_heads;          /* H */
    int32_t head_dim;          /* D */
    int32_t elem_bytes;        /* e */
    int32_t block_size;        /* B, tokens per paged block */
    int32_t chunk_tokens;      /* C, tokens per staged chunk */
    int64_t num_blocks;        /* NB, paged blocks per layer */
    int64_t num_slots;         /* S, staging slots */
    int64_t paged_kv_stride;   /* bytes from the K plane to the V plane of a layer */
    int64_t paged_block_stride;/* bytes between consecutive blocks of one plane */
} kv_layout;

/* One chunk transfer: staging slot <-> chunk `chunk` of request `req`, whose
 * C/B paged blocks are block_tables[req*bt_stride + chunk*C/B + i]. 16 bytes;
 * `reserved` must be 0. */
typedef struct kv_job {
    int32_t slot, req, chunk, reserved;
} kv_job;

/* ----------------------------------------------------------------------- */
/* Prefix hash                                                              */
/* ----------------------------------------------------------------------- */

/* Chained block hashes of a ragged batch of token sequences.  The paper
 * identifies reusable KV through LMCache's prefix lookup without defining it
 * (Section 4); this library fixes the hash, over complete 16-token blocks
 * (a trailing partial block has no hash, as the final incomplete chunk stays
 * uncached, Section 5 "Workload").  With M the SplitMix64 finalizer and
 * G = 0x9E3779B97F4A7C15, for request r and block b:
 *     d_b = sum_{j<16} M(uint32(tok[16b+j]) + ((j+1) << 32))   (mod 2^64)
 *     h_{-1} = seed,   h_b = M(h_{b-1} ^ d_b ^ G)
 * d_tokens    int32 [d_tok_off[num_reqs]]  token ids, requests back to back
 * d_tok_off   int64 [num_reqs+1]           token offsets (non-decreasing)
 * d_blk_off   int64 [num_reqs+1]           output offsets; d_blk_off[r+1] -
 *             d_blk_off[r] must equal floor(n_r/16) (not checked on device:
 *             a request whose span differs writes min of the two counts)
 * d_block_hash uint64 [d_blk_off[num_reqs]] output
 * num_reqs == 0 enqueues nothing.  Errors: KV_EINVAL (null pointer, num_reqs
 * < 0), KV_EHIP. */
int kv_hash_prefix(const int32_t *d_tokens, const int64_t *d_tok_off, int32_t num_reqs,
                   uint64_t seed, const int64_t *d_blk_off, uint64_t *d_block_hash, void *stream);

/* ----------------------------------------------------------------------- */
/* Staged-chunk index and lookup                                            */
/* ----------------------------------------------------------------------- */

/* Key -> staging slot map.  A KV object (Section 2.1) is one staged chunk,
 * identified by its chunk key: the block hash at the chunk's last block, so a
 * key names the whole token prefix that ends with that chunk.  The index is
 * kept on the host (it is mutated by host policy) and mirrored to a device
 * open-addressing table that kv_lookup probes.  Owns its host and device
 * memory. */
typedef struct kv_index kv_index;

/* Create an index for up to max_entries live keys on the current device.
 * Errors: KV_EINVAL (max_entries <= 0 or > 2^28, null out), KV_EHIP. */
int kv_index_create(int64_t max_entries, kv_index **out);
int kv_index_destroy(kv_index *idx);

/* Insert or update n (key, slot) pairs given in host memory (slot >= 0), then
 * enqueue the device-table update on `stream`; later work on that stream sees
 * it.  A key already present takes the new slot.  Errors: KV_EINVAL,
 * KV_ENOSPC (more than max_entries live keys; the pairs before the failing
 * one stay inserted), KV_EHIP. */
int kv_index_insert(kv_index *idx, const uint64_t *h_keys, const int32_t *h_slots, int32_t n,
                    void *stream);

/* Allocation-free kv_index_insert, for callers that cannot allocate memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, host-table result and stream ordering as
 * kv_index_insert, and it makes no hipMalloc, hipFree or other allocating
 * call (its host-side change list and a rebuild of the host table use memory
 * that kv_index_create reserved).  The (position, entry) pairs of an
 * incremental device-table update are staged in a fixed device array of
 * KV_INDEX_STATIC_MAX_PAIRS pairs (32 bytes each, 2 MiB) that the library
 * holds on each GPU it runs on until the process ends, instead of in the
 * index's own device lists; an update that changes more entries than the
 * index's incremental limit sends the whole table image, which needs no
 * staging.  Every call on one GPU shares that array and leaves the last
 * call's pairs in it, so calls on one GPU must be ordered on one stream (or
 * separated by a synchronisation): calls that overlap on one GPU race.
 * Errors: those of kv_index_insert, and KV_ELIMIT (nothing inserted) when
 * n > KV_INDEX_STATIC_MAX_PAIRS. */
#define KV_INDEX_STATIC_MAX_PAIRS 65536
int kv_index_insert_static(kv_index *idx, const uint64_t *h_keys, const int32_t *h_slots, int32_t n,
                           void *stream);

/* Remove n keys (absent keys are ignored), then enqueue the device-table
 * update on `stream`. Errors: KV_EINVAL, KV_EHIP. */
int kv_index_erase(kv_index *idx, const uint64_t *h_keys, int32_t n, void *stream);

/* Number of live keys (host view). */
int kv_index_size(const kv_index *idx, int64_t *out);

/* Slot of one key on the host view, or -1.  For tests and host policy. */
int kv_index_find(const kv_index *idx, uint64_t key, int32_t *slot_out);

/* Prefix match (Section 2.1: matching a request's prefix already tells
 * which objects it will read, and in what order).  For request r with nb_r block hashes
 * and bpc = blocks_per_chunk, chunk j < floor(nb_r/bpc) has key
 * K[r][j] = d_block_hash[d_blk_off[r] + (j+1)*bpc - 1];
 *   d_chunk_slot[d_chunk_off[r] + j] = slot of K[r][j], or -1 if absent
 *   d_hit_chunks[r] = largest k such that every chunk j < k is present
 * d_chunk_off int64 [num_reqs+1] must hold the prefix sums of
 * floor(nb_r/bpc).  Errors: KV_EINVAL, KV_EHIP. */
int kv_lookup(const kv_index *idx, const uint64_t *d_block_hash, const int64_t *d_blk_off,
              int32_t num_reqs, int32_t blocks_per_chunk, const int64_t *d_chunk_off,
              int32_t *d_chunk_slot, int32_t *d_hit_chunks, void *stream);

/* ----------------------------------------------------------------------- */
/* Host job build                                                           */
/* ----------------------------------------------------------------------- */

/* Chunk keys of a batch from its block hashes (host arrays): for request r
 * and chunk j < floor(nb_r / blocks_per_chunk),
 *     h_keys[h_chunk_off[r] + j] = h_block_hash[h_blk_off[r] + (j+1)*blocks_per_chunk - 1],
 * the key kv_lookup probes (the hash at the chunk's last block).  Errors:
 * KV_EINVAL (null pointer, offsets inconsistent with blocks_per_chunk). */
int kv_chunk_keys(const uint64_t *h_block_hash, const int64_t *h_blk_off, int32_t num_reqs,
                  int32_t blocks_per_chunk, const int64_t *h_chunk_off, uint64_t *h_keys);

/* Turn a lookup result (copied to the host) into transfer jobs.
 *   retrieve jobs: {chunk_slot, r, j} for every j < h_hit_chunks[r], in (r, j)
 *     order -- the matched KV that retrieval moves to the GPU (Section 3.1);
 *   store jobs: for chunks j >= h_hit_chunks[r] with chunk_slot == -1, in
 *     (r, j) order, one job per distinct key (the first occurrence wins:
 *     staging of one KV object is coalesced, Section 3.2 "Shared staging and
 *     resource lifecycle"), with slots taken from h_free_slots in order.
 *     h_store_keys[i] receives the key of store job i.
 * h_retrieve and h_store must each hold h_chunk_off[num_reqs] jobs.
 * Distinct missing keys beyond num_free get no job; *dropped counts them and
 * the call returns KV_ENOSPC with the emitted jobs valid.  Errors: KV_EINVAL. */
int kv_build_jobs(const int32_t *h_hit_chunks, const int32_t *h_chunk_slot,
                  const uint64_t *h_block_hash, const int64_t *h_blk_off, const int64_t *h_chunk_off,
                  int32_t num_reqs, int32_t blocks_per_chunk, const int32_t *h_free_slots,
                  int32_t num_free, kv_job *h_retrieve, int32_t *num_retrieve, kv_job *h_store,
                  uint64_t *h_store_keys, int32_t *num_store, int32_t *dropped);

/* ----------------------------------------------------------------------- */
/* Retrieve scatter and store gather                                        */
/* ----------------------------------------------------------------------- */

/* Retrieve (fast tier -> GPU, the transfer TTU counts down to, Section 3.1):
 * for every job, layer l, plane kv and block i < C/B, copy the B-token
 * segment at staging byte
 *     slot*slot_bytes + ((l*2 + kv)*C + i*B)*H*D*e
 * to paged block block_tables[req*bt_stride + chunk*C/B + i] of (l, kv).
 * d_staging      device-accessible staging buffer [num_slots * slot_bytes]
 * h_layer_ptrs   HOST array of num_layers device pointers (paged tensors)
 * d_block_tables int32 [num_reqs][bt_stride] block ids
 * d_jobs         kv_job [num_jobs] (device)
 * Jobs whose slot, req or chunk is out of range, and segments whose block id
 * is outside [0, num_blocks), are skipped: the kernel reads and writes only
 * inside the described buffers.  Destinations must be disjoint within one
 * call (kv_validate_jobs checks it); many jobs may read one slot.  One kernel
 * launch per call; num_jobs == 0 enqueues nothing.
 * Errors: KV_EINVAL, KV_EALIGN, KV_EHIP. */
int kv_retrieve_scatter(const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                        const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs,
                        const kv_job *d_jobs, int32_t num_jobs, void *stream);

/* Variants of the retrieve.  All give the bytes of kv_retrieve_scatter for
 * any job list; they differ in speed by the way jobs share staged chunks. */
typedef enum kv_retrieve_kind {
    KV_RETRIEVE_UNIT = 0,   /* one workgroup per (job, layer, plane) unit; jobs that share a chunk read it
                               through the L2 (kv_retrieve_scatter) */
    KV_RETRIEVE_PAIR = 1,   /* one workgroup per pair of consecutive jobs: a pair naming one chunk reads each
                               stage once and writes it twice (32 KiB segments; other sizes use UNIT) */
    KV_RETRIEVE_STREAM = 2, /* 1024-lane workgroups, non-temporal loads of the staged chunks: for lists that
                               read each chunk once */
    KV_RETRIEVE_QUAD = 3    /* one 1024-lane workgroup per (layer, plane, 4 consecutive jobs, segment): jobs of
                               the window that share a chunk load it together, one read from memory and the
                               rest from L2.  Segments of 4, 8, 16, 32 or 64 KiB (other sizes use the generic
                               copy).  Never returned by kv_retrieve_plan: whether it beats PAIR/UNIT depends on
                               where the paged pool lies in physical memory (it does on most placements
                               measured, by about 6 %, and loses where scattered writes run fast), so a caller
                               picks it by timing both on its own pool. */
} kv_retrieve_kind;

/* Pick the variant for a job list from its host copy (grouped by slot, as
 * kv_group_jobs_by_slot leaves it): STREAM when every slot appears once; PAIR
 * when the segments are 32 KiB, at least 90 % of the job pairs (0,1), (2,3),
 * ... name one slot and the groups of equal slots average at most 16 jobs;
 * UNIT otherwise.  The thresholds are measured (lists with groups of 8, as in
 * a batch whose requests share a handful of prefixes, gain 3-13 % from PAIR;
 * irregular or very large groups lose 1-3 %).  Returns a kv_retrieve_kind, or
 * KV_EINVAL / a layout error. */
int kv_retrieve_plan(const kv_layout *layout, const kv_job *h_jobs, int32_t num_jobs);

/* kv_retrieve_scatter with an explicit variant (a kv_retrieve_kind).  Same
 * arguments, checks and errors, plus KV_EINVAL for an unknown kind. */
int kv_retrieve_scatter_as(int32_t kind, const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                           const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs,
                           const kv_job *d_jobs, int32_t num_jobs, void *stream);

/* Store (retaining the KV of complete chunks, Section 5 "Workload"): the
 * inverse walk, paged blocks of (req, chunk) -> staging slot.  Slots must be
 * disjoint within one call.  Same arguments, checks and errors. */
int kv_store_gather(const kv_layout *layout, void *d_staging, const void *const *h_layer_ptrs,
                    const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs,
                    const kv_job *d_jobs, int32_t num_jobs, void *stream);

/* Reorder a job list in host memory so that jobs naming the same staging
 * slot are adjacent (stable: by slot, then original order).  The copies'
 * results do not depend on job order (destinations are disjoint within a
 * call); the retrieve kernel reads a staged chunk once per unit when the
 * jobs sharing it run back to back.  Errors: KV_EINVAL. */
int kv_group_jobs_by_slot(kv_job *h_jobs, int32_t num_jobs);

/* ----------------------------------------------------------------------- */
/* Staging into HBM and the stage-ready-gated retrieve                      */
/* ----------------------------------------------------------------------- */

/* The paper separates staging (SSD -> fast tier) from retrieval (fast tier ->
 * GPU), and calls the matched KV stage-ready once every object it needs
 * sits in the fast tier under protection (Section 2.2).  Here pinned host
 * memory stands in for the lower tier and the HBM staging buffer is the fast
 * tier: h_lower_tier holds slots in the same [S][L][2][C][H][D] layout, slot
 * s at byte s*slot_bytes of both buffers.  h_lower_tier should come from
 * hipHostMalloc (pageable memory also works, but its copies do not overlap). */

/* Stage slots h_slots[0..n) of the lower tier into the same slots of
 * d_staging: DMA copies (hipMemcpyAsync) on `stream`, one per run of
 * consecutive slot ids.  Every slot is checked before anything is enqueued.
 * Errors: KV_EINVAL, KV_ERANGE (slot outside [0, num_slots)), KV_EHIP. */
int kv_stage_in(const kv_layout *layout, const void *h_lower_tier, void *d_staging, const int32_t *h_slots,
                int32_t n, void *stream);

/* The reverse copy, fast tier -> lower tier, for the same slots (retaining
 * stored chunks below the fast tier).  Same checks and errors. */
int kv_stage_out(const kv_layout *layout, const void *d_staging, void *h_lower_tier, const int32_t *h_slots,
                 int32_t n, void *stream);

/* Events for kv_retrieve_pipelined (one per batch, up to max_batches batches
 * per call), created on the current device; the caller owns the object and
 * frees it with kv_pipeline_destroy, which first waits for its events.  One
 * object serves one call at a time; calls that overlap on two host threads
 * race.  Errors: KV_EINVAL, KV_EHIP. */
typedef struct kv_pipeline kv_pipeline;
int kv_pipeline_create(int32_t max_batches, kv_pipeline **out);
int kv_pipeline_destroy(kv_pipeline *pl);

/* Retrieve whose staged chunks start in the lower tier.  The jobs should be
 * grouped by slot (kv_group_jobs_by_slot); h_jobs is their host copy, d_jobs
 * the same array on the device.  They are cut into batches of
 * `slots_per_batch` distinct slots (raised if needed so that at most the
 * pipeline's max_batches batches are formed).  For each batch its slots are
 * staged on copy_stream, an event recorded after those copies marks them
 * stage-ready, and `stream` waits for that event before the retrieve scatter
 * of the batch's jobs: retrieval of a chunk begins only once it is
 * stage-ready (Sections 2.2 and 3.2), and the copy of the next batch overlaps
 * the scatter of this one.  Afterwards the staged slots are also resident in
 * d_staging.  Passing one stream as both copy_stream and stream serialises
 * every copy with its scatter.  Ungrouped jobs give the same result, but a
 * slot is then staged once per batch that names it.  The copies are not
 * ordered after earlier work on `stream`: the caller makes copy_stream wait
 * for any such work that still reads or writes the staged slots.  Every
 * argument and job slot is checked before anything is enqueued; a KV_EHIP
 * part-way leaves the batches before it enqueued.  Errors: those of
 * kv_retrieve_scatter and kv_stage_in, and KV_EINVAL when the current device
 * is not the pipeline's. */
int kv_retrieve_pipelined(kv_pipeline *pl, const kv_layout *layout, const void *h_lower_tier, void *d_staging,
                          void *const *h_layer_ptrs, const int32_t *d_block_tables, int32_t bt_stride,
                          int32_t num_reqs, const kv_job *h_jobs, const kv_job *d_jobs, int32_t num_jobs,
                          int32_t slots_per_batch, void *copy_stream, void *stream);

/* Host check of a job batch against copies of its tables: KV_ERANGE if any
 * slot, request, chunk or (valid-job) block id is out of range or any
 * reserved field is non-zero, KV_EDUP if two jobs write the same destination
 * (scatter: paged block of a plane; gather, is_store != 0: staging slot),
 * else KV_OK. */
int kv_validate_jobs(const kv_layout *layout, const int32_t *h_block_tables, int32_t bt_stride,
                     int32_t num_reqs, const kv_job *h_jobs, int32_t num_jobs, int is_store);

/* The same check on the device, for a batch whose jobs and block tables are
 * already in device memory (race detection before a scatter or gather: two
 * jobs of one launch writing the same paged block or staging slot are the
 * only writes that can race; many jobs may read one slot).  d_marks is
 * caller-owned device scratch of 2 + (is_store ? num_slots : num_blocks)
 * int32, overwritten; d_status (one int32 in device memory) receives
 * KV_ERANGE, KV_EDUP or KV_OK, with the meaning and precedence of
 * kv_validate_jobs, once the enqueued work completes: read it after `stream`
 * synchronizes.  Three launches on `stream` (clear, mark, status), no
 * allocation, no memset, no host synchronization.  Returns KV_OK once
 * enqueued; KV_EINVAL (bad layout, negative count, null pointer) or KV_EALIGN
 * (d_jobs not 16-byte aligned, an int32 pointer not 4-byte aligned) with
 * nothing enqueued; KV_EHIP if a launch fails. */
int kv_validate_jobs_device(const kv_layout *layout, const int32_t *d_block_tables, int32_t bt_stride,
                            int32_t num_reqs, const kv_job *d_jobs, int32_t num_jobs, int is_store,
                            int32_t *d_marks, int32_t *d_status, void *stream);

/* ----------------------------------------------------------------------- */
/* Commitment rule (host)                                                   */
/* ----------------------------------------------------------------------- */

typedef enum kv_commit_decision {
    KV_DEFER = 0,    /* not eligible yet: laxity positive and no retrieval request */
    KV_COMMIT = 1,   /* eligible and the footprint fits: request the commitment */
    KV_BLOCKED = 2,  /* eligible, does not fit, no retrieval request: stays PLANNED */
    KV_ORDINARY = 3  /* retrieval requested and protection unavailable: ordinary path */
} kv_commit_decision;

/* Section 3.2: laxity L = TTU - TTR; eligible iff L <= 0 (evaluated as
 * ttu_s <= ttr_s, so infinite estimates behave) or retrieval_requested.  A
 * commitment needs the claim's full footprint within the protected budget
 * (claim_total_bytes <= budget_bytes) and its newly reserved bytes -- those
 * that no earlier commitment protects yet -- within the free protected
 * capacity (claim_new_bytes <= free_protected_bytes).  Returns a
 * kv_commit_decision, or KV_EINVAL for a NaN estimate or claim_new_bytes >
 * claim_total_bytes.  Aging TTU by elapsed time is the caller's job. */
int kv_commit_should_stage(double ttu_s, double ttr_s, uint64_t free_protected_bytes,
                           uint64_t claim_new_bytes, uint64_t claim_total_bytes,
                           uint64_t budget_bytes, int retrieval_requested);

/* The same rule for the n claims of one batch, each decided on its own
 * against the same free protected capacity and budget:
 *   h_out[i] = kv_commit_should_stage(h_ttu[i], h_ttr[i], free_protected_bytes,
 *                                     h_claim_new[i], h_claim_total[i],
 *                                     budget_bytes, h_requested[i])
 * (h_requested: one byte per claim, nonzero = retrieval requested).  An
 * element with invalid inputs gets KV_EINVAL in h_out; the others are still
 * decided.  Host arrays only; nothing is kept.  Returns KV_OK, or KV_EINVAL
 * for n < 0 or a null array with n > 0. */
int kv_commit_should_stage_n(int32_t n, const double *h_ttu, const double *h_ttr, uint64_t free_protected_bytes,
                             const uint64_t *h_claim_new, const uint64_t *h_claim_total, uint64_t budget_bytes,
                             const uint8_t *h_requested, int32_t *h_out);

/* Commitment decisions for the claims of one batch (Section 3.2).  Claim r
 * is the matched prefix of request r: its KV objects are the distinct staging
 * slots h_chunk_slot[h_chunk_off[r] + j], j < h_hit_chunks[r] (as a lookup
 * leaves them), slot_bytes bytes each.  Claims are evaluated in the order of
 * "Commitment and replanning": those with a pending retrieval request
 * (h_requested[r] != 0) first, then the others, each group in request order;
 * a claim that cannot commit does not block the ones after it.  For each claim
 *   total = its objects x slot_bytes,  new = bytes of its objects not yet
 *   protected (h_protected[slot] == 0),  free = budget_bytes - *reserved_bytes
 *   (0 when the reservations exceed the budget),
 *   h_decision[r] = kv_commit_should_stage(h_ttu[r], h_ttr[r], free, new,
 *                                          total, budget_bytes, h_requested[r]).
 * A KV_COMMIT protects the claim's objects and adds `new` to *reserved_bytes:
 * objects shared by claims are reserved once ("Shared staging and resource
 * lifecycle").  h_protected (uint8 [num_slots]) and *reserved_bytes are the
 * protected-capacity ledger, read and updated in place; start them at zero
 * when no earlier commitment is still in force.  Host arrays only.  Errors:
 * KV_EINVAL (null pointer, inconsistent offsets or hit counts), KV_ERANGE (a
 * matched slot outside [0, num_slots)); a claim with a NaN estimate gets
 * KV_EINVAL as its decision. */
int kv_decide_claims(int32_t num_reqs, const int32_t *h_hit_chunks, const int32_t *h_chunk_slot,
                     const int64_t *h_chunk_off, const double *h_ttu, const double *h_ttr,
                     const uint8_t *h_requested, uint64_t slot_bytes, uint64_t budget_bytes, int64_t num_slots,
                     uint8_t *h_protected, uint64_t *reserved_bytes, int32_t *h_decision);

/* kv_build_jobs for a batch whose claims were decided (kv_decide_claims).
 * Only requests whose retrieval is requested (h_requested[r] != 0) run in
 * this batch and get jobs; the others have none yet.  A running request's
 * matched chunks become retrieve jobs in h_retrieve when its decision is
 * KV_COMMIT (the protected, staged route) and in h_ordinary when it is
 * KV_ORDINARY (the ordinary retrieval path, "Protected capacity and on-demand
 * retrieval"); its store jobs follow the rule of kv_build_jobs over the
 * running requests only.  h_ordinary must hold h_chunk_off[num_reqs] jobs
 * like the other two lists.  Errors: those of kv_build_jobs, and KV_EINVAL
 * for a running request whose decision is neither KV_COMMIT nor KV_ORDINARY. */
int kv_build_jobs_routed(const int32_t *h_hit_chunks, const int32_t *h_chunk_slot,
                         const uint64_t *h_block_hash, const int64_t *h_blk_off, const int64_t *h_chunk_off,
                         int32_t num_reqs, int32_t blocks_per_chunk, const int32_t *h_free_slots,
                         int32_t num_free, const uint8_t *h_requested, const int32_t *h_decision,
                         kv_job *h_retrieve, int32_t *num_retrieve, kv_job *h_ordinary, int32_t *num_ordinary,
                         kv_job *h_store, uint64_t *h_store_keys, int32_t *num_store, int32_t *dropped);

/* ----------------------------------------------------------------------- */
/* Time-to-ready estimates (host)                                           */
/* ----------------------------------------------------------------------- */

/* The two TTR estimators of Section 3.1 ("Storage-estimated time-to-ready")
 * and Section 5 ("Policies"), over the distinct KV objects h_objs[0..n) of one
 * claim (ids below num_objects; per-object arrays are indexed by id).  They
 * feed kv_commit_should_stage, and the simulator (kv_sim_run) uses the same
 * code.
 * Static (TempoKV-Static): the claim's non-resident bytes over a fixed rate,
 * as if the claim were staged in isolation:
 *     *ttr_s = sum over non-resident o of h_obj_bytes[o] / static_rate. */
int kv_ttr_static(int32_t n, const int32_t *h_objs, int32_t num_objects, const double *h_obj_bytes,
                  const uint8_t *h_resident, double static_rate, double *ttr_s);

/* State-aware: the staging device's queue projected from now_s.  An object
 * already queued (h_queued[o] != 0) becomes resident at h_ready_at[o]; each
 * non-resident object not yet queued is appended, in claim order, behind the
 * queue's tail max(busy_until_s, now_s) at stage_rate bytes/s; the claim is
 * ready when its last object is: *ttr_s = (latest such time, at least now_s)
 * - now_s.  Errors (both): KV_EINVAL for a null pointer, an object id out of
 * range, a rate <= 0 or a NaN time. */
int kv_ttr_state_aware(int32_t n, const int32_t *h_objs, int32_t num_objects, const double *h_obj_bytes,
                       const uint8_t *h_resident, const uint8_t *h_queued, const double *h_ready_at,
                       double now_s, double busy_until_s, double stage_rate, double *ttr_s);

/* ----------------------------------------------------------------------- */
/* Claim controller and staging simulator (host)                            */
/* ----------------------------------------------------------------------- */

/* Commitment policies (Section 5, "Policies"): when a PLANNED claim becomes
 * eligible for a commitment attempt.  Retrieval requested by the runtime makes
 * any claim eligible. */
typedef enum kv_policy {
    KV_POLICY_DEMAND = 0,        /* only when retrieval is requested */
    KV_POLICY_IMMEDIATE = 1,     /* as soon as the claim is reported */
    KV_POLICY_QUEUE_K = 2,       /* when at most K-1 waiting requests are ahead of it */
    KV_POLICY_TEMPO_STATIC = 3,  /* TTU <= TTR, TTR = non-resident bytes / static rate, in isolation */
    KV_POLICY_TEMPO = 4          /* TTU <= TTR, TTR from a projection of the staging queue */
} kv_policy;

/* Simulation of the controller (Section 3) with a runtime and staging-device
 * model.  Fast tier of capacity_bytes with a protected budget; one FIFO
 * staging server at stage_rate bytes/s; FCFS runtime with max_active slots;
 * retrieval at gpu_rate bytes/s, then prefill_s per uncached token and
 * decode_s per output token; control points after every event and every
 * tick_s seconds.  Byte counts must be integers below 2^53. */
typedef struct kv_sim_config {
    double budget_bytes, capacity_bytes, stage_rate, static_rate, gpu_rate, prefill_s, decode_s, tick_s;
    int32_t max_active, policy, queue_k, reserved;   /* reserved must be 0 */
} kv_sim_config;

typedef struct kv_sim_result {
    double area_byte_s;            /* integral of reserved protected bytes P(t) over time */
    double cost_gib_s_per_request; /* C = area / 2^30 / N (Section 5, "Metrics") */
    double end_s;                  /* time the last request ended */
    double p_max_bytes;            /* largest P(t) */
    int32_t committed;             /* claims committed */
    int32_t blocked;               /* requests whose claim was blocked by capacity at least once */
    int32_t ordinary;              /* requests that took the ordinary (demand) path */
    int32_t reserved;
    int64_t events;                /* events processed */
} kv_sim_result;

typedef enum kv_sim_trace_kind {
    KV_TR_ARRIVE = 0, KV_TR_ADMIT, KV_TR_COMMIT, KV_TR_ORDINARY, KV_TR_READY, KV_TR_STAGEREADY,
    KV_TR_TRANSFER, KV_TR_FETCH, KV_TR_RELEASE, KV_TR_DONE, KV_TR_EVICT
} kv_sim_trace_kind;

typedef struct kv_sim_event {
    double t;
    int32_t kind;   /* kv_sim_trace_kind */
    int32_t id;     /* request id, or object id for READY / EVICT */
} kv_sim_event;

/* Run one simulation.  Objects 0..num_objects-1 have h_obj_bytes[o] bytes;
 * request i arrives at h_arrival[i] (non-decreasing not required), needs the
 * objects h_manifest_objs[h_manifest_off[i] .. h_manifest_off[i+1]) in that
 * order, and has h_uncached[i] uncached and h_out_tokens[i] output tokens.
 * Outputs: first-token and end times per request, the result summary, and
 * (optional, h_trace may be NULL) the event trace, truncated to trace_cap
 * entries with *trace_len the full length.  Errors: KV_EINVAL. */
int kv_sim_run(const kv_sim_config *cfg, const double *h_obj_bytes, int32_t num_objects,
               const double *h_arrival, const int64_t *h_manifest_off, const int32_t *h_manifest_objs,
               const int32_t *h_uncached, const int32_t *h_out_tokens, int32_t num_requests,
               double *h_first_token, double *h_done, kv_sim_result *result, kv_sim_event *h_trace,
               int64_t trace_cap, int64_t *trace_len);

/* ----------------------------------------------------------------------- */
/* Measurement reference (not part of the path)                             */
/* ----------------------------------------------------------------------- */

/* For callers that time the retrieve against what its bytes cost on their
 * own pool: moves kv_retrieve_scatter's algorithmic bytes with no dependence
 * between them, in one launch.  Every segment of the num_read_slots slots in
 * d_slots (int32, device) is read once, and every destination segment of the
 * jobs (the blocks kv_retrieve_scatter would write) is written with the
 * 32-bit word `fill` repeated; the reads are spread evenly among the writes
 * in dispatch order, and no written byte depends on a read.  It OVERWRITES
 * those destination blocks (re-run the retrieve to restore them) and touches
 * nothing else; jobs, slots and block ids out of range are skipped as in the
 * copies.  Same layout and pointer arguments as kv_retrieve_scatter; one
 * launch per call.  Errors: KV_EINVAL (also when the jobs' and slots'
 * segments number 2^31 or more), KV_EALIGN, KV_EHIP. */
int kv_probe_mixed_traffic(const kv_layout *layout, const void *d_staging, void *const *h_layer_ptrs,
                           const int32_t *d_block_tables, int32_t bt_stride, int32_t num_reqs,
                           const kv_job *d_jobs, int32_t num_jobs, const int32_t *d_slots,
                           int32_t num_read_slots, uint32_t fill, void *stream);

/* ----------------------------------------------------------------------- */
/* Misc                                                                     */
/* ----------------------------------------------------------------------- */

/* Static description of a status code. */
const char *kv_strerror(int status);

/* Device address of mapped pinned host memory (hipHostMalloc'd), for staging
 * buffers read zero-copy from host memory.  Errors: KV_EINVAL, KV_EHIP. */
int kv_host_device_pointer(const void *h_ptr, void **d_ptr_out);

/* Library version, e.g. "tempokv 0.1.0 gfx950". */
const char *kv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TEMPOKV_H */

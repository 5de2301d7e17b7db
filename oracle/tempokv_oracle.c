/*
 * tempokv_oracle.c -- plain, slow, single-threaded CPU oracle for the TempoKV
 * staging hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline use it.  It shares no header, helper or constant table with the HIP
 * library: every definition below is written out again from the method text.
 *
 * What the paper fixes and what it leaves open
 * --------------------------------------------
 * TempoKV (Section 4, "Runtime and controller integration") takes the prefix
 * matching and the fast-tier-to-GPU copy from LMCache as they are and does
 * not describe them.
 * The data-parallel path computed here is therefore defined as follows; each
 * function names the passage it follows and the reading taken where the
 * paper is silent.
 *
 *   - Reusable prefix KV is handled as separately named objects that are
 *     only read while reused, and matching a request's prefix already tells
 *     which objects it needs and in what order (Section 2.1).  Here one object is one
 *     LMCache chunk of C tokens; only complete chunks are retained and the
 *     final incomplete chunk stays uncached (Section 5, "Workload").
 *   - Objects are identified by a chained 64-bit hash over 16-token blocks
 *     (definition below); the chunk key is the chained hash at the chunk's
 *     last block, so a key identifies the whole token prefix up to it.
 *   - Lookup is a prefix match: the hits of a request are its longest run of
 *     indexed chunks starting at chunk 0.
 *   - Retrieval copies a staged chunk [L][2][C][H][D] into paged blocks named
 *     by the request's block table (the fast-tier-to-GPU retrieval that TTU
 *     counts down to, Section 3.1); the store direction is its inverse.
 *   - The commitment rule follows Section 3.2: eligible iff laxity
 *     TTU - TTR <= 0 or retrieval was requested; a commitment needs the full
 *     footprint to fit the protected budget; otherwise the claim stays
 *     PLANNED, or takes the ordinary path when retrieval was requested.
 *
 * Element loops throughout, no memcpy, no blocking or reordering: each output
 * element is produced by the index arithmetic written in the comments.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>

/* ------------------------------------------------------------------------- */
/* Chained prefix hash                                                        */
/* ------------------------------------------------------------------------- */

/* M(z): the SplitMix64 output finalizer (Steele, Lea & Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014, in the variant
 * used by Java's SplittableRandom and by Vigna's public-domain splitmix64.c:
 * xor-shift 30, multiply, xor-shift 27, multiply, xor-shift 31).  It is a
 * bijection on 64-bit words.  All arithmetic is modulo 2^64. */
uint64_t or_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* The golden-ratio increment of SplitMix64 (same source). */
#define OR_GAMMA 0x9E3779B97F4A7C15ull
#define OR_HASH_BLOCK 16

/* One SplitMix64 draw: state += gamma, return M(state).  Used only by the
 * tests to check M against the generator's published output sequence. */
uint64_t or_splitmix64_next(uint64_t *state)
{
    *state += OR_GAMMA;
    return or_mix64(*state);
}

/* Digest of one 16-token block: d = sum over j of M(tok_j + ((j+1) << 32)),
 * with tok_j taken as an unsigned 32-bit word.  The position j is folded into
 * the high half, so the word of (j, tok) is distinct for every pair. */
uint64_t or_block_digest(const int32_t *tok16)
{
    uint64_t d = 0;
    for (int j = 0; j < OR_HASH_BLOCK; j++) {
        uint64_t word = (uint64_t)(uint32_t)tok16[j] + ((uint64_t)(j + 1) << 32);
        d += or_mix64(word);
    }
    return d;
}

/* Chained block hashes of every request (the chain is sequential across
 * blocks: h_{-1} = seed, h_b = M(h_{b-1} xor d_b xor gamma)).  A trailing
 * partial block produces no hash.
 *   tokens   : all requests' token ids back to back
 *   tok_off  : [num_reqs+1] token offsets
 *   blk_off  : [num_reqs+1] block-hash offsets; blk_off[r+1]-blk_off[r] must
 *              equal floor(n_r / 16)
 *   out      : [blk_off[num_reqs]] block hashes
 * Returns 0, or -1 if an offset array is inconsistent. */
int or_hash_prefix(const int32_t *tokens, const int64_t *tok_off, int32_t num_reqs,
                   uint64_t seed, const int64_t *blk_off, uint64_t *out)
{
    if (num_reqs < 0) return -1;
    for (int32_t r = 0; r < num_reqs; r++) {
        int64_t n = tok_off[r + 1] - tok_off[r];
        if (n < 0) return -1;
        int64_t nb = n / OR_HASH_BLOCK;
        if (blk_off[r + 1] - blk_off[r] != nb) return -1;
        uint64_t h = seed;
        for (int64_t b = 0; b < nb; b++) {
            uint64_t d = or_block_digest(tokens + tok_off[r] + b * OR_HASH_BLOCK);
            h = or_mix64(h ^ d ^ OR_GAMMA);
            out[blk_off[r] + b] = h;
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Lookup: prefix match against the staged-chunk index                        */
/* ------------------------------------------------------------------------- */

/* The index is given as its live (key, slot) pairs; keys are distinct.  A
 * linear scan finds a key's slot, or -1. */
static int32_t or_index_find(const uint64_t *keys, const int32_t *slots, int64_t n, uint64_t key)
{
    for (int64_t i = 0; i < n; i++)
        if (keys[i] == key) return slots[i];
    return -1;
}

/* For request r with nb_r block hashes, chunk j (j < floor(nb_r / bpc)) has
 * the key K[r][j] = h_{(j+1)*bpc - 1}, bpc = blocks per chunk = C / 16.
 *   chunk_slot[chunk_off[r] + j] = slot of K[r][j] in the index, or -1
 *   hit_chunks[r] = largest k with every chunk j < k present
 * Returns 0, or -1 on inconsistent offsets. */
int or_lookup(const uint64_t *idx_keys, const int32_t *idx_slots, int64_t idx_n,
              const uint64_t *block_hash, const int64_t *blk_off, int32_t num_reqs,
              int32_t blocks_per_chunk, const int64_t *chunk_off,
              int32_t *chunk_slot, int32_t *hit_chunks)
{
    if (blocks_per_chunk <= 0 || num_reqs < 0) return -1;
    for (int32_t r = 0; r < num_reqs; r++) {
        int64_t nb = blk_off[r + 1] - blk_off[r];
        int64_t nc = nb / blocks_per_chunk;
        if (chunk_off[r + 1] - chunk_off[r] != nc) return -1;
        int32_t hits = 0;
        int still_prefix = 1;
        for (int64_t j = 0; j < nc; j++) {
            uint64_t key = block_hash[blk_off[r] + (j + 1) * blocks_per_chunk - 1];
            int32_t s = or_index_find(idx_keys, idx_slots, idx_n, key);
            chunk_slot[chunk_off[r] + j] = s;
            if (s < 0) still_prefix = 0;
            if (still_prefix) hits++;
        }
        hit_chunks[r] = hits;
    }
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Host job build                                                             */
/* ------------------------------------------------------------------------- */

typedef struct { int32_t slot, req, chunk, reserved; } or_job;

/* From a lookup result, emit
 *   retrieve jobs {slot, r, j} for every j < hit_chunks[r], in (r, j) order;
 *   store jobs {slot, r, j} for every chunk j >= hit_chunks[r] whose key is not
 *     in the index, skipping a key already given a store job earlier in this
 *     batch (the first (r, j) in order wins: one staged copy per KV object,
 *     as staging of the same object is coalesced, Section 3.2 "Shared staging
 *     and resource lifecycle"); slots are taken from free_slots in the order
 *     given.
 * When the free slots run out, the remaining distinct missing keys get no
 * store job and *dropped counts them.  store_keys[i] is the key of store
 * job i.  Returns 0, or -1 if scratch memory cannot be had. */
int or_build_jobs(const int32_t *hit_chunks, const int32_t *chunk_slot, const uint64_t *block_hash,
                  const int64_t *blk_off, const int64_t *chunk_off, int32_t num_reqs,
                  int32_t blocks_per_chunk, const int32_t *free_slots, int32_t num_free,
                  or_job *retrieve, int32_t *num_retrieve,
                  or_job *store, uint64_t *store_keys, int32_t *num_store, int32_t *dropped)
{
    int32_t nr = 0, ns = 0, nd = 0;
    int64_t nmiss = 0;
    /* every distinct missing key met so far, stored or dropped */
    uint64_t *miss_keys = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)(chunk_off[num_reqs] + 1));
    if (!miss_keys) return -1;
    for (int32_t r = 0; r < num_reqs; r++) {
        int64_t nc = chunk_off[r + 1] - chunk_off[r];
        for (int64_t j = 0; j < nc; j++) {
            int32_t s = chunk_slot[chunk_off[r] + j];
            if (j < hit_chunks[r]) {
                retrieve[nr].slot = s;
                retrieve[nr].req = r;
                retrieve[nr].chunk = (int32_t)j;
                retrieve[nr].reserved = 0;
                nr++;
                continue;
            }
            if (s >= 0) continue;              /* indexed, but after the first miss */
            uint64_t key = block_hash[blk_off[r] + (j + 1) * blocks_per_chunk - 1];
            int seen = 0;
            for (int64_t q = 0; q < nmiss; q++)
                if (miss_keys[q] == key) { seen = 1; break; }
            if (seen) continue;
            miss_keys[nmiss++] = key;
            if (ns >= num_free) { nd++; continue; }
            store[ns].slot = free_slots[ns];
            store[ns].req = r;
            store[ns].chunk = (int32_t)j;
            store[ns].reserved = 0;
            store_keys[ns] = key;
            ns++;
        }
    }
    free(miss_keys);
    *num_retrieve = nr;
    *num_store = ns;
    *dropped = nd;
    return 0;
}

/* ------------------------------------------------------------------------- */
/* Retrieve scatter and store gather                                          */
/* ------------------------------------------------------------------------- */

/* Shape of the two layouts (all sizes in elements unless named *_bytes).
 *   staging slot s : [L][2][C][H][D] elements of e bytes, slot_bytes apart
 *   paged layer l  : base layers[l]; the B-token block `blk` of plane kv
 *                    (0 = K, 1 = V) starts at kv*kv_stride + blk*block_stride
 *                    bytes and holds [B][H][D] elements.                     */
typedef struct {
    int32_t L, H, D, e, B, C;
    int64_t num_blocks, num_slots, kv_stride, block_stride;
} or_layout;

static int or_job_ok(const or_layout *lo, const or_job *jb, int32_t num_reqs, int32_t bt_stride)
{
    int32_t nseg = lo->C / lo->B;
    if (jb->slot < 0 || jb->slot >= lo->num_slots) return 0;
    if (jb->req < 0 || jb->req >= num_reqs) return 0;
    if (jb->chunk < 0 || ((int64_t)jb->chunk + 1) * nseg > bt_stride) return 0;
    return 1;
}

/* Retrieve: for every job, layer l, plane kv, block i of the chunk, token t and
 * element x, byte c:
 *   blk = bt[req][chunk*C/B + i]
 *   paged[l] byte kv*kv_stride + blk*block_stride + (t*H*D + x)*e + c
 *     = staging byte slot*slot_bytes + (((l*2+kv)*C + i*B + t)*H*D + x)*e + c
 * A job with slot, req or chunk out of range, and a block id outside
 * [0, num_blocks), are skipped (no byte is read or written for them). */
void or_retrieve_scatter(const or_layout *lo, const uint8_t *staging, uint8_t *const *layers,
                         const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                         const or_job *jobs, int32_t num_jobs)
{
    int64_t HD = (int64_t)lo->H * lo->D;
    int64_t slot_bytes = (int64_t)lo->L * 2 * lo->C * HD * lo->e;
    int32_t nseg = lo->C / lo->B;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        for (int32_t l = 0; l < lo->L; l++)
            for (int32_t kv = 0; kv < 2; kv++)
                for (int32_t i = 0; i < nseg; i++) {
                    int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i];
                    if (blk < 0 || blk >= lo->num_blocks) continue;
                    for (int32_t t = 0; t < lo->B; t++)
                        for (int64_t x = 0; x < HD; x++)
                            for (int32_t c = 0; c < lo->e; c++) {
                                int64_t src = jb->slot * slot_bytes
                                    + ((((int64_t)l * 2 + kv) * lo->C + (int64_t)i * lo->B + t) * HD + x) * lo->e + c;
                                int64_t dst = kv * lo->kv_stride + blk * lo->block_stride
                                    + ((int64_t)t * HD + x) * lo->e + c;
                                layers[l][dst] = staging[src];
                            }
                }
    }
}

/* Store: the same walk with source and destination exchanged (paged blocks
 * of request req's chunk -> staging slot). */
void or_store_gather(const or_layout *lo, uint8_t *staging, const uint8_t *const *layers,
                     const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                     const or_job *jobs, int32_t num_jobs)
{
    int64_t HD = (int64_t)lo->H * lo->D;
    int64_t slot_bytes = (int64_t)lo->L * 2 * lo->C * HD * lo->e;
    int32_t nseg = lo->C / lo->B;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        for (int32_t l = 0; l < lo->L; l++)
            for (int32_t kv = 0; kv < 2; kv++)
                for (int32_t i = 0; i < nseg; i++) {
                    int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i];
                    if (blk < 0 || blk >= lo->num_blocks) continue;
                    for (int32_t t = 0; t < lo->B; t++)
                        for (int64_t x = 0; x < HD; x++)
                            for (int32_t c = 0; c < lo->e; c++) {
                                int64_t dst = jb->slot * slot_bytes
                                    + ((((int64_t)l * 2 + kv) * lo->C + (int64_t)i * lo->B + t) * HD + x) * lo->e + c;
                                int64_t src = kv * lo->kv_stride + blk * lo->block_stride
                                    + ((int64_t)t * HD + x) * lo->e + c;
                                staging[dst] = layers[l][src];
                            }
                }
    }
}

/* One-layer forms of the two copies, for complete checks of buffers too large
 * to hold on the host at once: the walk of or_retrieve_scatter and
 * or_store_gather for the single layer `layer`, with the staging side given
 * as that layer's part of every slot, back to back:
 *   stg_layer byte s*(2*C*H*D*e) + ((kv*C + i*B + t)*H*D + x)*e + c
 *     is staging byte s*slot_bytes + (((layer*2 + kv)*C + i*B + t)*H*D + x)*e + c
 * and `paged` that layer's paged tensor.  The job and block checks are those
 * of the full walks. */
void or_retrieve_scatter_layer(const or_layout *lo, const uint8_t *stg_layer, uint8_t *paged,
                               const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                               const or_job *jobs, int32_t num_jobs)
{
    int64_t HD = (int64_t)lo->H * lo->D;
    int64_t part_bytes = (int64_t)2 * lo->C * HD * lo->e;    /* one layer of one slot */
    int32_t nseg = lo->C / lo->B;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        for (int32_t kv = 0; kv < 2; kv++)
            for (int32_t i = 0; i < nseg; i++) {
                int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i];
                if (blk < 0 || blk >= lo->num_blocks) continue;
                for (int32_t t = 0; t < lo->B; t++)
                    for (int64_t x = 0; x < HD; x++)
                        for (int32_t c = 0; c < lo->e; c++) {
                            int64_t src = jb->slot * part_bytes
                                + (((int64_t)kv * lo->C + (int64_t)i * lo->B + t) * HD + x) * lo->e + c;
                            int64_t dst = kv * lo->kv_stride + blk * lo->block_stride
                                + ((int64_t)t * HD + x) * lo->e + c;
                            paged[dst] = stg_layer[src];
                        }
            }
    }
}

void or_store_gather_layer(const or_layout *lo, uint8_t *stg_layer, const uint8_t *paged,
                           const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                           const or_job *jobs, int32_t num_jobs)
{
    int64_t HD = (int64_t)lo->H * lo->D;
    int64_t part_bytes = (int64_t)2 * lo->C * HD * lo->e;
    int32_t nseg = lo->C / lo->B;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        for (int32_t kv = 0; kv < 2; kv++)
            for (int32_t i = 0; i < nseg; i++) {
                int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i];
                if (blk < 0 || blk >= lo->num_blocks) continue;
                for (int32_t t = 0; t < lo->B; t++)
                    for (int64_t x = 0; x < HD; x++)
                        for (int32_t c = 0; c < lo->e; c++) {
                            int64_t dst = jb->slot * part_bytes
                                + (((int64_t)kv * lo->C + (int64_t)i * lo->B + t) * HD + x) * lo->e + c;
                            int64_t src = kv * lo->kv_stride + blk * lo->block_stride
                                + ((int64_t)t * HD + x) * lo->e + c;
                            stg_layer[dst] = paged[src];
                        }
            }
    }
}

/* One-by-one forms of the two copies, for sampled checks on buffers too large
 * to hold twice on the host.  They scan the job list in order; the last job
 * that reaches the asked-for location decides (with disjoint destinations,
 * which callers guarantee, at most one does).
 *
 * or_scatter_source: where does paged block (layer, kv, blk) get its bytes?
 *   Returns 1 and the staging byte offset of the B-token segment copied there,
 *   or 0 if no job writes it. */
int or_scatter_source(const or_layout *lo, const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                      const or_job *jobs, int32_t num_jobs, int32_t layer, int32_t kv, int64_t blk,
                      int64_t *src_off)
{
    int64_t HD = (int64_t)lo->H * lo->D;
    int64_t slot_bytes = (int64_t)lo->L * 2 * lo->C * HD * lo->e;
    int32_t nseg = lo->C / lo->B;
    int found = 0;
    if (blk < 0 || blk >= lo->num_blocks) return 0;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        for (int32_t i = 0; i < nseg; i++) {
            if (bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i] != blk) continue;
            *src_off = jb->slot * slot_bytes + (((int64_t)layer * 2 + kv) * lo->C + (int64_t)i * lo->B) * HD * lo->e;
            found = 1;
        }
    }
    return found;
}

/* or_gather_source: which paged block lands in staging (slot, layer, kv,
 * segment i)?  Returns 1 and the block id, or 0 if no job writes there. */
int or_gather_source(const or_layout *lo, const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                     const or_job *jobs, int32_t num_jobs, int32_t slot, int32_t seg, int32_t *blk_out)
{
    int32_t nseg = lo->C / lo->B;
    int found = 0;
    if (seg < 0 || seg >= nseg) return 0;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (!or_job_ok(lo, jb, num_reqs, bt_stride)) continue;
        if (jb->slot != slot) continue;
        int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + seg];
        if (blk < 0 || blk >= lo->num_blocks) continue;
        *blk_out = blk;
        found = 1;
    }
    return found;
}

/* ------------------------------------------------------------------------- */
/* Validity of a job batch: the only races a copy launch can have            */
/* ------------------------------------------------------------------------- */

/* Jobs of one launch run concurrently, so two of them must not write the same
 * bytes: in the scatter the destinations are paged blocks (a job writes block
 * bt[req][chunk*C/B + i] of both planes of every layer, so two (job, segment)
 * pairs naming one block id race), in the gather they are staging slots (two
 * jobs naming one slot race); any number of jobs may read one slot or block.
 * A batch is
 *   OR_VERANGE  if some job has its slot, request or chunk out of range or a
 *               non-zero reserved field, or names (with those fields in range)
 *               a block id outside [0, num_blocks);
 *   OR_VEDUP    otherwise, if two of its destinations coincide;
 *   OR_VOK      otherwise.
 * The duplicate test compares every pair of destinations. */
enum { OR_VOK = 0, OR_VERANGE = -3, OR_VEDUP = -6 };

int or_validate_jobs(const or_layout *lo, const int32_t *bt, int32_t bt_stride, int32_t num_reqs,
                     const or_job *jobs, int32_t num_jobs, int is_store)
{
    int32_t nseg = lo->C / lo->B;
    for (int32_t q = 0; q < num_jobs; q++) {
        const or_job *jb = &jobs[q];
        if (jb->reserved != 0 || !or_job_ok(lo, jb, num_reqs, bt_stride)) return OR_VERANGE;
        for (int32_t i = 0; i < nseg; i++) {
            int32_t blk = bt[(int64_t)jb->req * bt_stride + (int64_t)jb->chunk * nseg + i];
            if (blk < 0 || blk >= lo->num_blocks) return OR_VERANGE;
        }
    }
    for (int32_t q = 0; q < num_jobs; q++) {
        for (int32_t p = 0; p < q; p++) {
            if (is_store) {
                if (jobs[p].slot == jobs[q].slot) return OR_VEDUP;
                continue;
            }
            for (int32_t i = 0; i < nseg; i++)
                for (int32_t k = 0; k < nseg; k++)
                    if (bt[(int64_t)jobs[q].req * bt_stride + (int64_t)jobs[q].chunk * nseg + i]
                        == bt[(int64_t)jobs[p].req * bt_stride + (int64_t)jobs[p].chunk * nseg + k])
                        return OR_VEDUP;
        }
        /* two segments of one job naming the same block */
        if (!is_store)
            for (int32_t i = 0; i < nseg; i++)
                for (int32_t k = 0; k < i; k++)
                    if (bt[(int64_t)jobs[q].req * bt_stride + (int64_t)jobs[q].chunk * nseg + i]
                        == bt[(int64_t)jobs[q].req * bt_stride + (int64_t)jobs[q].chunk * nseg + k])
                        return OR_VEDUP;
    }
    return OR_VOK;
}

/* ------------------------------------------------------------------------- */
/* Commitment decision (Section 3.2)                                          */
/* ------------------------------------------------------------------------- */

enum { OR_DEFER = 0, OR_COMMIT = 1, OR_BLOCKED = 2, OR_ORDINARY = 3, OR_EINVAL = -1 };

/* Eligibility: laxity TTU - TTR <= 0, evaluated as TTU <= TTR so that it also
 * holds for infinite estimates, or retrieval requested.  Capacity: the whole
 * claim footprint must fit the protected budget, and the bytes the claim
 * newly reserves (those no earlier commitment protects yet) must fit
 * the free protected capacity.  An eligible claim that does not fit stays
 * PLANNED (BLOCKED) unless retrieval was requested, in which case it takes
 * the ordinary retrieval path (ORDINARY). */
int or_commit_should_stage(double ttu, double ttr, uint64_t free_protected_bytes,
                           uint64_t claim_new_bytes, uint64_t claim_total_bytes,
                           uint64_t budget_bytes, int retrieval_requested)
{
    if (isnan(ttu) || isnan(ttr)) return OR_EINVAL;
    if (claim_new_bytes > claim_total_bytes) return OR_EINVAL;
    int eligible = (ttu <= ttr) || (retrieval_requested != 0);
    if (!eligible) return OR_DEFER;
    int fits = (claim_total_bytes <= budget_bytes) && (claim_new_bytes <= free_protected_bytes);
    if (fits) return OR_COMMIT;
    return retrieval_requested ? OR_ORDINARY : OR_BLOCKED;
}

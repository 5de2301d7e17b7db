/* Sanitizer driver for the oracle (test infrastructure): calls every oracle
 * function on random small inputs and checks a few identities, so that a
 * build with -fsanitize=address,undefined exercises all of its code. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

typedef struct { int32_t slot, req, chunk, reserved; } or_job;
typedef struct { int32_t L, H, D, e, B, C; int64_t num_blocks, num_slots, kv_stride, block_stride; } or_layout;
uint64_t or_mix64(uint64_t);
int or_hash_prefix(const int32_t *, const int64_t *, int32_t, uint64_t, const int64_t *, uint64_t *);
int or_lookup(const uint64_t *, const int32_t *, int64_t, const uint64_t *, const int64_t *, int32_t, int32_t,
              const int64_t *, int32_t *, int32_t *);
int or_build_jobs(const int32_t *, const int32_t *, const uint64_t *, const int64_t *, const int64_t *, int32_t,
                  int32_t, const int32_t *, int32_t, or_job *, int32_t *, or_job *, uint64_t *, int32_t *, int32_t *);
void or_retrieve_scatter(const or_layout *, const uint8_t *, uint8_t *const *, const int32_t *, int32_t, int32_t,
                         const or_job *, int32_t);
void or_store_gather(const or_layout *, uint8_t *, const uint8_t *const *, const int32_t *, int32_t, int32_t,
                     const or_job *, int32_t);
int or_scatter_source(const or_layout *, const int32_t *, int32_t, int32_t, const or_job *, int32_t, int32_t, int32_t,
                      int64_t, int64_t *);
int or_gather_source(const or_layout *, const int32_t *, int32_t, int32_t, const or_job *, int32_t, int32_t, int32_t,
                     int32_t *);
int or_commit_should_stage(double, double, uint64_t, uint64_t, uint64_t, uint64_t, int);

static uint64_t rs = 88172645463325252ull;
static uint64_t rnd(void) { rs ^= rs << 13; rs ^= rs >> 7; rs ^= rs << 17; return rs; }

int main(void)
{
    for (int trial = 0; trial < 200; trial++) {
        int R = 1 + (int)(rnd() % 5);
        int64_t tok_off[8], blk_off[8], chunk_off[8];
        tok_off[0] = blk_off[0] = chunk_off[0] = 0;
        const int bpc = 2;   /* chunk of 32 tokens */
        for (int r = 0; r < R; r++) {
            int64_t n = (int64_t)(rnd() % 140);
            tok_off[r + 1] = tok_off[r] + n;
            blk_off[r + 1] = blk_off[r] + n / 16;
            chunk_off[r + 1] = chunk_off[r] + (n / 16) / bpc;
        }
        int32_t *toks = malloc(sizeof(int32_t) * (size_t)(tok_off[R] + 1));
        for (int64_t i = 0; i < tok_off[R]; i++) toks[i] = (int32_t)(rnd() % 3);
        uint64_t *bh = malloc(sizeof(uint64_t) * (size_t)(blk_off[R] + 1));
        if (or_hash_prefix(toks, tok_off, R, rnd(), blk_off, bh) != 0) return 1;
        uint64_t keys[4];
        int32_t slots[4];
        int nk = 0;
        for (int64_t b = bpc - 1; b < blk_off[R] && nk < 4; b += bpc) { keys[nk] = bh[b]; slots[nk] = nk; nk++; }
        int64_t nch = chunk_off[R];
        int32_t *cs = malloc(sizeof(int32_t) * (size_t)(nch + 1)), hit[8];
        if (or_lookup(keys, slots, nk, bh, blk_off, R, bpc, chunk_off, cs, hit) != 0) return 2;
        int32_t freel[3] = {10, 11, 12};
        or_job *retr = malloc(sizeof(or_job) * (size_t)(nch + 1)), *store = malloc(sizeof(or_job) * (size_t)(nch + 1));
        uint64_t *sk = malloc(sizeof(uint64_t) * (size_t)(nch + 1));
        int32_t nr, ns, nd;
        if (or_build_jobs(hit, cs, bh, blk_off, chunk_off, R, bpc, freel, 3, retr, &nr, store, sk, &ns, &nd)) return 3;
        free(toks); free(bh); free(cs); free(retr); free(store); free(sk);
    }
    /* copies: 2 layers, 2 heads, 16 dims, 2 bytes, B 16, C 32 */
    or_layout lo = {2, 2, 16, 2, 16, 32, 9, 3, 0, 0};
    int64_t seg = 16 * 2 * 16 * 2;
    lo.kv_stride = 9 * seg;
    lo.block_stride = seg;
    int64_t slot_bytes = 2 * 2 * 32 * 2 * 16 * 2;
    uint8_t *stg = malloc((size_t)(3 * slot_bytes)), *back = calloc(1, (size_t)(3 * slot_bytes));
    uint8_t *l0 = calloc(1, (size_t)(2 * 9 * seg)), *l1 = calloc(1, (size_t)(2 * 9 * seg));
    for (int64_t i = 0; i < 3 * slot_bytes; i++) stg[i] = (uint8_t)rnd();
    int32_t bt[2][4] = {{3, 7, 0, 5}, {8, 1, 2, 6}};
    or_job jobs[4] = {{0, 0, 0, 0}, {2, 1, 1, 0}, {1, 0, 1, 0}, {0, 5, 0, 0}};
    uint8_t *layers[2] = {l0, l1};
    or_retrieve_scatter(&lo, stg, layers, &bt[0][0], 4, 2, jobs, 4);
    or_store_gather(&lo, back, (const uint8_t *const *)layers, &bt[0][0], 4, 2, jobs, 3);
    if (memcmp(back, stg, (size_t)(3 * slot_bytes)) != 0) return 4;
    int64_t off;
    int32_t blk;
    if (!or_scatter_source(&lo, &bt[0][0], 4, 2, jobs, 4, 1, 1, 3, &off)) return 5;
    if (!or_gather_source(&lo, &bt[0][0], 4, 2, jobs, 4, 2, 1, &blk) || blk != 6) return 6;
    if (or_commit_should_stage(0.0, 1.0, 5, 1, 2, 9, 0) != 1) return 7;
    (void)or_mix64(0);
    free(stg); free(back); free(l0); free(l1);
    puts("oracle selftest ok");
    return 0;
}

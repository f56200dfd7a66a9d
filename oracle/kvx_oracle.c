/*
 * CPU oracle for the shared-KV store/load path -- TEST INFRASTRUCTURE ONLY.
 * (Called only by tests/, __graft_entry__.smoke() and the benchmark's CPU
 * baseline; never by the product path.  Shares no code with the HIP library.)
 *
 * Plain, slow, obviously correct: every copied row is located by explicit
 * index arithmetic straight from the definition in kvx_oracle.h, in the order
 * chunk -> layer -> K/V -> token -> head.  The copy is one memcpy of D*E
 * opaque bytes per (token, head) row; values never pass through a float.
 *
 * Paper grounding: Sec. 2.2 (state is opaque addressable bytes; attention
 * contributes the K/V pages preceding a prefix boundary), Sec. 3.1 (a logical
 * chunk is a whole number of paged blocks; layout constraints are validated).
 */
#include "kvx_oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

int64_t oracle_slot_bytes(const oracle_layout *lay)
{
    if (!lay || lay->num_layers <= 0 || lay->num_kv_heads <= 0 || lay->head_dim <= 0 ||
        lay->elem_bytes <= 0 || lay->block_size <= 0 || lay->chunk_tokens <= 0)
        return -1;
    int64_t token_bytes = 2LL * lay->num_layers * lay->num_kv_heads * lay->head_dim * lay->elem_bytes;
    return (int64_t)lay->chunk_tokens * token_bytes;
}

int oracle_validate(const oracle_layout *lay, int64_t num_blocks, int64_t block_stride,
                    const int32_t *block_table, int64_t n_tokens, int64_t num_slots,
                    const int64_t *chunk_ids, int for_pack)
{
    if (oracle_slot_bytes(lay) < 0)
        return ORACLE_EINVAL;
    int64_t E = lay->elem_bytes;
    if (E != 1 && E != 2 && E != 4)
        return ORACLE_EINVAL;
    /* Sec. 3.1: a chunk must be a whole number of pages. */
    if (lay->chunk_tokens % lay->block_size != 0)
        return ORACLE_EINVAL;
    if (n_tokens < 0 || num_blocks <= 0 || num_slots < 0)
        return ORACLE_EINVAL;
    int64_t block_bytes = 2LL * lay->num_kv_heads * lay->block_size * lay->head_dim * E;
    if (block_stride < block_bytes)
        return ORACLE_EINVAL;
    if (n_tokens == 0)
        return ORACLE_OK;
    if (!block_table || !chunk_ids)
        return ORACLE_EINVAL;

    int64_t BS = lay->block_size, C = lay->chunk_tokens;
    int64_t n_blocks_used = (n_tokens + BS - 1) / BS;
    for (int64_t k = 0; k < n_blocks_used; ++k)
        if (block_table[k] < 0 || block_table[k] >= num_blocks)
            return ORACLE_EINVAL;

    int64_t nc = (n_tokens + C - 1) / C;
    for (int64_t i = 0; i < nc; ++i)
        if (chunk_ids[i] < 0 || chunk_ids[i] >= num_slots)
            return ORACLE_EINVAL;
    if (for_pack) {
        /* Two chunks written to one slot would make the result order dependent. */
        for (int64_t i = 0; i < nc; ++i)
            for (int64_t j = i + 1; j < nc; ++j)
                if (chunk_ids[i] == chunk_ids[j])
                    return ORACLE_EINVAL;
    }
    return ORACLE_OK;
}

/* Everything one worker needs; chunks [first, last) are its share. */
typedef struct oracle_job {
    const oracle_layout *lay;
    int block_order;
    uint8_t *const *cache_layers; /* written by unpack, read by pack */
    int64_t block_stride;
    const int32_t *block_table;
    int64_t n_tokens;
    uint8_t *pool;                /* written by pack, read by unpack */
    const int64_t *chunk_ids;
    int64_t first, last;
    int to_pool;                  /* 1 = pack, 0 = unpack */
} oracle_job;

/* Byte offset of cache row (kv, h, slot s) inside block b of one layer. */
static int64_t cache_row_offset(const oracle_layout *lay, int block_order, int64_t block_stride,
                                int64_t b, int64_t kv, int64_t h, int64_t s)
{
    int64_t H = lay->num_kv_heads, BS = lay->block_size;
    int64_t row_bytes = (int64_t)lay->head_dim * lay->elem_bytes;
    if (block_order == ORACLE_BLOCK_NHD)
        return b * block_stride + ((kv * BS + s) * H + h) * row_bytes;
    return b * block_stride + ((kv * H + h) * BS + s) * row_bytes;
}

/* Byte offset of chunk row (l, kv, u, h) inside a slot holding r tokens. */
static int64_t chunk_row_offset(const oracle_layout *lay, int64_t r, int64_t l, int64_t kv,
                                int64_t u, int64_t h)
{
    int64_t H = lay->num_kv_heads;
    int64_t row_bytes = (int64_t)lay->head_dim * lay->elem_bytes;
    return (((l * 2 + kv) * r + u) * H + h) * row_bytes;
}

static void *oracle_worker(void *arg)
{
    const oracle_job *job = (const oracle_job *)arg;
    const oracle_layout *lay = job->lay;
    int64_t L = lay->num_layers, H = lay->num_kv_heads, BS = lay->block_size, C = lay->chunk_tokens;
    int64_t row_bytes = (int64_t)lay->head_dim * lay->elem_bytes;
    int64_t slot_bytes = oracle_slot_bytes(lay);

    for (int64_t i = job->first; i < job->last; ++i) {
        int64_t r = job->n_tokens - i * C;          /* tokens in chunk i */
        if (r > C)
            r = C;
        uint8_t *slot = job->pool + job->chunk_ids[i] * slot_bytes;
        for (int64_t l = 0; l < L; ++l) {
            uint8_t *layer = job->cache_layers[l];
            for (int64_t kv = 0; kv < 2; ++kv) {
                for (int64_t u = 0; u < r; ++u) {
                    int64_t t = i * C + u;           /* logical token */
                    int64_t b = job->block_table[t / BS];
                    int64_t s = t % BS;
                    for (int64_t h = 0; h < H; ++h) {
                        uint8_t *cache_row =
                            layer + cache_row_offset(lay, job->block_order, job->block_stride, b, kv, h, s);
                        uint8_t *chunk_row = slot + chunk_row_offset(lay, r, l, kv, u, h);
                        if (job->to_pool)
                            memcpy(chunk_row, cache_row, (size_t)row_bytes);
                        else
                            memcpy(cache_row, chunk_row, (size_t)row_bytes);
                    }
                }
            }
        }
    }
    return NULL;
}

static int oracle_run(const oracle_layout *lay, int block_order, uint8_t *const *layers,
                      int64_t num_blocks, int64_t block_stride, const int32_t *block_table,
                      int64_t n_tokens, uint8_t *pool, int64_t num_slots,
                      const int64_t *chunk_ids, int nthreads, int to_pool)
{
    if (block_order != ORACLE_BLOCK_HND && block_order != ORACLE_BLOCK_NHD)
        return ORACLE_EINVAL;
    int rc = oracle_validate(lay, num_blocks, block_stride, block_table, n_tokens, num_slots,
                             chunk_ids, to_pool);
    if (rc != ORACLE_OK)
        return rc;
    if (n_tokens == 0)
        return ORACLE_OK;
    if (!layers || !pool)
        return ORACLE_EINVAL;
    for (int32_t l = 0; l < lay->num_layers; ++l)
        if (!layers[l])
            return ORACLE_EINVAL;

    int64_t nc = (n_tokens + lay->chunk_tokens - 1) / lay->chunk_tokens;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > nc)
        nthreads = (int)nc;

    oracle_job *jobs = (oracle_job *)calloc((size_t)nthreads, sizeof(oracle_job));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !tids) {
        free(jobs);
        free(tids);
        return ORACLE_EINVAL;
    }
    for (int k = 0; k < nthreads; ++k) {
        jobs[k].lay = lay;
        jobs[k].block_order = block_order;
        jobs[k].cache_layers = layers;
        jobs[k].block_stride = block_stride;
        jobs[k].block_table = block_table;
        jobs[k].n_tokens = n_tokens;
        jobs[k].pool = pool;
        jobs[k].chunk_ids = chunk_ids;
        jobs[k].first = nc * k / nthreads;
        jobs[k].last = nc * (k + 1) / nthreads;
        jobs[k].to_pool = to_pool;
    }
    int started = 0;
    for (int k = 1; k < nthreads; ++k) {
        if (pthread_create(&tids[k], NULL, oracle_worker, &jobs[k]) != 0)
            break;
        started = k;
    }
    oracle_worker(&jobs[0]);
    for (int k = 1; k <= started; ++k)
        pthread_join(tids[k], NULL);
    /* A thread that failed to start leaves its share to this thread. */
    for (int k = started + 1; k < nthreads; ++k)
        oracle_worker(&jobs[k]);
    free(jobs);
    free(tids);
    return ORACLE_OK;
}

int oracle_pack(const oracle_layout *lay, int block_order, const uint8_t *const *layer_ptrs,
                int64_t num_blocks, int64_t block_stride, const int32_t *block_table,
                int64_t n_tokens, uint8_t *pool, int64_t num_slots, const int64_t *chunk_ids,
                int nthreads)
{
    /* The cache is only read in this direction. */
    return oracle_run(lay, block_order, (uint8_t *const *)layer_ptrs, num_blocks, block_stride,
                      block_table, n_tokens, pool, num_slots, chunk_ids, nthreads, 1);
}

int oracle_unpack(const oracle_layout *lay, int block_order, uint8_t *const *layer_ptrs,
                  int64_t num_blocks, int64_t block_stride, const int32_t *block_table,
                  int64_t n_tokens, const uint8_t *pool, int64_t num_slots,
                  const int64_t *chunk_ids, int nthreads)
{
    /* The pool is only read in this direction. */
    return oracle_run(lay, block_order, layer_ptrs, num_blocks, block_stride, block_table,
                      n_tokens, (uint8_t *)pool, num_slots, chunk_ids, nthreads, 0);
}

/* ---- Recurrent-state snapshot pages (Sec. 2.2) ---------------------------------- */

int oracle_state_validate(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                          const int64_t *pages, int64_t n, int64_t num_state_slots, const int64_t *slot_ids,
                          int for_pack)
{
    if (num_layers < 1 || page_bytes < 1 || page_stride < page_bytes || num_pages < 1 || n < 0 ||
        num_state_slots < 0)
        return ORACLE_EINVAL;
    if (n == 0)
        return ORACLE_OK;
    if (!pages || !slot_ids)
        return ORACLE_EINVAL;
    for (int64_t k = 0; k < n; ++k) {
        if (pages[k] < 0 || pages[k] >= num_pages)
            return ORACLE_EINVAL;
        if (slot_ids[k] < 0 || slot_ids[k] >= num_state_slots)
            return ORACLE_EINVAL;
    }
    /* The side written must not be named twice. */
    const int64_t *written = for_pack ? slot_ids : pages;
    for (int64_t k = 0; k < n; ++k)
        for (int64_t m = k + 1; m < n; ++m)
            if (written[k] == written[m])
                return ORACLE_EINVAL;
    return ORACLE_OK;
}

static int oracle_state_run(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                            uint8_t *const *state_layers, const int64_t *pages, int64_t n, uint8_t *state_pool,
                            int64_t num_state_slots, const int64_t *slot_ids, int to_pool)
{
    int rc = oracle_state_validate(num_layers, page_bytes, page_stride, num_pages, pages, n, num_state_slots,
                                   slot_ids, to_pool);
    if (rc != ORACLE_OK)
        return rc;
    if (n == 0)
        return ORACLE_OK;
    if (!state_layers || !state_pool)
        return ORACLE_EINVAL;
    for (int64_t g = 0; g < num_layers; ++g)
        if (!state_layers[g])
            return ORACLE_EINVAL;
    int64_t snapshot_bytes = num_layers * page_bytes;
    for (int64_t k = 0; k < n; ++k) {
        uint8_t *slot = state_pool + slot_ids[k] * snapshot_bytes;
        for (int64_t g = 0; g < num_layers; ++g) {
            uint8_t *page = state_layers[g] + pages[k] * page_stride;
            uint8_t *packed = slot + g * page_bytes;
            if (to_pool)
                memcpy(packed, page, (size_t)page_bytes);
            else
                memcpy(page, packed, (size_t)page_bytes);
        }
    }
    return ORACLE_OK;
}

int oracle_state_pack(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                      const uint8_t *const *state_layers, const int64_t *pages, int64_t n,
                      uint8_t *state_pool, int64_t num_state_slots, const int64_t *slot_ids)
{
    /* The pages are only read in this direction. */
    return oracle_state_run(num_layers, page_bytes, page_stride, num_pages, (uint8_t *const *)state_layers,
                            pages, n, state_pool, num_state_slots, slot_ids, 1);
}

int oracle_state_unpack(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                        uint8_t *const *state_layers, const int64_t *pages, int64_t n,
                        const uint8_t *state_pool, int64_t num_state_slots, const int64_t *slot_ids)
{
    /* The state pool is only read in this direction. */
    return oracle_state_run(num_layers, page_bytes, page_stride, num_pages, state_layers, pages, n,
                            (uint8_t *)state_pool, num_state_slots, slot_ids, 0);
}

/*
 * CPU oracle for the shared-KV store/load path -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, __graft_entry__.smoke() and the benchmark's CPU-baseline leg
 * may call this library.  It shares no code, header, table or helper with the
 * HIP library; the GPU product path never loads it.
 *
 * What it computes (the plain definition, exact; no approximation):
 *   Paper, Sec. 2.2 -- KV state is moved as opaque bytes; full-attention layers
 *   contribute the K/V pages that precede a prefix boundary.
 *   Paper, Sec. 3.1 -- a logical chunk spans several paged cache blocks, and the
 *   chunk length must be a whole number of pages (the paper's instance: a
 *   1,568-token logical block is 49 pages of 32 tokens).
 *
 * Cache element (l, b, kv, h, s, d) sits at byte
 *     b*block_stride + ((kv*H + h)*BS + s)*D*E + d*E      of layer_ptrs[l]   (block_order 0)
 * (per-layer [NB][2][H][BS][D], "HND" as in the paper's Table 1; kv 0 = K), or at
 *     b*block_stride + ((kv*BS + s)*H + h)*D*E + d*E                       (block_order 1)
 * (per-layer [NB][2][BS][H][D], "NHD", the layout the paper's patch rejected, Sec. 3.1).
 * Token t lives in block bt[t / BS], slot t % BS.
 * Chunk i (of nc = ceil(n / C)) holds tokens [i*C, i*C + r_i), r_i = min(C, n - i*C),
 * packed plane-major [L][2][r_i][H][D] at pool + chunk_ids[i]*slot_bytes,
 * slot_bytes = C * 2*L*H*D*E.  Bytes [r_i*TB, slot_bytes) of a slot are neither
 * written by pack nor read by unpack.  Unpack is the exact inverse and touches
 * no cache byte outside the named token slots.
 */
#ifndef KVX_ORACLE_H
#define KVX_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct oracle_layout {
    int32_t num_layers;   /* L  */
    int32_t num_kv_heads; /* H  */
    int32_t head_dim;     /* D  */
    int32_t elem_bytes;   /* E  */
    int32_t block_size;   /* BS: tokens per paged block */
    int32_t chunk_tokens; /* C : tokens per packed chunk */
} oracle_layout;

/* Token order inside a cache block. */
#define ORACLE_BLOCK_HND 0 /* [2][H][BS][D] */
#define ORACLE_BLOCK_NHD 1 /* [2][BS][H][D] */

/* Error codes (negative). */
#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)

/* Bytes of one packed slot: C * 2*L*H*D*E. Returns -1 on an invalid layout. */
int64_t oracle_slot_bytes(const oracle_layout *lay);

/*
 * Validation (Sec. 3.1: layout constraints are checked, never inferred):
 * positive sizes, E in {1,2,4}, C % BS == 0, n >= 0, block_stride >= 2*H*BS*D*E,
 * every bt[0 .. ceil(n/BS)) in [0, num_blocks), every chunk id in
 * [0, num_slots), and (pack only) chunk ids pairwise distinct.
 * Returns ORACLE_OK or ORACLE_EINVAL.
 */
int oracle_validate(const oracle_layout *lay, int64_t num_blocks, int64_t block_stride,
                    const int32_t *block_table, int64_t n_tokens, int64_t num_slots,
                    const int64_t *chunk_ids, int for_pack);

/*
 * Pack (store): copy every named token row of the cache into its chunk row.
 * block_order: ORACLE_BLOCK_HND or ORACLE_BLOCK_NHD (anything else is ORACLE_EINVAL).
 * layer_ptrs: L host pointers.  pool: num_slots * slot_bytes host bytes.
 * nthreads >= 1: chunks are split over that many POSIX threads (each chunk is
 * independent).  Returns ORACLE_OK or ORACLE_EINVAL (nothing written then).
 */
int oracle_pack(const oracle_layout *lay, int block_order, const uint8_t *const *layer_ptrs,
                int64_t num_blocks, int64_t block_stride, const int32_t *block_table,
                int64_t n_tokens, uint8_t *pool, int64_t num_slots, const int64_t *chunk_ids,
                int nthreads);

/* Unpack (load): the exact inverse of oracle_pack. */
int oracle_unpack(const oracle_layout *lay, int block_order, uint8_t *const *layer_ptrs,
                  int64_t num_blocks, int64_t block_stride, const int32_t *block_table,
                  int64_t n_tokens, const uint8_t *pool, int64_t num_slots,
                  const int64_t *chunk_ids, int nthreads);

/*
 * Recurrent-state snapshot pages of a hybrid model (Sec. 2.2): each of G recurrent
 * layers keeps its boundary snapshot -- convolution state, recurrent state and
 * padding -- as one page of page_bytes opaque bytes.  Layer g's page p sits at
 * state_layers[g] + p*page_stride.  Snapshot k (pages[k] in every layer) is stored
 * in state slot slot_ids[k] of a state pool of state slots G*page_bytes bytes each,
 * layer-major: layer g's page at byte g*page_bytes of the slot.  Unpack is the
 * exact inverse; no other byte of either side is touched.
 *
 * Validation: G >= 1, page_bytes >= 1, page_stride >= page_bytes, num_pages >= 1,
 * n >= 0, every page id in [0, num_pages), every slot id in [0, num_state_slots);
 * pack: slot ids pairwise distinct; unpack: page ids pairwise distinct (either
 * repetition would make the result depend on the copy order).
 */
int oracle_state_validate(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                          const int64_t *pages, int64_t n, int64_t num_state_slots, const int64_t *slot_ids,
                          int for_pack);

int oracle_state_pack(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                      const uint8_t *const *state_layers, const int64_t *pages, int64_t n,
                      uint8_t *state_pool, int64_t num_state_slots, const int64_t *slot_ids);

int oracle_state_unpack(int64_t num_layers, int64_t page_bytes, int64_t page_stride, int64_t num_pages,
                        uint8_t *const *state_layers, const int64_t *pages, int64_t n,
                        const uint8_t *state_pool, int64_t num_state_slots, const int64_t *slot_ids);

#ifdef __cplusplus
}
#endif

#endif /* KVX_ORACLE_H */

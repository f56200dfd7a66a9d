/*
 * kvx -- store and load of paged KV state between a GPU KV cache and a pinned
 * host-memory chunk pool, on AMD Instinct MI355X (gfx950).
 *
 * The operation is the state transfer of shared host-memory KV caching between
 * inference replicas (arxiv 2609.15021): a replica stores the KV pages that
 * precede a prefix boundary into a shared host tier as packed chunks (Sec. 2,
 * Fig. 1; Sec. 2.2), and another replica loads them back into its own paged
 * cache instead of recomputing the prefix (Sec. 5.1).  Every entry point is
 * ordered against the caller's stream: omitting that dependency is the fault
 * the paper diagnoses (Sec. 3.2).
 *
 * Plain C ABI: no C++ types, no torch types; pointers are explicit host or
 * device addresses; streams are hipStream_t values passed as void*.  No entry
 * point throws; all return a kv_status (0 = success, negative = error) unless
 * stated.  kv_last_error() describes the most recent failure on the calling
 * thread.
 *
 * ---------------------------------------------------------------------------
 * Byte layout (normative; "E" = elem_bytes, all offsets 64-bit):
 *
 *  Cache: layer l is one device buffer layer_ptrs[l] holding num_blocks blocks,
 *    block b at byte b*block_stride.  Inside a block, element (kv, h, s, d) is at
 *    ((kv*H + h)*BS + s)*D*E + d*E, i.e. [2][H][BS][D] ("HND", kv 0 = K, 1 = V;
 *    the paper's replicas run HND, Table 1), or with block_order KV_BLOCK_NHD at
 *    ((kv*BS + s)*H + h)*D*E + d*E, i.e. [2][BS][H][D] (the token-major variant
 *    the paper's patch could not read, Sec. 3.1).  Token t of a prefix lives in
 *    block block_table[t / BS] at slot t % BS.  The chunk format below does not
 *    depend on the block order: caches of either order share one pool.
 *
 *  Chunks: a prefix of n tokens is cut into nc = ceil(n / C) chunks; chunk i
 *    holds tokens [i*C, i*C + r_i), r_i = min(C, n - i*C) (only the last chunk
 *    may be partial).  Chunk i is stored in pool slot chunk_ids[i], plane-major
 *    [L][2][r_i][H][D]: element (l, kv, u, h, d) at
 *    (((l*2 + kv)*r_i + u)*H + h)*D*E + d*E.  A slot is C*TB bytes, TB = 2*L*H*D*E
 *    bytes per token; a partial chunk occupies exactly its first r_i*TB bytes and
 *    the slot's remaining bytes are neither written by kv_store nor read by
 *    kv_load.  The layout is fixed by this descriptor, never inferred from a
 *    tensor's rank or shape (the representation fault of Sec. 3.1).
 *
 *  State snapshots (hybrid models, Sec. 2.2): each of G recurrent layers keeps
 *    its boundary snapshot -- convolution state, recurrent state and padding --
 *    as one page of page_bytes opaque bytes; layer g's page p sits at
 *    layer_ptrs[g] + p*page_stride on the device.  Snapshot k of a request
 *    (page pages[k] of every layer) is stored in state slot slot_ids[k] of the
 *    pool's state area, layer-major [G][page_bytes]: layer g's page at byte
 *    g*page_bytes of the slot.  A state slot is G*page_bytes bytes.  Under
 *    aligned recovery (Sec. 2.2) a prefix is restorable only where both its
 *    chunks and the snapshot at its boundary were stored; the two transfers are
 *    separate calls ordered on one stream.
 *
 * Ordering contract (Sec. 3.2 and Fig. 2):
 *  (i)   every device read (store) or write (load) of the cache, and every pool
 *        access, happens after all work enqueued on `stream` before the call;
 *  (ii)  work enqueued on `stream` after the call observes all of the call's
 *        writes (the pool for store, the cache for load);
 *  (iii) returning from a call establishes nothing: the host may touch the pool
 *        only after synchronising `stream` (or an event recorded on it after the
 *        call) -- the paper's host-side completion handling;
 *  (iv)  use of one pool from two streams is ordered by the caller (event or
 *        synchronisation), as between two replicas.
 * ---------------------------------------------------------------------------
 */
#ifndef KVX_H
#define KVX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Every entry point below is exported; everything else in the library is hidden. */
#if defined(__GNUC__) || defined(__clang__)
#define KV_API __attribute__((visibility("default")))
#else
#define KV_API
#endif

typedef int32_t kv_status;

#define KV_OK 0
#define KV_EINVAL (-1)        /* invalid argument or layout; nothing was enqueued */
#define KV_ENOMEM (-2)        /* pinned host or device allocation failed; no fallback was taken */
#define KV_EHIP (-3)          /* a HIP runtime call failed (name and message in kv_last_error) */
#define KV_EUNSUPPORTED (-4)  /* valid per the definition, but outside what the GPU path handles */
#define KV_EASYNC (-5)        /* a device-side check failed in an earlier call (kv_pool_async_error) */
#define KV_EBUSY (-6)         /* pool index: no slot can be freed (every slot is pinned or pending) */

/* Host transfer modes (chosen explicitly; nothing is selected silently, cf. Sec. 3.2). */
#define KV_MODE_ZERO_COPY 1u  /* gather/scatter kernels on `stream` access mapped pinned memory directly */
#define KV_MODE_STAGED 2u     /* pack/unpack in device staging on `stream`; DMA copies on event-gated side streams */

/* Pool memory kinds. */
#define KV_HOST_COHERENT 0u     /* fine-grained pinned memory (default) */
#define KV_HOST_NONCOHERENT 1u  /* coarse-grained pinned memory */
#define KV_POOL_DEVICE 2u       /* device memory (HBM) of the current device, no host address: kv_store and
                                   kv_load are then the pack/unpack kernels alone, device to device.  For a
                                   device-resident chunk tier, the first hop of a peer (xGMI) exchange, and the
                                   kernels' HBM roofline without the host link.  Zero-copy mode only. */

/* Token order inside a cache block (kv_cache.block_order). */
#define KV_BLOCK_HND 0  /* [2][H][BS][D] */
#define KV_BLOCK_NHD 1  /* [2][BS][H][D] */

/* Async error bits reported by kv_pool_async_error. */
#define KV_ASYNC_BAD_BLOCK 1   /* a block_table entry was outside [0, num_blocks): no cache byte of it was
                                  touched; a store wrote zeros for its chunk rows */

/* Tokens' geometry; identical for a cache and the pool it talks to. */
typedef struct kv_layout {
    int32_t num_layers;   /* L  >= 1 */
    int32_t num_kv_heads; /* H  >= 1 */
    int32_t head_dim;     /* D  >= 1 */
    int32_t elem_bytes;   /* E in {1, 2, 4}; values are moved as opaque bytes */
    int32_t block_size;   /* BS >= 1: tokens per paged block */
    int32_t chunk_tokens; /* C  >= 1: tokens per packed chunk; C % BS == 0 (Sec. 3.1) */
} kv_layout;

/* A replica's paged KV cache.  The caller owns all memory it names. */
typedef struct kv_cache {
    kv_layout layout;
    int32_t num_blocks;          /* blocks per layer buffer */
    int32_t device;              /* HIP device ordinal the buffers live on */
    int32_t block_order;         /* KV_BLOCK_HND or KV_BLOCK_NHD */
    int32_t reserved;            /* must be 0 */
    void *const *layer_ptrs;     /* HOST array of num_layers DEVICE pointers, read during the call only */
    int64_t block_stride_bytes;  /* bytes between blocks; 0 = packed (2*H*BS*D*E) */
} kv_cache;

/* Pool creation options.  Zero-initialised fields take the documented defaults. */
typedef struct kv_pool_options {
    uint32_t mode;             /* KV_MODE_ZERO_COPY or KV_MODE_STAGED (required, no default) */
    uint32_t host_kind;        /* KV_HOST_COHERENT (0), KV_HOST_NONCOHERENT or KV_POOL_DEVICE */
    int32_t staging_slots;     /* staged ring depth K >= 2 per direction (default 3; stores and loads
                                  each have their own ring); with mode zero-copy, > 0 also allocates
                                  staging so kv_pool_set_mode can switch later */
    int32_t chunks_per_batch;  /* chunks per staging slot / per kernel launch, 1..256 (default 16
                                  staged and for a device pool, 256 zero-copy); applies to the mode
                                  given here */
    int32_t side_streams;      /* staged: DMA side streams per direction, 1..8 (default 1) */
    int32_t profile;           /* nonzero: time every pack/unpack launch (kv_pool_kernel_stats) */
    int64_t num_state_slots;   /* state-snapshot slots (0 = no state area) */
    int64_t state_slot_bytes;  /* bytes of one state slot = G*page_bytes, a multiple of 16 (0 if none) */
} kv_pool_options;

typedef struct kv_pool kv_pool;

typedef struct kv_pool_info {
    int64_t num_slots;
    int64_t slot_bytes;        /* C * TB */
    int64_t pool_bytes;        /* num_slots * slot_bytes, pinned as one region */
    int64_t staging_bytes;     /* device staging of both directions (0 without staging) */
    double alloc_seconds;      /* wall time of the pinned allocation (cf. Sec. 3.3) */
    int32_t device;
    uint32_t mode;             /* mode of stores (and of loads unless kv_pool_set_modes split them) */
    uint32_t host_kind;
    int32_t is_pinned;         /* 1: the runtime reports the pool as pinned host memory (0 for a
                                  KV_POOL_DEVICE pool) */
    int32_t staging_slots;
    int32_t chunks_per_batch;
    int32_t side_streams;
    int32_t staging_contiguous; /* always 0: staging is plain device memory (field kept for layout) */
    void *host_base;           /* host address of slot 0 (NULL for a KV_POOL_DEVICE pool) */
    void *device_base;         /* device address of slot 0 (mapped pinned memory, or HBM) */
    int64_t num_state_slots;
    int64_t state_slot_bytes;
    void *state_host_base;     /* host address of state slot 0 (NULL without a state area); the
                                  state area follows the chunk slots in the same pinned region */
    uint32_t load_mode;        /* mode of loads; `mode` above is the mode of stores */
    uint32_t pad;
} kv_pool_info;

/* A replica's recurrent-state page buffers (hybrid models).  The caller owns all memory. */
typedef struct kv_state {
    int32_t num_layers;        /* G >= 1 recurrent layers */
    int32_t device;            /* HIP device ordinal the buffers live on */
    int64_t page_bytes;        /* bytes of one layer's snapshot page (opaque) */
    int64_t page_stride;       /* bytes between pages in a layer buffer; 0 = page_bytes */
    int64_t num_pages;         /* pages per layer buffer */
    void *const *layer_ptrs;   /* HOST array of G DEVICE pointers, read during the call only */
} kv_state;

/*
 * kv_pool_create -- allocate the shared host tier (Sec. 2: a host-RAM pool
 * shared by the replicas; Sec. 3.3: the full pool must really be pinned).
 * Pins exactly num_slots * slot_bytes bytes as ONE region (Sec. 3.2 notes a
 * workaround registering the whole pool together), mapped for device access,
 * verifies with the runtime that it is pinned, and times the allocation.  On
 * the current HIP device it creates, for stores and for loads separately, a
 * staging ring, side streams (default priority, non-blocking) and events, so
 * that a store and a load in flight at once do not wait for each other.  Never falls back to pageable memory:
 * failure is KV_ENOMEM.  *out receives the pool (owned by the library until
 * kv_pool_destroy).  With host_kind KV_POOL_DEVICE the same region is device
 * memory of the current device instead (hipMalloc; is_pinned 0, no host
 * address, kv_pool_slot returns NULL); the mode must be KV_MODE_ZERO_COPY and
 * no staging is made.  Errors: KV_EINVAL (layout, num_slots <= 0, options),
 * KV_ENOMEM, KV_EHIP.
 */
KV_API kv_status kv_pool_create(const kv_layout *layout, int64_t num_slots, const kv_pool_options *opts,
                         kv_pool **out);

/* Waits until every store/load enqueued on the pool has completed on its caller stream
 * and the pool's side streams are idle, then frees everything: no memory an enqueued
 * kernel or copy may still touch is released early (Sec. 3.2 cites premature reuse of
 * asynchronous-copy buffers as a related failure).  NULL is a no-op.  Errors: KV_EHIP
 * (the first failing runtime call; teardown continues past it). */
KV_API kv_status kv_pool_destroy(kv_pool *pool);

/* Fills *info: sizes, the modes in use, and whether the runtime reports the pool as pinned
 * with its allocation time (Sec. 3.3: the full pool must really be pinned, and the paper times
 * that allocation).  KV_EINVAL on NULL arguments. */
KV_API kv_status kv_pool_get_info(const kv_pool *pool, kv_pool_info *info);

/* Host address of state slot `slot` (NULL if out of range or without a state area).  As for
 * kv_pool_slot, touch it only after the host has seen every call using it complete (Sec. 3.2). */
KV_API void *kv_pool_state_slot(kv_pool *pool, int64_t slot);

/* Host address of a slot (NULL if out of range or pool NULL), for the host-side consumer
 * of stored chunks.  Host-side completion handling precedes host consumption (Sec. 3.2 and
 * the Fig. 2 caption): read or write a slot only after synchronising the stream (or an
 * event recorded on it) of every call that uses it; returning from kv_store establishes
 * nothing.  The address stays valid until kv_pool_destroy. */
KV_API void *kv_pool_slot(kv_pool *pool, int64_t slot);
/* Bytes of one slot, C*TB (Sec. 3.1: the chunk is a logical view over whole blocks), and
 * the pool's slot count (Sec. 2: a fixed-size host tier).  -1 on NULL. */
KV_API int64_t kv_pool_slot_bytes(const kv_pool *pool);
KV_API int64_t kv_pool_num_slots(const kv_pool *pool);

/* Switch mode between calls, for stores and loads alike.  The transfer path is chosen by the
 * pool's owner and reported in kv_pool_info, never selected silently (Sec. 3.2: a CLI default
 * selected the allocator whose raw-pointer fallback dropped the stream dependency).  Both modes
 * keep the ordering contract.  Affects calls made after it returns; calls already enqueued keep
 * their mode.  KV_EINVAL for a NULL pool, an unknown mode or staged mode without staging. */
KV_API kv_status kv_pool_set_mode(kv_pool *pool, uint32_t mode);

/* Switch mode between calls, separately for stores and loads (e.g. a tier that stores staged and
 * restores zero-copy, the faster mode of each direction across processes).  The pool reports both
 * in kv_pool_info.  Same errors as kv_pool_set_mode. */
KV_API kv_status kv_pool_set_modes(kv_pool *pool, uint32_t store_mode, uint32_t load_mode);

/*
 * Device-side faults seen since the last clear (bitmask of KV_ASYNC_*; 0 if
 * none), meaningful after the caller has synchronised the streams it used.  A
 * zero result is not an integrity check (Sec. 1: success signals are not).
 * clear != 0 resets the word.  Returns the mask, or KV_EINVAL on NULL.
 */
KV_API int32_t kv_pool_async_error(kv_pool *pool, int clear);

/*
 * Accumulated pack (which = 0), unpack (1), state pack (2) or state unpack (3) kernel time of a pool
 * created with opts.profile != 0.  Call after synchronising the streams used;
 * each launch's start/end events were recorded on the caller stream around it.
 * *launches, *total_ms and *bytes (algorithmic bytes: payload read + written)
 * receive the totals since the last reset (reset != 0 clears them).
 */
KV_API kv_status kv_pool_kernel_stats(kv_pool *pool, int which, int reset, int64_t *launches, double *total_ms,
                               double *bytes);

/*
 * Host-only validation of a store/load request, no HIP call (Sec. 3.1: layout
 * constraints are validated, never inferred).  Checks: cache layout equals
 * pool_layout field by field; positive sizes; E in {1,2,4}; C % BS == 0;
 * block_stride 0 or >= 2*H*BS*D*E; block_order KV_BLOCK_HND or KV_BLOCK_NHD
 * and reserved 0; n_tokens >= 0; for n_tokens > 0 non-NULL
 * layer pointers and chunk_ids, chunk ids in [0, pool_slots), and for a store
 * pairwise distinct (duplicates make the result order dependent).  GPU-path
 * limits give KV_EUNSUPPORTED: D*E % 16 != 0, a layer pointer or
 * block_stride not 16-byte aligned, more than 2^31-1 slots, a block
 * (2*H*BS*D*E bytes) over 2 GiB.
 * Returns KV_OK / KV_EINVAL / KV_EUNSUPPORTED with kv_last_error set.
 */
KV_API kv_status kv_check(const kv_cache *cache, const kv_layout *pool_layout, int64_t pool_slots,
                   int64_t n_tokens, const int64_t *chunk_ids, int for_store);

/*
 * kv_store -- store (Sec. 2.2: the K/V pages preceding a prefix boundary, as
 * opaque bytes) the first n_tokens tokens of `cache`, addressed through
 * block_table, into pool slots chunk_ids[0 .. nc) in the chunk layout above.
 *   block_table: DEVICE int32[ceil(n_tokens / BS)], owned by the caller, valid
 *                and unmodified until the call completes on `stream`;
 *   chunk_ids:   HOST int64[nc], read before return;
 *   stream:      hipStream_t (NULL = the null stream).
 * Enqueues only: never blocks the host on device work.  n_tokens == 0 is a
 * no-op.  Argument errors return before anything is enqueued.  An entry of
 * block_table outside [0, num_blocks) is flagged in kv_pool_async_error; its
 * cache block is not read and its chunk rows are written as zeros (never stale
 * bytes).  Calls on one pool are serialised internally.
 */
KV_API kv_status kv_store(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                   const int64_t *chunk_ids, void *stream);

/*
 * kv_load -- the exact inverse of kv_store into `cache` (Sec. 5.1: the receiving
 * replica restores the shared prefix instead of recomputing it).  Writes only
 * the token slots named by (block_table, n_tokens); every other cache byte is
 * untouched, including slots s >= n % BS of a partial last block.
 * Destination blocks must be distinct (precondition; otherwise the result
 * depends on write order).  Duplicate chunk ids are allowed (they are reads).
 * Ownership, ordering and errors as kv_store.
 */
KV_API kv_status kv_load(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                  const int64_t *chunk_ids, void *stream);

/*
 * kv_load_noalloc -- kv_load for callers that cannot allocate: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  Same arguments, result, ordering
 * contract and argument errors as kv_load, for a host pool in either mode.  It allocates
 * nothing: no hipMalloc/hipFree, no stream, no event, no host heap memory.  Each batch of
 * chunks is copied from the pool into the library's static device scratch of
 * KV_NOALLOC_SCRATCH_BYTES with hipMemcpyAsync and unpacked from there, every copy and kernel
 * on `stream` in order.  The first call on a device looks up that device's scratch address.
 * Limits: KV_EUNSUPPORTED if one chunk (C*TB bytes) exceeds the scratch; KV_EINVAL for a
 * KV_POOL_DEVICE pool.  Every call on one GPU uses that GPU's one scratch array: calls that
 * overlap on one GPU (on two streams at once) race, and the caller must order them.
 * kv_pool_destroy does not wait for these calls: synchronise `stream` first.
 */
#define KV_NOALLOC_SCRATCH_BYTES ((int64_t)64 << 20)
KV_API kv_status kv_load_noalloc(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                                 kv_pool *pool, const int64_t *chunk_ids, void *stream);

/*
 * Host-only validation of a state-snapshot request, no HIP call.  Checks:
 * G >= 1; page_bytes >= 1; page_stride 0 or >= page_bytes; num_pages >= 1;
 * G*page_bytes == pool_state_slot_bytes (the pool's snapshot format); n >= 0;
 * for n > 0 non-NULL layer pointers, pages and slot_ids, page ids in
 * [0, num_pages), slot ids in [0, pool_state_slots); a store's slot ids and a
 * load's page ids pairwise distinct (the written side named twice would make
 * the result order dependent).  GPU-path limits give KV_EUNSUPPORTED: G > 64,
 * page_bytes, page_stride or a layer pointer not a multiple of 16.
 */
KV_API kv_status kv_check_state(const kv_state *state, int64_t pool_state_slot_bytes, int64_t pool_state_slots,
                                int64_t n, const int64_t *pages, const int64_t *slot_ids, int for_store);

/*
 * kv_store_state -- store n recurrent-state snapshots (Sec. 2.2: the boundary
 * snapshots of the recurrent layers, as opaque pages) into the pool's state
 * area: page pages[k] of every layer into state slot slot_ids[k], in the
 * state-slot format above.  The pool's mode applies (zero-copy kernels on
 * `stream`, or packing into device staging plus DMA copies on the side streams,
 * with the same ordering contract (i)-(iv) as kv_store).
 *   pages, slot_ids: HOST int64[n], read before return.
 * Enqueues only; n == 0 is a no-op; argument errors (kv_check_state) return
 * before anything is enqueued; KV_EINVAL if the pool has no state area.
 */
KV_API kv_status kv_store_state(const kv_state *state, const int64_t *pages, int64_t n, kv_pool *pool,
                                const int64_t *slot_ids, void *stream);

/* kv_load_state -- the exact inverse: state slot slot_ids[k] into page pages[k] of every
 * layer.  Writes only those pages' first page_bytes bytes.  As kv_store_state otherwise. */
KV_API kv_status kv_load_state(const kv_state *state, const int64_t *pages, int64_t n, kv_pool *pool,
                               const int64_t *slot_ids, void *stream);

/* ---------------------------------------------------------------------------
 * Pool index (host only; no HIP call).  Manages the pool's slots above the
 * transfer path, as the shared tier of the paper does (Table 1: a fixed RAM
 * budget of chunks with LRU eviction):
 *  - a whole chunk i of a prompt is keyed by a 128-bit hash chained over the
 *    cache salt and tokens [0, (i+1)*C): a key names the whole prefix it
 *    completes, and a new salt gives new keys (Sec. 3.2: a new cache salt forced
 *    zero hits).  Only whole chunks are keyed, so hits are whole chunks (Sec.
 *    3.1-3.2: 25,088 and 127,008 hit tokens are 16 and 81 chunks of 1,568);
 *  - under aligned recovery (Sec. 2.2) a hit also needs the recurrent snapshot
 *    at its boundary: the longest run of leading chunks whose last chunk carries
 *    a committed snapshot;
 *  - stores are two-phase: kv_index_reserve returns a slot for every whole
 *    chunk and marks the ones the caller must store (pending entries are
 *    invisible to lookups and never evicted); after the host has seen the
 *    stores complete on their stream (Sec. 3.2's host-side completion), the
 *    caller commits -- or aborts -- them.  Only the caller that created a
 *    pending entry publishes or aborts it; an aborted entry loses its key at
 *    once and frees its slot when its last pin is released;
 *  - a new entry takes the lowest-numbered free slot; with none free, the least
 *    recently used committed, unpinned entry is evicted (with its snapshot).  An
 *    operation on a prefix touches its chunks from last to first, so eviction
 *    trims prefixes from the end.  Snapshots have their own slot budget and LRU;
 *    evicting one keeps its chunk; a snapshot is evictable only while its chunk
 *    entry is committed and unpinned.
 * Pins (reserve, or lookup with KV_LOOKUP_PIN) keep entries from eviction while
 * their slots are read or written; release them with kv_index_commit or
 * kv_index_unpin.  All calls on one index are serialised internally.  Slot
 * numbers are the pool's chunk slots [0, num_slots) and state slots
 * [0, num_state_slots).
 * --------------------------------------------------------------------------- */
typedef struct kv_index kv_index;

#define KV_LOOKUP_REQUIRE_STATE 1u  /* aligned recovery: a hit needs the snapshot at its boundary */
#define KV_LOOKUP_PIN 2u            /* pin the hit entries (release with kv_index_unpin) */

typedef struct kv_lookup {
    int64_t kv_chunks;   /* leading whole chunks whose K/V pages are committed */
    int64_t hit_chunks;  /* restorable chunks (kv_chunks unless KV_LOOKUP_REQUIRE_STATE) */
    int64_t hit_tokens;  /* hit_chunks * C */
    int64_t state_slot;  /* state slot of the snapshot after the last hit chunk, or -1 */
} kv_lookup;

typedef struct kv_index_stats {
    int64_t entries;          /* committed chunk entries */
    int64_t pending;          /* reserved, not yet committed or aborted */
    int64_t free_slots;
    int64_t state_entries;    /* committed snapshots */
    int64_t free_state_slots;
    int64_t evictions;        /* chunk entries evicted */
    int64_t state_evictions;  /* snapshots evicted */
} kv_index_stats;

/* An index over num_slots chunk slots of chunk_tokens tokens and num_state_slots
 * (>= 0) snapshot slots.  KV_EINVAL on chunk_tokens < 1 or num_slots < 1. */
KV_API kv_status kv_index_create(int32_t chunk_tokens, int64_t num_slots, int64_t num_state_slots,
                                 kv_index **out);
KV_API kv_status kv_index_destroy(kv_index *index);  /* NULL is a no-op */

/* The keys of the floor(n_tokens / C) whole chunks of a prompt: keys[2*i], keys[2*i+1]
 * for chunk i.  tokens: HOST int32[n_tokens]. */
KV_API kv_status kv_index_keys(const kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                               uint64_t *keys);

/* Longest hit of a prompt (see above): slots[0 .. hit_chunks) receive the chunk slots
 * (slots: HOST int64, room for floor(n_tokens / C)); *out the counts.  Hit entries (and
 * the snapshot) become the most recently used.  flags: KV_LOOKUP_*. */
KV_API kv_status kv_index_lookup(kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                                 uint32_t flags, int64_t *slots, kv_lookup *out);

/* Release one pin of each listed slot (KV_EINVAL, nothing released, if one is not pinned). */
KV_API kv_status kv_index_unpin(kv_index *index, const int64_t *slots, int64_t n);

/* Reserve the whole chunks of a prompt: slots[i] and is_new[i] for every chunk
 * i < *n_chunks = floor(n_tokens / C) (HOST arrays with that much room).  is_new[i] = 1:
 * a new pending entry the caller stores; 0: an existing (committed or pending) entry.
 * Every returned entry is pinned.  KV_EBUSY if a slot cannot be freed: the call then
 * holds nothing (entries it evicted stay evicted). */
KV_API kv_status kv_index_reserve(kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                                  int64_t *slots, uint8_t *is_new, int64_t *n_chunks);

/* Finish a reservation: with ok != 0 the entries this caller created (is_new[i] = 1)
 * become visible, otherwise they are aborted; every listed pin is released.  Pass
 * exactly what kv_index_reserve returned.  KV_EINVAL (nothing changed) on a mismatch. */
KV_API kv_status kv_index_commit(kv_index *index, const int64_t *slots, const uint8_t *is_new, int64_t n,
                                 int ok);

/* Reserve the snapshot slot for the boundary after the chunk in `slot` (an entry the
 * caller holds pinned).  *is_new = 1: a new pending snapshot the caller stores (then
 * kv_index_commit_state); 0: one exists already.  KV_EBUSY if no snapshot slot can be
 * freed. */
KV_API kv_status kv_index_reserve_state(kv_index *index, int64_t slot, int64_t *state_slot, int32_t *is_new);
KV_API kv_status kv_index_commit_state(kv_index *index, int64_t slot, int ok);

KV_API kv_status kv_index_get_stats(kv_index *index, kv_index_stats *out);

/* ---------------------------------------------------------------------------
 * Tier: one process owns the pool; replicas in other processes store into it
 * and load from it (the paper's two replicas sharing one host tier, Sec. 2 and
 * Fig. 1).  A tier process calls kv_tier_serve on a connected stream socket per
 * replica.  A replica calls kv_tier_store / kv_tier_load on its end.  They pass
 * its cache as HIP IPC handles: each layer pointer names an allocation that
 * the tier opens once per connection and closes when the connection ends.  The
 * handshake is the host-side completion handling of Sec. 3.2 in both
 * directions:
 *  - the replica synchronises `stream` before sending, so every producer write
 *    to its cache (store) and every earlier use of the destination (load) has
 *    completed;
 *  - the tier enqueues kv_store / kv_load on its own stream, synchronises it
 *    and only then replies, so a stored chunk is committed (visible to any
 *    later request of any replica) and a loaded cache is complete when the
 *    call returns.
 * Requests from all connections to one pool are served one at a time, on one
 * stream the pool keeps for this (made by kv_tier_run before it accepts a
 * connection, or by the first request; released by kv_pool_destroy).
 * Device-side faults of a request (KV_ASYNC_*) are returned to its sender as
 * KV_EASYNC.
 * --------------------------------------------------------------------------- */

/* Largest allocation shared through IPC (exclusive): opening larger ones has not
 * returned on the machines this library was measured on. */
#define KV_IPC_MAX_ALLOCATION_BYTES ((int64_t)2 << 30)

typedef struct kv_ipc_buffer {
    uint8_t handle[64];  /* hipIpcMemHandle_t of the allocation that holds the buffer */
    int64_t offset;      /* byte offset of the buffer inside that allocation */
    int64_t allocation_bytes;
} kv_ipc_buffer;

/* Export a device pointer of this process.  KV_EUNSUPPORTED if its allocation is
 * KV_IPC_MAX_ALLOCATION_BYTES or larger, KV_EHIP if the runtime refuses. */
KV_API kv_status kv_ipc_export(const void *dev_ptr, kv_ipc_buffer *out);

/* Host-only check of an IPC buffer as a tier receives it, no HIP call: the declared
 * allocation is positive and below KV_IPC_MAX_ALLOCATION_BYTES, and [offset, offset + need)
 * lies inside it.  The tier applies it to every buffer of a request before opening the
 * allocation (hipIpcOpenMemHandle), so a frame that names a larger allocation ends as
 * KV_EUNSUPPORTED instead of an open that may not return; after opening, the size of the
 * mapping itself bounds every access again.  KV_EINVAL for NULL or a range outside the
 * declared allocation. */
KV_API kv_status kv_ipc_check(const kv_ipc_buffer *buf, int64_t need);

/* Serve one replica connection: read requests from the connected stream socket
 * `fd` until the peer closes it, run each on `pool` (current device = the
 * pool's), reply.  `index` (may be NULL) manages the pool's slots for the
 * prefix requests below; it must cover at most the pool's slots and use the
 * pool's chunk length.  Blocks.  Returns KV_OK on an orderly close, an error
 * if the connection failed or sent a malformed frame (the socket is left open
 * for the caller to close). */
KV_API kv_status kv_tier_serve(kv_pool *pool, kv_index *index, int fd);

/* A listening stream socket at filesystem path `path` (which must not exist yet):
 * *listen_fd receives it.  KV_EINVAL on failure (reason in kv_last_error). */
KV_API kv_status kv_tier_listen(const char *path, int *listen_fd);

/* Accept `connections` replica connections on listen_fd (0 = until the listening
 * socket fails), serve each on its own thread as kv_tier_serve does, close them,
 * and return when all have ended: KV_OK, or the first connection's error. */
KV_API kv_status kv_tier_run(kv_pool *pool, kv_index *index, int listen_fd, int32_t connections);

/* Replica side.  cache: this process's cache (layer pointers are exported);
 * block_table: HOST int32[ceil(n_tokens / BS)], read before return; chunk_ids:
 * HOST int64[nc]; stream: synchronised before the request is sent.  Blocks
 * until the tier replied; returns the tier's status (its message in
 * kv_last_error) or a transport error (KV_EHIP for HIP, KV_EINVAL for a
 * closed or failed connection). */
KV_API kv_status kv_tier_store(int fd, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                               const int64_t *chunk_ids, void *stream);
KV_API kv_status kv_tier_load(int fd, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                              const int64_t *chunk_ids, void *stream);

/* Prefix requests (a tier served with an index): the replica names its prompt
 * (tokens: HOST int32[n_tokens], cache salt) and the tier picks the slots.
 *   kv_tier_store_prefix: reserve the prompt's whole chunks, store those not yet
 *     in the pool (runs of consecutive new chunks, one kv_store each; the
 *     partial last chunk is not kept), commit them after the stores completed,
 *     or abort them all if a store failed.  With `state` (hybrid models, Sec.
 *     2.2), page `state_page` of the replica's recurrent layers is the snapshot
 *     at the boundary after the prompt's last whole chunk; it is stored into a
 *     snapshot slot of the index unless that chunk already has one.
 *     *stored_chunks = chunks written, *stored_state = 1 if a snapshot was
 *     written (either may be NULL).
 *   kv_tier_load_prefix: the longest whole-chunk hit (Sec. 3.1-3.2: hits are
 *     whole chunks), pinned while it is loaded into the cache's first
 *     hit_tokens token slots.  With `state` the hit follows aligned recovery
 *     (Sec. 2.2): only a prefix whose boundary snapshot is present counts, and
 *     that snapshot is loaded into page `state_page`.  *hit_tokens = hit chunks
 *     * C (0: nothing loaded).
 * block_table: HOST int32[ceil(n_tokens / BS)] for the whole prompt; state: as
 * for kv_store_state (its buffers exported like the cache's), or NULL.  The
 * tier's pool needs a state area of G*page_bytes slots for state requests, and
 * its index as many snapshot slots at most.  KV_EBUSY if the index cannot free
 * enough slots (then nothing was stored). */
KV_API kv_status kv_tier_store_prefix(int fd, const kv_cache *cache, const int32_t *block_table,
                                      const kv_state *state, int64_t state_page, uint64_t salt,
                                      const int32_t *tokens, int64_t n_tokens, int64_t *stored_chunks,
                                      int32_t *stored_state, void *stream);
KV_API kv_status kv_tier_load_prefix(int fd, const kv_cache *cache, const int32_t *block_table,
                                     const kv_state *state, int64_t state_page, uint64_t salt,
                                     const int32_t *tokens, int64_t n_tokens, int64_t *hit_tokens, void *stream);

/* Thread-local text of the last failure on this thread: the HIP error name and message and the
 * library call site, or the violated rule.  The paper's service log kept only a generic
 * allocation failure and lost the underlying exception (Sec. 3.3); every failing entry point
 * here records its cause.  The string is owned by the library and valid until the next failing
 * call on the same thread; "" if none failed yet. */
KV_API const char *kv_last_error(void);

/* Name of a status code ("KV_OK", "KV_EINVAL", ...). */
KV_API const char *kv_status_name(kv_status status);

/* Library version string. */
KV_API const char *kv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVX_H */

// Internal declarations shared by the kvx host code and kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <exception>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kvx.h"

namespace kvx {

#ifndef KVX_THREADS
#define KVX_THREADS 256
#endif
constexpr int kThreads = KVX_THREADS;  // work-items per workgroup (wave64s x 64)
constexpr int kMaxLaunchLayers = 64;   // layer pointers carried in one launch's kernel arguments
constexpr int kMaxLaunchChunks = 256;  // slot ids carried in one launch's kernel arguments
constexpr int kMaxStateLayers = 64;    // recurrent layers of a state snapshot (one launch carries all)
constexpr int kMaxLaunchSnapshots = 128;  // snapshots carried in one state launch's arguments
// Bytes of a page one workgroup moves (at most).  Paired on MI355X (48 x 3.06 MiB pages, device-side
// launches, two orders): 16 KiB pieces moved 3.4-4.0% more on unpack than 64 KiB and the same as 32 KiB,
// and pack followed (+5.5% over 64 KiB).
constexpr int64_t kStatePiece = 16 * 1024;
constexpr int64_t kMaxLaunchPieces = int64_t(1) << 22;  // workgroups of one state launch

// Derived sizes of a layout (all bytes, 64-bit).
struct Geometry {
    int64_t L, H, D, E, BS, C;
    int64_t row_bytes;     // D*E: one (head, token) row
    int64_t vec_per_row;   // row_bytes / 16
    int64_t block_bytes;   // 2*H*BS*D*E
    int64_t block_stride;  // bytes between blocks in a layer buffer
    int64_t token_bytes;   // TB = 2*L*H*D*E
    int64_t slot_bytes;    // C*TB
    int64_t blocks_per_chunk;  // C / BS
};

Geometry geometry(const kv_layout &lay, int64_t block_stride_bytes);

// Kernel arguments of one gather (pack) or scatter (unpack) launch.  A launch covers
// chunks [chunk0, chunk0 + nchunks) of the prefix and layers [layer0, layer0 + nlayers).
// Passed by value so that every pointer and id is captured at enqueue time.
struct GatherArgs {
    uint8_t *layer[kMaxLaunchLayers];  // cache layer base pointers (device) of layers layer0..
    uint8_t *chunk_base;               // device-visible address of slot 0 (pool or staging)
    const int32_t *block_table;        // device int32[ceil(n/BS)]
    int32_t *err;                      // device-visible async error word
    int64_t slot_stride;               // bytes between slot ids at chunk_base
    int64_t block_stride;
    int64_t n_tokens;                  // prefix length (for r_i of every chunk)
    int64_t chunk0;                    // global index of the launch's first chunk
    int32_t num_blocks;
    int32_t layer0, nlayers;
    int32_t H, BS, C;
    int32_t vec_per_row;
    int32_t blocks_per_chunk;
    int32_t nchunks;
    int32_t nhd;                       // cache blocks are [2][BS][H][D] (token-major)
    int32_t slot[kMaxLaunchChunks];    // slot id of each chunk of the launch
};

enum Direction { kPack = 0, kUnpack = 1 };

// Kernel arguments of one state-snapshot launch.  Pages are cut into pieces of `piece`
// bytes (the last piece of a page may be shorter); piece q of the launch is piece
// j = q % ppp of layer g = (q / ppp) % G of snapshot k = q / (G*ppp).  The launch covers
// pieces [q0, q0 + gridDim.x) of snapshots 0..nsnap-1 of its own lists.
struct StateArgs {
    uint8_t *layer[kMaxStateLayers];   // device base of each recurrent layer's page buffer
    uint8_t *base;                     // device-visible packed side (state pool or staging)
    int64_t page_stride, page_bytes, piece;
    int64_t q0;
    int64_t npieces;  // pieces in this launch (set by launch_state)
    int32_t G, ppp, nsnap, pad;
    int64_t page[kMaxLaunchSnapshots];  // device page id of each snapshot
    int64_t off[kMaxLaunchSnapshots];   // byte offset at `base` of each snapshot's packed bytes
};

hipError_t launch_state(const StateArgs &args, int64_t pieces, Direction dir, bool host_side,
                        hipStream_t stream);

// Enqueue one launch on `stream`; host_side: the chunk side is mapped pinned host memory.
// Returns the launch error (hipSuccess on success).
hipError_t launch_gather(const GatherArgs &args, Direction dir, bool host_side, hipStream_t stream);

// Largest chunk count per launch that keeps the grid within the 32-bit work-item limit.
int max_chunks_per_launch(const Geometry &g, int nlayers);

// Enqueue the pack/unpack launches for chunks [chunk0, chunk0 + nchunks) of a prefix of `cache`
// (layers split over launches of at most kMaxLaunchLayers): slots[c] is the slot of chunk
// chunk0 + c at chunk_base, slot_stride bytes apart.  No host allocation, no event.
hipError_t launch_gathers(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, Direction dir,
                          int64_t chunk0, int nchunks, const int32_t *slots, uint8_t *chunk_base, int64_t slot_stride,
                          bool host_side, int32_t *err, hipStream_t stream);

// Thread-local error reporting.
kv_status fail(kv_status code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
kv_status hip_fail(hipError_t err, const char *what, const char *file, int line);
void set_last_error(const std::string &msg);

// Runs an entry point's body so that no C++ exception crosses the C ABI: a failed host
// allocation becomes KV_ENOMEM, any other exception KV_EINVAL with its message.
template <class F>
kv_status guarded(F &&body) noexcept {
    try {
        return body();
    } catch (const std::bad_alloc &) {
        return fail(KV_ENOMEM, "host memory allocation failed");
    } catch (const std::exception &e) {
        return fail(KV_EINVAL, "internal error: %s", e.what());
    } catch (...) {
        return fail(KV_EINVAL, "internal error");
    }
}

#define KVX_HIP(expr)                                                         \
    do {                                                                      \
        hipError_t kvx_e_ = (expr);                                           \
        if (kvx_e_ != hipSuccess)                                             \
            return ::kvx::hip_fail(kvx_e_, #expr, __FILE__, __LINE__);        \
    } while (0)

// Host-only request validation shared by kv_check, kv_store and kv_load.
kv_status check_layout(const kv_layout &lay);
kv_status check_request(const kv_cache *cache, const kv_layout *pool_layout, int64_t pool_slots,
                        int64_t n_tokens, const int64_t *chunk_ids, int for_store);
kv_status check_state_request(const kv_state *state, int64_t pool_state_slot_bytes, int64_t pool_state_slots,
                              int64_t n, const int64_t *pages, const int64_t *slot_ids, int for_store);

// Geometry of a pool index (for the tier's consistency check).
int32_t index_chunk_tokens(const kv_index *index);
int64_t index_num_slots(const kv_index *index);
int64_t index_num_state_slots(const kv_index *index);

}  // namespace kvx

// The pool: one pinned host region plus the staging ring and its streams/events.
struct kv_pool {
    kv_layout layout{};
    kvx::Geometry geo{};
    int64_t num_slots = 0, pool_bytes = 0;
    // Recurrent-state snapshot area: num_state_slots slots of state_slot_bytes each, starting
    // state_offset bytes into the pinned region (after the chunk slots).
    int64_t num_state_slots = 0, state_slot_bytes = 0, state_offset = 0;
    int device = 0;
    uint32_t mode_of[2] = {0, 0};     // transfer mode per direction: [kPack] stores, [kUnpack] loads
    uint32_t host_kind = 0;
    uint8_t *host_base = nullptr;   // host address of slot 0 (nullptr for a device pool)
    uint8_t *dev_base = nullptr;    // device address of slot 0
    bool on_device = false;         // KV_POOL_DEVICE: the region is device memory (HBM)
    int32_t *err_host = nullptr;    // async error word (pinned, mapped)
    int32_t *err_dev = nullptr;
    double alloc_seconds = 0.0;
    bool pinned = false;

    // Staged mode: one lane per direction, each with its own staging ring, DMA side streams and
    // events, so a store and a load in flight at once never wait for each other's slots or streams.
    struct Lane {
        uint8_t *staging = nullptr;        // K slots of cpb*slot_bytes each
        std::vector<hipStream_t> sides;    // DMA side streams of this direction
        std::vector<hipEvent_t> ev_free;   // staging slot k may be overwritten once this completes
        std::vector<bool> free_recorded;
        std::vector<hipEvent_t> ev_ready;  // staging slot k holds the current batch
        std::vector<hipEvent_t> ev_join;   // per side stream: exit join of a store
        hipEvent_t ev_entry = nullptr;     // entry gate of a load
        int ring = 0;
    };
    int K = 0, cpb = 0, S = 0;       // ring depth, chunks per slot, side streams: per direction
    uint8_t *staging = nullptr;      // both lanes' staging (one allocation)
    bool staging_contiguous = false;  // always false: staging is plain device memory
    Lane lane[2];                    // [kPack] stores, [kUnpack] loads
    int zc_chunks = 0;                 // chunks per zero-copy launch
    // Last use of the pool on each caller stream (recorded after every store/load), so that
    // kv_pool_destroy never frees memory that queued kernels or copies still touch.
    std::vector<std::pair<hipStream_t, hipEvent_t>> last_use;

    // Profiling of pack/unpack and state launches.
    bool profile = false;
    struct Timed {
        hipEvent_t start, stop;
        double bytes;
    };
    // Index: 0 pack, 1 unpack, 2 state pack, 3 state unpack.
    std::vector<Timed> pending[4];
    std::vector<hipEvent_t> spare_events;
    int64_t launches[4] = {0, 0, 0, 0};
    double total_ms[4] = {0.0, 0.0, 0.0, 0.0};
    double total_bytes[4] = {0.0, 0.0, 0.0, 0.0};

    std::mutex mu;
    std::mutex tier_mu;  // serialises tier requests (one request's faults are its own)
    // Tier serving: every request runs under tier_mu on this one stream, its block table staged
    // through these buffers.  Made by the first request (or by kv_tier_run before it accepts a
    // connection) and kept until kv_pool_destroy, so later connections create no runtime objects
    // (a new stream and its first copy measured tens of ms on the request's path).
    hipStream_t tier_stream = nullptr;
    int32_t *tier_table = nullptr;         // device copy of the request's block table
    int32_t *tier_table_pinned = nullptr;  // pinned host staging of it
    size_t tier_table_cap = 0;             // bytes of each
};

namespace kvx {
// Make the pool's tier stream and block-table buffers (at least `table_bytes` each) if they are
// missing or too small.  Caller holds pool->tier_mu and has made the pool's device current.
kv_status tier_resources(kv_pool *pool, size_t table_bytes);
}  // namespace kvx

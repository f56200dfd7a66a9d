// kvx pool and transfer engine: the pinned host tier, the staging ring, and the ordering
// of pack/unpack kernels and DMA copies against the caller's stream.
//
// Ordering (the dependency whose omission the paper diagnoses, Sec. 3.2 and Fig. 2):
//  * zero-copy mode: every kernel runs on the caller's stream, so it follows all earlier
//    work on that stream and all later work follows it;
//  * staged mode, store: pack kernels run on the caller's stream into staging slot k; the
//    D2H copy of slot k runs on a side stream gated by an event recorded right after the
//    pack; before exit the caller's stream waits for every side stream's last copy;
//  * staged mode, load: an entry event on the caller's stream gates every side-stream H2D
//    copy (so pool reads follow earlier stream work, e.g. a store); each unpack kernel on
//    the caller's stream waits for its copy;
//  * staging slot k is reused only after the event of its last use (copy or unpack)
//    completed -- premature reuse of an asynchronous-copy buffer is the related failure
//    the paper cites (Sec. 3.2).
// No call ever blocks the host on device work.
#include <chrono>
#include <cstring>

#include "kvx_internal.h"

using kvx::Direction;
using kvx::Geometry;

namespace {

constexpr int kDefaultStagingSlots = 3;
constexpr int kDefaultChunksPerBatch = 16;
constexpr int kDefaultSideStreams = 2;

kv_status release(kv_pool *p) {
    // Best-effort teardown: keep going after a failure, report the first one.
    kv_status first = KV_OK;
    auto note = [&](hipError_t e, const char *what) {
        if (e != hipSuccess && first == KV_OK)
            first = kvx::hip_fail(e, what, __FILE__, __LINE__);
    };
    // Work queued on caller streams (kernels writing the pool or staging) must finish first.
    for (auto &use : p->last_use)
        note(hipEventSynchronize(use.second), "hipEventSynchronize(last use)");
    for (auto &use : p->last_use)
        note(hipEventDestroy(use.second), "hipEventDestroy");
    for (hipStream_t s : p->sides)
        note(hipStreamSynchronize(s), "hipStreamSynchronize(side)");
    for (hipStream_t s : p->sides)
        note(hipStreamDestroy(s), "hipStreamDestroy");
    for (auto *vec : {&p->ev_free, &p->ev_ready, &p->ev_join})
        for (hipEvent_t e : *vec)
            note(hipEventDestroy(e), "hipEventDestroy");
    if (p->ev_entry)
        note(hipEventDestroy(p->ev_entry), "hipEventDestroy");
    for (int w = 0; w < 2; ++w)
        for (auto &t : p->pending[w]) {
            note(hipEventSynchronize(t.stop), "hipEventSynchronize");
            note(hipEventDestroy(t.start), "hipEventDestroy");
            note(hipEventDestroy(t.stop), "hipEventDestroy");
        }
    for (hipEvent_t e : p->spare_events)
        note(hipEventDestroy(e), "hipEventDestroy");
    if (p->staging)
        note(hipFree(p->staging), "hipFree(staging)");
    if (p->err_host)
        note(hipHostFree(p->err_host), "hipHostFree(err)");
    if (p->host_base)
        note(hipHostFree(p->host_base), "hipHostFree(pool)");
    delete p;
    return first;
}

kv_status make_event(hipEvent_t *e, bool timing) {
    KVX_HIP(hipEventCreateWithFlags(e, timing ? hipEventDefault : hipEventDisableTiming));
    return KV_OK;
}

kv_status take_timing_event(kv_pool *p, hipEvent_t *e) {
    if (!p->spare_events.empty()) {
        *e = p->spare_events.back();
        p->spare_events.pop_back();
        return KV_OK;
    }
    return make_event(e, true);
}

// Check the current device and the cache's device against the pool's.
kv_status check_device(const kv_pool *p, const kv_cache *cache) {
    int cur = -1;
    KVX_HIP(hipGetDevice(&cur));
    if (cur != p->device || cache->device != p->device)
        return kvx::fail(KV_EINVAL, "pool is on device %d, cache on device %d, current device %d", p->device,
                         cache->device, cur);
    return KV_OK;
}

// Enqueue the pack/unpack kernels for chunks [chunk0, chunk0 + nchunks) of the prefix.
// slots[c] is the slot id of chunk chunk0 + c relative to chunk_base (slot_stride apart);
// host_side: chunk_base is the mapped pinned pool (zero-copy) rather than device staging.
kv_status enqueue_gather(kv_pool *p, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                         Direction dir, int64_t chunk0, int nchunks, const int32_t *slots, uint8_t *chunk_base,
                         int64_t slot_stride, bool host_side, hipStream_t stream) {
    const Geometry &g0 = p->geo;
    const Geometry g = kvx::geometry(cache->layout, cache->block_stride_bytes);
    hipEvent_t t_start = nullptr, t_stop = nullptr;
    if (p->profile) {
        kv_status st = take_timing_event(p, &t_start);
        if (st != KV_OK)
            return st;
        st = take_timing_event(p, &t_stop);
        if (st != KV_OK)
            return st;
        KVX_HIP(hipEventRecord(t_start, stream));
    }
    int64_t payload = 0;
    for (int layer0 = 0; layer0 < g.L; layer0 += kvx::kMaxLaunchLayers) {
        const int nl = static_cast<int>(std::min<int64_t>(kvx::kMaxLaunchLayers, g.L - layer0));
        const int per_launch = kvx::max_chunks_per_launch(g, nl);
        for (int c0 = 0; c0 < nchunks; c0 += per_launch) {
            const int nc = std::min(per_launch, nchunks - c0);
            kvx::GatherArgs a;
            std::memset(&a, 0, sizeof(a));
            for (int l = 0; l < nl; ++l)
                a.layer[l] = static_cast<uint8_t *>(cache->layer_ptrs[layer0 + l]);
            a.chunk_base = chunk_base;
            a.block_table = block_table;
            a.err = p->err_dev;
            a.slot_stride = slot_stride;
            a.block_stride = g.block_stride;
            a.n_tokens = n_tokens;
            a.chunk0 = chunk0 + c0;
            a.num_blocks = cache->num_blocks;
            a.layer0 = layer0;
            a.nlayers = nl;
            a.H = static_cast<int32_t>(g.H);
            a.BS = static_cast<int32_t>(g.BS);
            a.C = static_cast<int32_t>(g.C);
            a.vec_per_row = static_cast<int32_t>(g.vec_per_row);
            a.blocks_per_chunk = static_cast<int32_t>(g.blocks_per_chunk);
            a.nchunks = nc;
            a.nhd = cache->block_order == KV_BLOCK_NHD ? 1 : 0;
            for (int c = 0; c < nc; ++c)
                a.slot[c] = slots[c0 + c];
            KVX_HIP(kvx::launch_gather(a, dir, host_side, stream));
        }
    }
    for (int c = 0; c < nchunks; ++c) {
        const int64_t i = chunk0 + c;
        const int64_t r = std::min<int64_t>(g0.C, n_tokens - i * g0.C);
        payload += r * g0.token_bytes;
    }
    if (p->profile) {
        KVX_HIP(hipEventRecord(t_stop, stream));
        p->pending[dir].push_back({t_start, t_stop, 2.0 * static_cast<double>(payload)});
    }
    return KV_OK;
}

// Contiguous host<->staging copy runs of one staged batch: consecutive chunks whose slots
// are consecutive and whose earlier members are full merge into one DMA copy.
struct CopyRun {
    int64_t first_chunk;  // index within the batch
    int64_t slot;         // pool slot of the first chunk
    int64_t bytes;
};

std::vector<CopyRun> copy_runs(const kv_pool *p, int64_t n_tokens, int64_t chunk0, int nchunks,
                               const int64_t *chunk_ids) {
    std::vector<CopyRun> runs;
    const Geometry &g = p->geo;
    for (int c = 0; c < nchunks; ++c) {
        const int64_t i = chunk0 + c;
        const int64_t r = std::min<int64_t>(g.C, n_tokens - i * g.C);
        const int64_t bytes = r * g.token_bytes;
        if (!runs.empty()) {
            CopyRun &last = runs.back();
            const int64_t members = c - last.first_chunk;
            const bool prev_full = last.bytes == members * g.slot_bytes;
            if (prev_full && chunk_ids[i] == last.slot + members) {
                last.bytes += bytes;
                continue;
            }
        }
        runs.push_back({c, chunk_ids[i], bytes});
    }
    return runs;
}

kv_status transfer(kv_pool *p, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                   const int64_t *chunk_ids, hipStream_t stream, Direction dir) {
    const Geometry &g = p->geo;
    const int64_t nc = (n_tokens + g.C - 1) / g.C;

    if (p->mode == KV_MODE_ZERO_COPY) {
        std::vector<int32_t> slots(static_cast<size_t>(nc));
        for (int64_t i = 0; i < nc; ++i)
            slots[static_cast<size_t>(i)] = static_cast<int32_t>(chunk_ids[i]);
        for (int64_t c0 = 0; c0 < nc; c0 += p->zc_chunks) {
            const int n = static_cast<int>(std::min<int64_t>(p->zc_chunks, nc - c0));
            kv_status st = enqueue_gather(p, cache, block_table, n_tokens, dir, c0, n, slots.data() + c0,
                                          p->dev_base, g.slot_bytes, true, stream);
            if (st != KV_OK)
                return st;
        }
        return KV_OK;
    }

    // Staged mode.
    std::vector<int32_t> local(static_cast<size_t>(p->cpb));
    for (int c = 0; c < p->cpb; ++c)
        local[static_cast<size_t>(c)] = c;
    const int64_t staging_slot_bytes = static_cast<int64_t>(p->cpb) * g.slot_bytes;
    std::vector<bool> side_used(p->sides.size(), false);

    if (dir == kvx::kUnpack)
        KVX_HIP(hipEventRecord(p->ev_entry, stream));  // entry gate for pool reads

    int64_t batch = 0;
    for (int64_t c0 = 0; c0 < nc; c0 += p->cpb, ++batch) {
        const int n = static_cast<int>(std::min<int64_t>(p->cpb, nc - c0));
        const int k = p->ring;
        p->ring = (p->ring + 1) % p->K;
        const size_t si = static_cast<size_t>(batch % static_cast<int64_t>(p->sides.size()));
        hipStream_t side = p->sides[si];
        uint8_t *stage = p->staging + static_cast<int64_t>(k) * staging_slot_bytes;
        const std::vector<CopyRun> runs = copy_runs(p, n_tokens, c0, n, chunk_ids);

        if (dir == kvx::kPack) {
            if (p->free_recorded[k])
                KVX_HIP(hipStreamWaitEvent(stream, p->ev_free[k], 0));
            kv_status st = enqueue_gather(p, cache, block_table, n_tokens, dir, c0, n, local.data(), stage,
                                          g.slot_bytes, false, stream);
            if (st != KV_OK)
                return st;
            KVX_HIP(hipEventRecord(p->ev_ready[k], stream));
            KVX_HIP(hipStreamWaitEvent(side, p->ev_ready[k], 0));
            for (const CopyRun &run : runs)
                KVX_HIP(hipMemcpyAsync(p->host_base + run.slot * g.slot_bytes, stage + run.first_chunk * g.slot_bytes,
                                       static_cast<size_t>(run.bytes), hipMemcpyDeviceToHost, side));
            KVX_HIP(hipEventRecord(p->ev_free[k], side));
            p->free_recorded[k] = true;
            side_used[si] = true;
        } else {
            if (!side_used[si]) {
                KVX_HIP(hipStreamWaitEvent(side, p->ev_entry, 0));
                side_used[si] = true;
            }
            if (p->free_recorded[k])
                KVX_HIP(hipStreamWaitEvent(side, p->ev_free[k], 0));
            for (const CopyRun &run : runs)
                KVX_HIP(hipMemcpyAsync(stage + run.first_chunk * g.slot_bytes, p->host_base + run.slot * g.slot_bytes,
                                       static_cast<size_t>(run.bytes), hipMemcpyHostToDevice, side));
            KVX_HIP(hipEventRecord(p->ev_ready[k], side));
            KVX_HIP(hipStreamWaitEvent(stream, p->ev_ready[k], 0));
            kv_status st = enqueue_gather(p, cache, block_table, n_tokens, dir, c0, n, local.data(), stage,
                                          g.slot_bytes, false, stream);
            if (st != KV_OK)
                return st;
            KVX_HIP(hipEventRecord(p->ev_free[k], stream));
            p->free_recorded[k] = true;
        }
    }
    if (dir == kvx::kPack) {
        // Exit join: later work on the caller's stream follows every D2H copy.
        for (size_t si = 0; si < p->sides.size(); ++si) {
            if (!side_used[si])
                continue;
            KVX_HIP(hipEventRecord(p->ev_join[si], p->sides[si]));
            KVX_HIP(hipStreamWaitEvent(stream, p->ev_join[si], 0));
        }
    }
    return KV_OK;
}

// Record the pool's last use on `stream` (one event per stream seen).
kv_status mark_use(kv_pool *p, hipStream_t stream) {
    for (auto &use : p->last_use)
        if (use.first == stream) {
            KVX_HIP(hipEventRecord(use.second, stream));
            return KV_OK;
        }
    hipEvent_t e = nullptr;
    kv_status st = make_event(&e, false);
    if (st != KV_OK)
        return st;
    p->last_use.emplace_back(stream, e);
    KVX_HIP(hipEventRecord(e, stream));
    return KV_OK;
}

kv_status run(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
              const int64_t *chunk_ids, void *stream, Direction dir) {
    if (!pool)
        return kvx::fail(KV_EINVAL, "pool must not be NULL");
    std::lock_guard<std::mutex> lock(pool->mu);
    kv_status st = kvx::check_request(cache, &pool->layout, pool->num_slots, n_tokens, chunk_ids,
                                      dir == kvx::kPack);
    if (st != KV_OK)
        return st;
    if (n_tokens == 0)
        return KV_OK;
    if (!block_table)
        return kvx::fail(KV_EINVAL, "block_table must not be NULL for n_tokens > 0");
    st = check_device(pool, cache);
    if (st != KV_OK)
        return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = transfer(pool, cache, block_table, n_tokens, chunk_ids, s, dir);
    // Record the last use on this stream even after a partial enqueue.
    const kv_status st_use = mark_use(pool, s);
    return st != KV_OK ? st : st_use;
}

}  // namespace

extern "C" {

kv_status kv_pool_create(const kv_layout *layout, int64_t num_slots, const kv_pool_options *opts, kv_pool **out) {
    if (!layout || !opts || !out)
        return kvx::fail(KV_EINVAL, "layout, opts and out must not be NULL");
    *out = nullptr;
    kv_status st = kvx::check_layout(*layout);
    if (st != KV_OK)
        return st;
    if (num_slots <= 0 || num_slots > INT32_MAX)
        return kvx::fail(KV_EINVAL, "num_slots must be in [1, 2^31-1] (got %lld)", static_cast<long long>(num_slots));
    if (opts->mode != KV_MODE_ZERO_COPY && opts->mode != KV_MODE_STAGED)
        return kvx::fail(KV_EINVAL, "opts->mode must be KV_MODE_ZERO_COPY or KV_MODE_STAGED (got %u)", opts->mode);
    if (opts->host_kind != KV_HOST_COHERENT && opts->host_kind != KV_HOST_NONCOHERENT)
        return kvx::fail(KV_EINVAL, "unknown host_kind %u", opts->host_kind);
    // chunks_per_batch applies to the mode chosen at creation; the other mode keeps its default.
    if (opts->chunks_per_batch < 0 || opts->chunks_per_batch > kvx::kMaxLaunchChunks)
        return kvx::fail(KV_EINVAL, "chunks_per_batch must be in [1, %d] (got %d)", kvx::kMaxLaunchChunks,
                         opts->chunks_per_batch);
    const bool staged = opts->mode == KV_MODE_STAGED;
    const int cpb = (staged && opts->chunks_per_batch) ? opts->chunks_per_batch : kDefaultChunksPerBatch;
    const int zc_chunks = (!staged && opts->chunks_per_batch) ? opts->chunks_per_batch : kvx::kMaxLaunchChunks;
    const bool want_staging = opts->mode == KV_MODE_STAGED || opts->staging_slots > 0;
    const int K = opts->staging_slots ? opts->staging_slots : kDefaultStagingSlots;
    if (want_staging && (K < 2 || K > 64))
        return kvx::fail(KV_EINVAL, "staging_slots must be in [2, 64] (got %d)", K);
    const int S = opts->side_streams ? opts->side_streams : kDefaultSideStreams;
    if (want_staging && (S < 1 || S > 8))
        return kvx::fail(KV_EINVAL, "side_streams must be in [1, 8] (got %d)", S);

    kv_pool *p = new kv_pool();
    p->layout = *layout;
    p->geo = kvx::geometry(*layout, 0);
    p->num_slots = num_slots;
    if (p->geo.slot_bytes > INT64_MAX / num_slots) {
        delete p;
        return kvx::fail(KV_EINVAL, "pool size overflows 64 bits");
    }
    p->pool_bytes = num_slots * p->geo.slot_bytes;
    p->mode = opts->mode;
    p->host_kind = opts->host_kind;
    p->profile = opts->profile != 0;
    p->zc_chunks = zc_chunks;

    // On failure: free what was made, keeping the original error text.
    auto bail = [&](kv_status code) {
        const std::string msg = kv_last_error();
        release(p);
        kvx::set_last_error(msg);
        return code;
    };

    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess)
        return bail(kvx::hip_fail(e, "hipGetDevice", __FILE__, __LINE__));

    // One pinned, mapped region of exactly pool_bytes (Sec. 3.3: no rounding allocator,
    // and never a silent fallback to pageable memory).
    const unsigned flags = hipHostMallocMapped | hipHostMallocPortable |
                           (p->host_kind == KV_HOST_COHERENT ? hipHostMallocCoherent : hipHostMallocNonCoherent);
    const auto t0 = std::chrono::steady_clock::now();
    void *host = nullptr;
    e = hipHostMalloc(&host, static_cast<size_t>(p->pool_bytes), flags);
    const auto t1 = std::chrono::steady_clock::now();
    if (e != hipSuccess || !host) {
        (void)hipGetLastError();
        const long long want = static_cast<long long>(p->pool_bytes);
        release(p);
        return kvx::fail(KV_ENOMEM, "pinned allocation of %lld bytes failed (%s); no pageable fallback", want,
                         hipGetErrorName(e));
    }
    p->host_base = static_cast<uint8_t *>(host);
    p->alloc_seconds = std::chrono::duration<double>(t1 - t0).count();

    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof(attr));
    e = hipPointerGetAttributes(&attr, host);
    if (e != hipSuccess)
        return bail(kvx::hip_fail(e, "hipPointerGetAttributes(pool)", __FILE__, __LINE__));
    p->pinned = attr.type == hipMemoryTypeHost;
    if (!p->pinned)
        return bail(kvx::fail(KV_ENOMEM, "pool memory is not reported as pinned host memory"));
    void *dptr = nullptr;
    e = hipHostGetDevicePointer(&dptr, host, 0);
    if (e != hipSuccess)
        return bail(kvx::hip_fail(e, "hipHostGetDevicePointer(pool)", __FILE__, __LINE__));
    p->dev_base = static_cast<uint8_t *>(dptr);

    e = hipHostMalloc(reinterpret_cast<void **>(&p->err_host), 256, hipHostMallocMapped | hipHostMallocCoherent);
    if (e != hipSuccess)
        return bail(kvx::hip_fail(e, "hipHostMalloc(err)", __FILE__, __LINE__));
    std::memset(p->err_host, 0, 256);
    e = hipHostGetDevicePointer(reinterpret_cast<void **>(&p->err_dev), p->err_host, 0);
    if (e != hipSuccess)
        return bail(kvx::hip_fail(e, "hipHostGetDevicePointer(err)", __FILE__, __LINE__));

    if (want_staging) {
        p->K = K;
        p->cpb = cpb;
        p->S = S;
        const size_t staging_bytes = static_cast<size_t>(K) * cpb * static_cast<size_t>(p->geo.slot_bytes);
        // Physically contiguous staging: the DMA engines read and write it, and staging placed in
        // fragmented (recycled) device memory was measured to slow D2H copies by ~5%.  If the
        // runtime refuses the flag, plain device memory is used and kv_pool_info reports it.
        e = hipExtMallocWithFlags(reinterpret_cast<void **>(&p->staging), staging_bytes, hipDeviceMallocContiguous);
        p->staging_contiguous = e == hipSuccess;
        if (e != hipSuccess) {
            (void)hipGetLastError();
            e = hipMalloc(reinterpret_cast<void **>(&p->staging), staging_bytes);
        }
        if (e != hipSuccess)
            return bail(kvx::hip_fail(e, "hipMalloc(staging)", __FILE__, __LINE__));
        for (int s = 0; s < S; ++s) {
            hipStream_t side = nullptr;
            // Default priority on purpose: every stream of the library shares one priority.
            e = hipStreamCreateWithFlags(&side, hipStreamNonBlocking);
            if (e != hipSuccess)
                return bail(kvx::hip_fail(e, "hipStreamCreateWithFlags", __FILE__, __LINE__));
            p->sides.push_back(side);
            hipEvent_t j = nullptr;
            if ((st = make_event(&j, false)) != KV_OK)
                return bail(st);
            p->ev_join.push_back(j);
        }
        for (int k = 0; k < K; ++k) {
            hipEvent_t a = nullptr, b = nullptr;
            if ((st = make_event(&a, false)) != KV_OK)
                return bail(st);
            p->ev_free.push_back(a);
            if ((st = make_event(&b, false)) != KV_OK)
                return bail(st);
            p->ev_ready.push_back(b);
        }
        p->free_recorded.assign(static_cast<size_t>(K), false);
        if ((st = make_event(&p->ev_entry, false)) != KV_OK)
            return bail(st);
    }
    *out = p;
    return KV_OK;
}

kv_status kv_pool_destroy(kv_pool *pool) {
    if (!pool)
        return KV_OK;
    return release(pool);
}

kv_status kv_pool_get_info(const kv_pool *pool, kv_pool_info *info) {
    if (!pool || !info)
        return kvx::fail(KV_EINVAL, "pool and info must not be NULL");
    std::memset(info, 0, sizeof(*info));
    info->num_slots = pool->num_slots;
    info->slot_bytes = pool->geo.slot_bytes;
    info->pool_bytes = pool->pool_bytes;
    info->staging_bytes = pool->staging ? static_cast<int64_t>(pool->K) * pool->cpb * pool->geo.slot_bytes : 0;
    info->alloc_seconds = pool->alloc_seconds;
    info->device = pool->device;
    info->mode = pool->mode;
    info->host_kind = pool->host_kind;
    info->is_pinned = pool->pinned ? 1 : 0;
    info->staging_slots = pool->K;
    info->chunks_per_batch = pool->staging ? pool->cpb : pool->zc_chunks;
    info->side_streams = pool->S;
    info->staging_contiguous = pool->staging_contiguous ? 1 : 0;
    info->host_base = pool->host_base;
    info->device_base = pool->dev_base;
    return KV_OK;
}

void *kv_pool_slot(kv_pool *pool, int64_t slot) {
    if (!pool || slot < 0 || slot >= pool->num_slots)
        return nullptr;
    return pool->host_base + slot * pool->geo.slot_bytes;
}

int64_t kv_pool_slot_bytes(const kv_pool *pool) { return pool ? pool->geo.slot_bytes : -1; }

int64_t kv_pool_num_slots(const kv_pool *pool) { return pool ? pool->num_slots : -1; }

kv_status kv_pool_set_mode(kv_pool *pool, uint32_t mode) {
    if (!pool)
        return kvx::fail(KV_EINVAL, "pool must not be NULL");
    std::lock_guard<std::mutex> lock(pool->mu);
    if (mode != KV_MODE_ZERO_COPY && mode != KV_MODE_STAGED)
        return kvx::fail(KV_EINVAL, "unknown mode %u", mode);
    if (mode == KV_MODE_STAGED && !pool->staging)
        return kvx::fail(KV_EINVAL, "pool was created without staging; staged mode unavailable");
    pool->mode = mode;
    return KV_OK;
}

int32_t kv_pool_async_error(kv_pool *pool, int clear) {
    if (!pool)
        return kvx::fail(KV_EINVAL, "pool must not be NULL");
    volatile int32_t *w = pool->err_host;
    const int32_t v = *w;
    if (clear)
        *w = 0;
    return v;
}

kv_status kv_pool_kernel_stats(kv_pool *pool, int which, int reset, int64_t *launches, double *total_ms,
                               double *bytes) {
    if (!pool || which < 0 || which > 1)
        return kvx::fail(KV_EINVAL, "pool must not be NULL and which must be 0 (pack) or 1 (unpack)");
    std::lock_guard<std::mutex> lock(pool->mu);
    auto &pend = pool->pending[which];
    size_t done = 0;
    for (; done < pend.size(); ++done) {
        float ms = 0.0f;
        hipError_t e = hipEventElapsedTime(&ms, pend[done].start, pend[done].stop);
        if (e == hipErrorNotReady)
            break;
        if (e != hipSuccess)
            return kvx::hip_fail(e, "hipEventElapsedTime", __FILE__, __LINE__);
        pool->launches[which] += 1;
        pool->total_ms[which] += ms;
        pool->total_bytes[which] += pend[done].bytes;
        pool->spare_events.push_back(pend[done].start);
        pool->spare_events.push_back(pend[done].stop);
    }
    pend.erase(pend.begin(), pend.begin() + static_cast<std::ptrdiff_t>(done));
    if (launches)
        *launches = pool->launches[which];
    if (total_ms)
        *total_ms = pool->total_ms[which];
    if (bytes)
        *bytes = pool->total_bytes[which];
    if (reset) {
        pool->launches[which] = 0;
        pool->total_ms[which] = 0.0;
        pool->total_bytes[which] = 0.0;
    }
    if (!pend.empty())
        return kvx::fail(KV_EINVAL, "%zu timed launches have not completed; synchronise first", pend.size());
    return KV_OK;
}

kv_status kv_store(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                   const int64_t *chunk_ids, void *stream) {
    return run(cache, block_table, n_tokens, pool, chunk_ids, stream, kvx::kPack);
}

kv_status kv_load(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                  const int64_t *chunk_ids, void *stream) {
    return run(cache, block_table, n_tokens, pool, chunk_ids, stream, kvx::kUnpack);
}

}  // extern "C"

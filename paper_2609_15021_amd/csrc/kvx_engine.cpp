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
//    the paper cites (Sec. 3.2);
//  * stores and loads each have their own lane (staging ring, side streams, events), so a
//    store and a load in flight at once use the host link in both directions.
// No call ever blocks the host on device work.
#include <algorithm>
#include <chrono>
#include <cstring>
#include <functional>

#include "kvx_internal.h"

using kvx::Direction;
using kvx::Geometry;

namespace kvx {

hipError_t launch_gathers(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, Direction dir,
                          int64_t chunk0, int nchunks, const int32_t *slots, uint8_t *chunk_base, int64_t slot_stride,
                          bool host_side, int32_t *err, hipStream_t stream) {
    const Geometry g = geometry(cache->layout, cache->block_stride_bytes);
    for (int layer0 = 0; layer0 < g.L; layer0 += kMaxLaunchLayers) {
        const int nl = static_cast<int>(std::min<int64_t>(kMaxLaunchLayers, g.L - layer0));
        const int per_launch = max_chunks_per_launch(g, nl);
        for (int c0 = 0; c0 < nchunks; c0 += per_launch) {
            const int nc = std::min(per_launch, nchunks - c0);
            GatherArgs a;
            std::memset(&a, 0, sizeof(a));
            for (int l = 0; l < nl; ++l)
                a.layer[l] = static_cast<uint8_t *>(cache->layer_ptrs[layer0 + l]);
            a.chunk_base = chunk_base;
            a.block_table = block_table;
            a.err = err;
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
            const hipError_t e = launch_gather(a, dir, host_side, stream);
            if (e != hipSuccess)
                return e;
        }
    }
    return hipSuccess;
}

}  // namespace kvx

namespace {

constexpr int kDefaultStagingSlots = 3;
constexpr int kDefaultChunksPerBatch = 16;
// One DMA side stream per direction: a store and a load in flight at once then move ~99 GB/s in total
// (two per direction measured 57-64 GB/s: the runtime spreads their copies over more copy engines).
constexpr int kDefaultSideStreams = 1;

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
    if (p->tier_stream) {
        note(hipStreamSynchronize(p->tier_stream), "hipStreamSynchronize(tier)");
        note(hipStreamDestroy(p->tier_stream), "hipStreamDestroy(tier)");
    }
    if (p->tier_table)
        note(hipFree(p->tier_table), "hipFree(tier table)");
    if (p->tier_table_pinned)
        note(hipHostFree(p->tier_table_pinned), "hipHostFree(tier table)");
    for (auto &lane : p->lane) {
        for (hipStream_t s : lane.sides)
            note(hipStreamSynchronize(s), "hipStreamSynchronize(side)");
        for (hipStream_t s : lane.sides)
            note(hipStreamDestroy(s), "hipStreamDestroy");
        for (auto *vec : {&lane.ev_free, &lane.ev_ready, &lane.ev_join})
            for (hipEvent_t e : *vec)
                note(hipEventDestroy(e), "hipEventDestroy");
        if (lane.ev_entry)
            note(hipEventDestroy(lane.ev_entry), "hipEventDestroy");
    }
    for (int w = 0; w < 4; ++w)
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
    if (p->on_device && p->dev_base)
        note(hipFree(p->dev_base), "hipFree(device pool)");
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

// Check the current device and the buffers' device against the pool's.
kv_status check_device(const kv_pool *p, int buffers_device) {
    int cur = -1;
    KVX_HIP(hipGetDevice(&cur));
    if (cur != p->device || buffers_device != p->device)
        return kvx::fail(KV_EINVAL, "pool is on device %d, buffers on device %d, current device %d", p->device,
                         buffers_device, cur);
    return KV_OK;
}

// Enqueue the pack/unpack kernels for chunks [chunk0, chunk0 + nchunks) of the prefix.
// slots[c] is the slot id of chunk chunk0 + c relative to chunk_base (slot_stride apart);
// host_side: chunk_base is the mapped pinned pool (zero-copy) rather than device staging.
kv_status enqueue_gather(kv_pool *p, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                         Direction dir, int64_t chunk0, int nchunks, const int32_t *slots, uint8_t *chunk_base,
                         int64_t slot_stride, bool host_side, hipStream_t stream) {
    const Geometry &g0 = p->geo;
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
    KVX_HIP(kvx::launch_gathers(cache, block_table, n_tokens, dir, chunk0, nchunks, slots, chunk_base, slot_stride,
                                host_side, p->err_dev, stream));
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

// One DMA copy of a staged batch: host_base + host_off <-> staging slot + stage_off.
struct Run {
    int64_t host_off;
    int64_t stage_off;
    int64_t bytes;
};

// Append a copy, merging it into the previous one when both sides are contiguous.
void add_run(std::vector<Run> &runs, int64_t host_off, int64_t stage_off, int64_t bytes) {
    if (!runs.empty()) {
        Run &last = runs.back();
        if (last.host_off + last.bytes == host_off && last.stage_off + last.bytes == stage_off) {
            last.bytes += bytes;
            return;
        }
    }
    runs.push_back({host_off, stage_off, bytes});
}

using BatchRuns = std::function<void(int64_t batch, std::vector<Run> &runs)>;
using BatchKernels = std::function<kv_status(int64_t batch, uint8_t *stage)>;

// The staged pipeline over `nbatches` batches, each filling at most one staging slot of the
// direction's own lane.  Store: kernels on the caller's stream pack batch b into staging slot k
// (after the copy that last read slot k), then a side stream copies it to the pool; the caller's
// stream finally waits for every side stream it used (exit join).  Load: an entry event on the
// caller's stream gates the side streams' pool reads; each batch's kernels wait for its copy.
kv_status staged_pipeline(kv_pool *p, int64_t nbatches, const BatchRuns &runs_of, const BatchKernels &kernels,
                          hipStream_t stream, Direction dir) {
    kv_pool::Lane &ln = p->lane[dir];
    const int64_t staging_slot_bytes = static_cast<int64_t>(p->cpb) * p->geo.slot_bytes;
    std::vector<bool> side_used(ln.sides.size(), false);
    std::vector<Run> runs;

    if (dir == kvx::kUnpack)
        KVX_HIP(hipEventRecord(ln.ev_entry, stream));  // entry gate for pool reads

    for (int64_t b = 0; b < nbatches; ++b) {
        const int k = ln.ring;
        ln.ring = (ln.ring + 1) % p->K;
        const size_t si = static_cast<size_t>(b % static_cast<int64_t>(ln.sides.size()));
        hipStream_t side = ln.sides[si];
        uint8_t *stage = ln.staging + static_cast<int64_t>(k) * staging_slot_bytes;
        runs.clear();
        runs_of(b, runs);

        if (dir == kvx::kPack) {
            if (ln.free_recorded[k])
                KVX_HIP(hipStreamWaitEvent(stream, ln.ev_free[k], 0));
            kv_status st = kernels(b, stage);
            if (st != KV_OK)
                return st;
            KVX_HIP(hipEventRecord(ln.ev_ready[k], stream));
            KVX_HIP(hipStreamWaitEvent(side, ln.ev_ready[k], 0));
            for (const Run &run : runs)
                KVX_HIP(hipMemcpyAsync(p->host_base + run.host_off, stage + run.stage_off,
                                       static_cast<size_t>(run.bytes), hipMemcpyDeviceToHost, side));
            KVX_HIP(hipEventRecord(ln.ev_free[k], side));
            ln.free_recorded[k] = true;
            side_used[si] = true;
        } else {
            if (!side_used[si]) {
                KVX_HIP(hipStreamWaitEvent(side, ln.ev_entry, 0));
                side_used[si] = true;
            }
            if (ln.free_recorded[k])
                KVX_HIP(hipStreamWaitEvent(side, ln.ev_free[k], 0));
            for (const Run &run : runs)
                KVX_HIP(hipMemcpyAsync(stage + run.stage_off, p->host_base + run.host_off,
                                       static_cast<size_t>(run.bytes), hipMemcpyHostToDevice, side));
            KVX_HIP(hipEventRecord(ln.ev_ready[k], side));
            KVX_HIP(hipStreamWaitEvent(stream, ln.ev_ready[k], 0));
            kv_status st = kernels(b, stage);
            if (st != KV_OK)
                return st;
            KVX_HIP(hipEventRecord(ln.ev_free[k], stream));
            ln.free_recorded[k] = true;
        }
    }
    if (dir == kvx::kPack) {
        // Exit join: later work on the caller's stream follows every D2H copy.
        for (size_t si = 0; si < ln.sides.size(); ++si) {
            if (!side_used[si])
                continue;
            KVX_HIP(hipEventRecord(ln.ev_join[si], ln.sides[si]));
            KVX_HIP(hipStreamWaitEvent(stream, ln.ev_join[si], 0));
        }
    }
    return KV_OK;
}

kv_status transfer(kv_pool *p, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                   const int64_t *chunk_ids, hipStream_t stream, Direction dir) {
    const Geometry &g = p->geo;
    const int64_t nc = (n_tokens + g.C - 1) / g.C;

    if (p->mode_of[dir] == KV_MODE_ZERO_COPY) {
        std::vector<int32_t> slots(static_cast<size_t>(nc));
        for (int64_t i = 0; i < nc; ++i)
            slots[static_cast<size_t>(i)] = static_cast<int32_t>(chunk_ids[i]);
        for (int64_t c0 = 0; c0 < nc; c0 += p->zc_chunks) {
            const int n = static_cast<int>(std::min<int64_t>(p->zc_chunks, nc - c0));
            kv_status st = enqueue_gather(p, cache, block_table, n_tokens, dir, c0, n, slots.data() + c0,
                                          p->dev_base, g.slot_bytes, !p->on_device, stream);
            if (st != KV_OK)
                return st;
        }
        return KV_OK;
    }

    // Staged mode: batch b holds chunks [b*cpb, b*cpb + cpb) in staging slots 0..cpb-1.
    std::vector<int32_t> local(static_cast<size_t>(p->cpb));
    for (int c = 0; c < p->cpb; ++c)
        local[static_cast<size_t>(c)] = c;
    const int64_t nbatches = (nc + p->cpb - 1) / p->cpb;
    auto runs_of = [&](int64_t b, std::vector<Run> &runs) {
        const int64_t c0 = b * p->cpb;
        const int64_t n = std::min<int64_t>(p->cpb, nc - c0);
        for (int64_t c = 0; c < n; ++c) {
            const int64_t i = c0 + c;
            const int64_t r = std::min<int64_t>(g.C, n_tokens - i * g.C);
            add_run(runs, chunk_ids[i] * g.slot_bytes, c * g.slot_bytes, r * g.token_bytes);
        }
    };
    auto kernels = [&](int64_t b, uint8_t *stage) {
        const int64_t c0 = b * p->cpb;
        const int n = static_cast<int>(std::min<int64_t>(p->cpb, nc - c0));
        return enqueue_gather(p, cache, block_table, n_tokens, dir, c0, n, local.data(), stage, g.slot_bytes,
                              false, stream);
    };
    return staged_pipeline(p, nbatches, runs_of, kernels, stream, dir);
}

// Piece arithmetic of one state request: n snapshots of G pages, each page cut into
// ppp pieces of `piece` bytes (the last piece of a page may be shorter).  Piece q is
// piece j of layer g of snapshot k with q = (k*G + g)*ppp + j; its packed bytes start
// at off(q) in the concatenation of the n packed snapshots.
struct StatePlan {
    int64_t n, G, page_bytes, page_stride, snap_bytes, piece, ppp, pieces;

    StatePlan(const kv_state *st, int64_t n_snap, int64_t piece_bytes)
        : n(n_snap), G(st->num_layers), page_bytes(st->page_bytes),
          page_stride(st->page_stride ? st->page_stride : st->page_bytes), snap_bytes(G * page_bytes),
          piece(std::min(piece_bytes, page_bytes)), ppp((page_bytes + piece - 1) / piece), pieces(n * G * ppp) {}

    int64_t off(int64_t q) const {
        const int64_t per = G * ppp;
        const int64_t k = q / per, rem = q - k * per;
        const int64_t g = rem / ppp, j = rem - g * ppp;
        return k * snap_bytes + g * page_bytes + j * piece;
    }
};

// Enqueue the state kernels for pieces [qa, qb) on `stream`.  base: device-visible packed
// side; snap_off(k): byte offset at base where snapshot k's packed bytes start.
kv_status enqueue_state(kv_pool *p, const kv_state *st, const StatePlan &plan, const int64_t *pages, int64_t qa,
                        int64_t qb, uint8_t *base, const std::function<int64_t(int64_t)> &snap_off, bool host_side,
                        hipStream_t stream, Direction dir) {
    hipEvent_t t_start = nullptr, t_stop = nullptr;
    if (p->profile) {
        kv_status e = take_timing_event(p, &t_start);
        if (e != KV_OK)
            return e;
        e = take_timing_event(p, &t_stop);
        if (e != KV_OK)
            return e;
        KVX_HIP(hipEventRecord(t_start, stream));
    }
    const int64_t per = plan.G * plan.ppp;
    for (int64_t q = qa; q < qb;) {
        const int64_t k_first = q / per;
        const int64_t q_end = std::min({qb, q + kvx::kMaxLaunchPieces, (k_first + kvx::kMaxLaunchSnapshots) * per});
        const int64_t k_last = (q_end - 1) / per;
        kvx::StateArgs a;
        std::memset(&a, 0, sizeof(a));
        for (int64_t g = 0; g < plan.G; ++g)
            a.layer[g] = static_cast<uint8_t *>(st->layer_ptrs[g]);
        a.base = base;
        a.page_stride = plan.page_stride;
        a.page_bytes = plan.page_bytes;
        a.piece = plan.piece;
        a.q0 = q - k_first * per;
        a.G = static_cast<int32_t>(plan.G);
        a.ppp = static_cast<int32_t>(plan.ppp);
        a.nsnap = static_cast<int32_t>(k_last - k_first + 1);
        for (int64_t k = k_first; k <= k_last; ++k) {
            a.page[k - k_first] = pages[k];
            a.off[k - k_first] = snap_off(k);
        }
        KVX_HIP(kvx::launch_state(a, q_end - q, dir, host_side, stream));
        q = q_end;
    }
    if (p->profile) {
        KVX_HIP(hipEventRecord(t_stop, stream));
        p->pending[2 + dir].push_back({t_start, t_stop, 2.0 * static_cast<double>(plan.off(qb) - plan.off(qa))});
    }
    return KV_OK;
}

kv_status transfer_state(kv_pool *p, const kv_state *st, const int64_t *pages, int64_t n, const int64_t *slot_ids,
                         hipStream_t stream, Direction dir) {
    const int64_t S = p->state_slot_bytes;
    if (p->mode_of[dir] == KV_MODE_ZERO_COPY) {
        const StatePlan plan(st, n, kvx::kStatePiece);
        auto off = [&](int64_t k) { return slot_ids[k] * S; };
        return enqueue_state(p, st, plan, pages, 0, plan.pieces, p->dev_base + p->state_offset, off, !p->on_device,
                             stream, dir);
    }

    // Staged mode: cut the pieces into batches of at most one staging slot of bytes.
    const int64_t cap = static_cast<int64_t>(p->cpb) * p->geo.slot_bytes;
    const StatePlan plan(st, n, std::min<int64_t>(kvx::kStatePiece, cap / 16 * 16));
    std::vector<int64_t> cut{0};
    while (cut.back() < plan.pieces) {
        const int64_t qa = cut.back(), oa = plan.off(qa);
        int64_t lo = qa + 1, hi = plan.pieces;  // a single piece always fits
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo + 1) / 2;
            if (plan.off(mid) - oa <= cap)
                lo = mid;
            else
                hi = mid - 1;
        }
        cut.push_back(lo);
    }
    const int64_t nbatches = static_cast<int64_t>(cut.size()) - 1;
    auto runs_of = [&](int64_t b, std::vector<Run> &runs) {
        const int64_t oa = plan.off(cut[b]), ob = plan.off(cut[b + 1]);
        for (int64_t k = oa / S; k * S < ob; ++k) {
            const int64_t lo = std::max(oa, k * S), hi = std::min(ob, (k + 1) * S);
            add_run(runs, p->state_offset + slot_ids[k] * S + (lo - k * S), lo - oa, hi - lo);
        }
    };
    auto kernels = [&](int64_t b, uint8_t *stage) {
        const int64_t oa = plan.off(cut[b]);
        auto off = [&](int64_t k) { return k * S - oa; };
        return enqueue_state(p, st, plan, pages, cut[b], cut[b + 1], stage, off, false, stream, dir);
    };
    return staged_pipeline(p, nbatches, runs_of, kernels, stream, dir);
}

// Record the pool's last use on `stream` (one event per stream with work in flight).  Entries of
// other streams whose recorded work has completed are dropped, so callers that use many
// short-lived streams do not grow the list.
kv_status mark_use(kv_pool *p, hipStream_t stream) {
    for (auto &use : p->last_use)
        if (use.first == stream) {
            KVX_HIP(hipEventRecord(use.second, stream));
            return KV_OK;
        }
    for (size_t i = 0; i < p->last_use.size();) {
        if (hipEventQuery(p->last_use[i].second) == hipSuccess) {
            KVX_HIP(hipEventDestroy(p->last_use[i].second));
            p->last_use[i] = p->last_use.back();
            p->last_use.pop_back();
        } else {
            ++i;
        }
    }
    (void)hipGetLastError();  // a not-ready query leaves no error behind
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
    st = check_device(pool, cache->device);
    if (st != KV_OK)
        return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = transfer(pool, cache, block_table, n_tokens, chunk_ids, s, dir);
    // Record the last use on this stream even after a partial enqueue.
    const kv_status st_use = mark_use(pool, s);
    return st != KV_OK ? st : st_use;
}

kv_status run_state(const kv_state *state, const int64_t *pages, int64_t n, kv_pool *pool, const int64_t *slot_ids,
                    void *stream, Direction dir) {
    if (!pool)
        return kvx::fail(KV_EINVAL, "pool must not be NULL");
    std::lock_guard<std::mutex> lock(pool->mu);
    if (pool->num_state_slots == 0)
        return kvx::fail(KV_EINVAL, "pool was created without a state area (num_state_slots = 0)");
    kv_status st = kvx::check_state_request(state, pool->state_slot_bytes, pool->num_state_slots, n, pages, slot_ids,
                                            dir == kvx::kPack);
    if (st != KV_OK)
        return st;
    if (n == 0)
        return KV_OK;
    st = check_device(pool, state->device);
    if (st != KV_OK)
        return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = transfer_state(pool, state, pages, n, slot_ids, s, dir);
    const kv_status st_use = mark_use(pool, s);
    return st != KV_OK ? st : st_use;
}

}  // namespace

extern "C" {

kv_status kv_pool_create(const kv_layout *layout, int64_t num_slots, const kv_pool_options *opts, kv_pool **out) {
    return kvx::guarded([&]() -> kv_status {
        if (!layout || !opts || !out)
            return kvx::fail(KV_EINVAL, "layout, opts and out must not be NULL");
        *out = nullptr;
        kv_status st = kvx::check_layout(*layout);
        if (st != KV_OK)
            return st;
        if (num_slots <= 0 || num_slots > INT32_MAX)
            return kvx::fail(KV_EINVAL, "num_slots must be in [1, 2^31-1] (got %lld)",
                             static_cast<long long>(num_slots));
        if (opts->mode != KV_MODE_ZERO_COPY && opts->mode != KV_MODE_STAGED)
            return kvx::fail(KV_EINVAL, "opts->mode must be KV_MODE_ZERO_COPY or KV_MODE_STAGED (got %u)", opts->mode);
        if (opts->host_kind != KV_HOST_COHERENT && opts->host_kind != KV_HOST_NONCOHERENT &&
            opts->host_kind != KV_POOL_DEVICE)
            return kvx::fail(KV_EINVAL, "unknown host_kind %u", opts->host_kind);
        const bool on_device = opts->host_kind == KV_POOL_DEVICE;
        if (on_device && (opts->mode != KV_MODE_ZERO_COPY || opts->staging_slots != 0))
            return kvx::fail(KV_EINVAL, "a device pool (KV_POOL_DEVICE) takes KV_MODE_ZERO_COPY and no staging");
        // chunks_per_batch applies to the mode chosen at creation; the other mode keeps its default.
        if (opts->chunks_per_batch < 0 || opts->chunks_per_batch > kvx::kMaxLaunchChunks)
            return kvx::fail(KV_EINVAL, "chunks_per_batch must be in [1, %d] (got %d)", kvx::kMaxLaunchChunks,
                             opts->chunks_per_batch);
        const bool staged = opts->mode == KV_MODE_STAGED;
        const int cpb = (staged && opts->chunks_per_batch) ? opts->chunks_per_batch : kDefaultChunksPerBatch;
        // Zero-copy launches into host memory default to the largest launch (they stride a capped grid);
        // device-pool launches default to the staged launch shape (one workgroup per slab).
        const int zc_chunks = (!staged && opts->chunks_per_batch) ? opts->chunks_per_batch
                              : on_device                        ? kDefaultChunksPerBatch
                                                                 : kvx::kMaxLaunchChunks;
        const bool want_staging = opts->mode == KV_MODE_STAGED || opts->staging_slots > 0;
        const int K = opts->staging_slots ? opts->staging_slots : kDefaultStagingSlots;
        if (want_staging && (K < 2 || K > 64))
            return kvx::fail(KV_EINVAL, "staging_slots must be in [2, 64] (got %d)", K);
        const int S = opts->side_streams ? opts->side_streams : kDefaultSideStreams;
        if (want_staging && (S < 1 || S > 8))
            return kvx::fail(KV_EINVAL, "side_streams must be in [1, 8] (got %d)", S);
        if (opts->num_state_slots < 0 || opts->state_slot_bytes < 0 ||
            (opts->num_state_slots > 0) != (opts->state_slot_bytes > 0))
            return kvx::fail(KV_EINVAL, "num_state_slots (%lld) and state_slot_bytes (%lld) must both be 0 or both > 0",
                             static_cast<long long>(opts->num_state_slots),
                             static_cast<long long>(opts->state_slot_bytes));
        if (opts->state_slot_bytes % 16 != 0)
            return kvx::fail(KV_EUNSUPPORTED, "state_slot_bytes %lld is not a multiple of 16",
                             static_cast<long long>(opts->state_slot_bytes));

        kv_pool *p = new kv_pool();
        p->layout = *layout;
        p->geo = kvx::geometry(*layout, 0);
        p->num_slots = num_slots;
        if (p->geo.slot_bytes > INT64_MAX / num_slots) {
            delete p;
            return kvx::fail(KV_EINVAL, "pool size overflows 64 bits");
        }
        p->pool_bytes = num_slots * p->geo.slot_bytes;
        // The state-snapshot area follows the chunk slots in the same region, 4 KiB aligned.
        p->num_state_slots = opts->num_state_slots;
        p->state_slot_bytes = opts->state_slot_bytes;
        p->state_offset = (p->pool_bytes + 4095) / 4096 * 4096;
        if (p->num_state_slots > 0 && p->state_slot_bytes > (INT64_MAX - p->state_offset) / p->num_state_slots) {
            delete p;
            return kvx::fail(KV_EINVAL, "pool size with the state area overflows 64 bits");
        }
        const int64_t region_bytes =
            p->num_state_slots > 0 ? p->state_offset + p->num_state_slots * p->state_slot_bytes : p->pool_bytes;
        // From here on the pool owns runtime resources: release them if a host container throws.
        try {
            p->mode_of[kvx::kPack] = p->mode_of[kvx::kUnpack] = opts->mode;
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

            if (on_device) {
                // The device-resident tier: one plain allocation of exactly region_bytes.
                p->on_device = true;
                const auto t0 = std::chrono::steady_clock::now();
                void *dptr = nullptr;
                e = hipMalloc(&dptr, static_cast<size_t>(region_bytes));
                const auto t1 = std::chrono::steady_clock::now();
                if (e != hipSuccess || !dptr) {
                    (void)hipGetLastError();
                    const long long want = static_cast<long long>(region_bytes);
                    release(p);
                    return kvx::fail(KV_ENOMEM, "device allocation of %lld bytes for the pool failed (%s)", want,
                                     hipGetErrorName(e));
                }
                p->dev_base = static_cast<uint8_t *>(dptr);
                p->alloc_seconds = std::chrono::duration<double>(t1 - t0).count();
            } else {
                // One pinned, mapped region of exactly region_bytes (Sec. 3.3: no rounding allocator,
                // and never a silent fallback to pageable memory).
                const unsigned flags = hipHostMallocMapped | hipHostMallocPortable |
                                       (p->host_kind == KV_HOST_COHERENT ? hipHostMallocCoherent
                                                                         : hipHostMallocNonCoherent);
                const auto t0 = std::chrono::steady_clock::now();
                void *host = nullptr;
                e = hipHostMalloc(&host, static_cast<size_t>(region_bytes), flags);
                const auto t1 = std::chrono::steady_clock::now();
                if (e != hipSuccess || !host) {
                    (void)hipGetLastError();
                    const long long want = static_cast<long long>(region_bytes);
                    release(p);
                    return kvx::fail(KV_ENOMEM, "pinned allocation of %lld bytes failed (%s); no pageable fallback",
                                     want, hipGetErrorName(e));
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
            }

            e = hipHostMalloc(reinterpret_cast<void **>(&p->err_host), 256,
                              hipHostMallocMapped | hipHostMallocCoherent);
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
                const size_t lane_bytes = static_cast<size_t>(K) * cpb * static_cast<size_t>(p->geo.slot_bytes);
                // Plain device memory.  Physically contiguous staging (hipExtMallocWithFlags with
                // hipDeviceMallocContiguous) was used before, but on MI355X with this runtime, once such
                // an allocation had been freed, later allocations of the process read and wrote wrong
                // bytes (156 of 480 seeded round trips in one process); plain staging measured the same
                // transfer rates.
                p->staging_contiguous = false;
                e = hipMalloc(reinterpret_cast<void **>(&p->staging), 2 * lane_bytes);
                if (e != hipSuccess)
                    return bail(kvx::hip_fail(e, "hipMalloc(staging)", __FILE__, __LINE__));
                for (int d = 0; d < 2; ++d) {
                    kv_pool::Lane &ln = p->lane[d];
                    ln.staging = p->staging + static_cast<size_t>(d) * lane_bytes;
                    for (int s = 0; s < S; ++s) {
                        hipStream_t side = nullptr;
                        // Default priority on purpose: every stream of the library shares one priority.
                        e = hipStreamCreateWithFlags(&side, hipStreamNonBlocking);
                        if (e != hipSuccess)
                            return bail(kvx::hip_fail(e, "hipStreamCreateWithFlags", __FILE__, __LINE__));
                        ln.sides.push_back(side);
                        hipEvent_t j = nullptr;
                        if ((st = make_event(&j, false)) != KV_OK)
                            return bail(st);
                        ln.ev_join.push_back(j);
                    }
                    for (int k = 0; k < K; ++k) {
                        hipEvent_t a = nullptr, b = nullptr;
                        if ((st = make_event(&a, false)) != KV_OK)
                            return bail(st);
                        ln.ev_free.push_back(a);
                        if ((st = make_event(&b, false)) != KV_OK)
                            return bail(st);
                        ln.ev_ready.push_back(b);
                    }
                    ln.free_recorded.assign(static_cast<size_t>(K), false);
                    if ((st = make_event(&ln.ev_entry, false)) != KV_OK)
                        return bail(st);
                }
            }
        } catch (...) {
            release(p);
            throw;
        }
        *out = p;
        return KV_OK;
    });
}

kv_status kv_pool_destroy(kv_pool *pool) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool)
            return KV_OK;
        return release(pool);
    });
}

kv_status kv_pool_get_info(const kv_pool *pool, kv_pool_info *info) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool || !info)
            return kvx::fail(KV_EINVAL, "pool and info must not be NULL");
        std::memset(info, 0, sizeof(*info));
        info->num_slots = pool->num_slots;
        info->slot_bytes = pool->geo.slot_bytes;
        info->pool_bytes = pool->pool_bytes;
        info->staging_bytes =
            pool->staging ? 2 * static_cast<int64_t>(pool->K) * pool->cpb * pool->geo.slot_bytes : 0;
        info->alloc_seconds = pool->alloc_seconds;
        info->device = pool->device;
        info->mode = pool->mode_of[kvx::kPack];
        info->load_mode = pool->mode_of[kvx::kUnpack];
        info->host_kind = pool->host_kind;
        info->is_pinned = pool->pinned ? 1 : 0;
        info->staging_slots = pool->K;
        info->chunks_per_batch = pool->staging ? pool->cpb : pool->zc_chunks;
        info->side_streams = pool->S;
        info->staging_contiguous = pool->staging_contiguous ? 1 : 0;
        info->host_base = pool->host_base;
        info->device_base = pool->dev_base;
        info->num_state_slots = pool->num_state_slots;
        info->state_slot_bytes = pool->state_slot_bytes;
        info->state_host_base =
            pool->num_state_slots > 0 && pool->host_base ? pool->host_base + pool->state_offset : nullptr;
        return KV_OK;
    });
}

void *kv_pool_state_slot(kv_pool *pool, int64_t slot) {
    if (!pool || !pool->host_base || slot < 0 || slot >= pool->num_state_slots)
        return nullptr;
    return pool->host_base + pool->state_offset + slot * pool->state_slot_bytes;
}

void *kv_pool_slot(kv_pool *pool, int64_t slot) {
    if (!pool || !pool->host_base || slot < 0 || slot >= pool->num_slots)
        return nullptr;
    return pool->host_base + slot * pool->geo.slot_bytes;
}

int64_t kv_pool_slot_bytes(const kv_pool *pool) { return pool ? pool->geo.slot_bytes : -1; }

int64_t kv_pool_num_slots(const kv_pool *pool) { return pool ? pool->num_slots : -1; }

kv_status kv_pool_set_modes(kv_pool *pool, uint32_t store_mode, uint32_t load_mode) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool)
            return kvx::fail(KV_EINVAL, "pool must not be NULL");
        std::lock_guard<std::mutex> lock(pool->mu);
        for (uint32_t mode : {store_mode, load_mode}) {
            if (mode != KV_MODE_ZERO_COPY && mode != KV_MODE_STAGED)
                return kvx::fail(KV_EINVAL, "unknown mode %u", mode);
            if (mode == KV_MODE_STAGED && !pool->staging)
                return kvx::fail(KV_EINVAL, "pool was created without staging; staged mode unavailable");
        }
        pool->mode_of[kvx::kPack] = store_mode;
        pool->mode_of[kvx::kUnpack] = load_mode;
        return KV_OK;
    });
}

kv_status kv_pool_set_mode(kv_pool *pool, uint32_t mode) { return kv_pool_set_modes(pool, mode, mode); }

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
    return kvx::guarded([&]() -> kv_status {
        if (!pool || which < 0 || which > 3)
            return kvx::fail(KV_EINVAL,
                             "pool must not be NULL and which must be 0 (pack), 1 (unpack), 2 (state pack) or "
                             "3 (state unpack)");
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
    });
}

kv_status kv_store(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                   const int64_t *chunk_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return run(cache, block_table, n_tokens, pool, chunk_ids, stream, kvx::kPack);
    });
}

kv_status kv_load(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                  const int64_t *chunk_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return run(cache, block_table, n_tokens, pool, chunk_ids, stream, kvx::kUnpack);
    });
}

}  // extern "C"

extern "C" {

kv_status kv_store_state(const kv_state *state, const int64_t *pages, int64_t n, kv_pool *pool,
                         const int64_t *slot_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return run_state(state, pages, n, pool, slot_ids, stream, kvx::kPack);
    });
}

kv_status kv_load_state(const kv_state *state, const int64_t *pages, int64_t n, kv_pool *pool,
                        const int64_t *slot_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return run_state(state, pages, n, pool, slot_ids, stream, kvx::kUnpack);
    });
}

}  // extern "C"

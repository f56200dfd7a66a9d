// kv_load_noalloc: a staged restore that allocates nothing.
//
// kv_load in staged mode copies each batch of chunks from the pinned pool into device staging on
// a side stream and unpacks it on the caller's stream; the staging ring, side streams and events
// are made when the pool is created, and every call records an event of its own.  Callers that
// cannot allocate at all (code under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc) get this variant: the staging is a file-scope device array, the copies and the unpack
// kernels all run on the caller's stream in order, and no runtime object is created per call.
//
// The array's address differs per device.  It is looked up with hipGetSymbolAddress once per
// device, with that device current, on the first call there, and only that address is ever
// handed to copies and kernels: in host code the array's name is a host-side stand-in, not a
// device address.
#include <algorithm>
#include <cstring>

#include "kvx_internal.h"

// 64 MiB: one chunk of the 27B-class layout (256 tokens x 256 KiB), or one 1,568-token chunk of
// the paper's FP8 attention layout (49 MiB).  Each device the library runs on holds it until the
// process ends.
static constexpr int64_t kScratchBytes = KV_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device (looked up once per device).
kv_status scratch_on_current_device(uint8_t **out) {
    int dev = -1;
    KVX_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return kvx::fail(KV_EUNSUPPORTED, "device ordinal %d is beyond the %d the library tracks", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        KVX_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p)
            return kvx::fail(KV_EHIP, "hipGetSymbolAddress(scratch) returned NULL on device %d", dev);
        g_scratch_ptr[dev] = static_cast<uint8_t *>(p);
    }
    *out = g_scratch_ptr[dev];
    return KV_OK;
}

}  // namespace

extern "C" {

kv_status kv_load_noalloc(const kv_cache *cache, const int32_t *block_table, int64_t n_tokens, kv_pool *pool,
                          const int64_t *chunk_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool)
            return kvx::fail(KV_EINVAL, "pool must not be NULL");
        std::lock_guard<std::mutex> lock(pool->mu);
        kv_status st = kvx::check_request(cache, &pool->layout, pool->num_slots, n_tokens, chunk_ids, 0);
        if (st != KV_OK)
            return st;
        if (n_tokens == 0)
            return KV_OK;
        if (!block_table)
            return kvx::fail(KV_EINVAL, "block_table must not be NULL for n_tokens > 0");
        if (pool->on_device || !pool->host_base)
            return kvx::fail(KV_EINVAL, "kv_load_noalloc restores from a host pool; a device pool needs no staging");
        const kvx::Geometry &g = pool->geo;
        if (g.slot_bytes > kScratchBytes)
            return kvx::fail(KV_EUNSUPPORTED, "a chunk of %lld bytes exceeds the %lld-byte static scratch",
                             static_cast<long long>(g.slot_bytes), static_cast<long long>(kScratchBytes));
        int cur = -1;
        KVX_HIP(hipGetDevice(&cur));
        if (cur != pool->device || cache->device != pool->device)
            return kvx::fail(KV_EINVAL, "pool is on device %d, buffers on device %d, current device %d", pool->device,
                             cache->device, cur);
        uint8_t *stage = nullptr;
        st = scratch_on_current_device(&stage);
        if (st != KV_OK)
            return st;

        hipStream_t s = static_cast<hipStream_t>(stream);
        const int64_t nc = (n_tokens + g.C - 1) / g.C;
        const int per_batch = static_cast<int>(std::min<int64_t>(kScratchBytes / g.slot_bytes, kvx::kMaxLaunchChunks));
        int32_t local[kvx::kMaxLaunchChunks];
        for (int c = 0; c < per_batch; ++c)
            local[c] = c;
        // Batch b: copy its chunks into scratch (consecutive slots merged into one copy), then unpack them.
        // The next batch's copy follows this batch's kernels on the same stream, so the scratch is free.
        for (int64_t c0 = 0; c0 < nc; c0 += per_batch) {
            const int nb = static_cast<int>(std::min<int64_t>(per_batch, nc - c0));
            int64_t run_src = -1, run_dst = 0, run_bytes = 0;
            for (int c = 0; c <= nb; ++c) {
                int64_t src = -1, bytes = 0;
                if (c < nb) {
                    const int64_t i = c0 + c;
                    src = chunk_ids[i] * g.slot_bytes;
                    bytes = std::min<int64_t>(g.C, n_tokens - i * g.C) * g.token_bytes;
                }
                const int64_t dst = static_cast<int64_t>(c) * g.slot_bytes;
                if (run_bytes && c < nb && run_src + run_bytes == src && run_dst + run_bytes == dst) {
                    run_bytes += bytes;
                    continue;
                }
                if (run_bytes)
                    KVX_HIP(hipMemcpyAsync(stage + run_dst, pool->host_base + run_src, static_cast<size_t>(run_bytes),
                                           hipMemcpyHostToDevice, s));
                run_src = src;
                run_dst = dst;
                run_bytes = bytes;
            }
            KVX_HIP(kvx::launch_gathers(cache, block_table, n_tokens, kvx::kUnpack, c0, nb, local, stage,
                                        g.slot_bytes, false, pool->err_dev, s));
        }
        return KV_OK;
    });
}

}  // extern "C"

// Host-only pieces of kvx: error reporting and request validation.  Nothing here calls
// the HIP runtime except hip_fail's error-name lookup, so kv_check works without a GPU.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <unordered_set>

#include "kvx_internal.h"

namespace kvx {

namespace {
thread_local std::string g_last_error;
}

kv_status fail(kv_status code, const char *fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = std::string(kv_status_name(code)) + ": " + buf;
    return code;
}

void set_last_error(const std::string &msg) { g_last_error = msg; }

kv_status hip_fail(hipError_t err, const char *what, const char *file, int line) {
    const kv_status code = (err == hipErrorOutOfMemory || err == hipErrorMemoryAllocation) ? KV_ENOMEM : KV_EHIP;
    return fail(code, "%s failed: %s (%s) at %s:%d", what, hipGetErrorName(err), hipGetErrorString(err), file, line);
}

Geometry geometry(const kv_layout &lay, int64_t block_stride_bytes) {
    Geometry g{};
    g.L = lay.num_layers;
    g.H = lay.num_kv_heads;
    g.D = lay.head_dim;
    g.E = lay.elem_bytes;
    g.BS = lay.block_size;
    g.C = lay.chunk_tokens;
    g.row_bytes = g.D * g.E;
    g.vec_per_row = g.row_bytes / 16;
    g.block_bytes = 2 * g.H * g.BS * g.row_bytes;
    g.block_stride = block_stride_bytes ? block_stride_bytes : g.block_bytes;
    g.token_bytes = 2 * g.L * g.H * g.row_bytes;
    g.slot_bytes = g.C * g.token_bytes;
    g.blocks_per_chunk = g.BS > 0 ? g.C / g.BS : 0;
    return g;
}

kv_status check_layout(const kv_layout &lay) {
    if (lay.num_layers <= 0 || lay.num_kv_heads <= 0 || lay.head_dim <= 0 || lay.block_size <= 0 ||
        lay.chunk_tokens <= 0)
        return fail(KV_EINVAL, "layout sizes must be positive (L=%d H=%d D=%d BS=%d C=%d)", lay.num_layers,
                    lay.num_kv_heads, lay.head_dim, lay.block_size, lay.chunk_tokens);
    if (lay.elem_bytes != 1 && lay.elem_bytes != 2 && lay.elem_bytes != 4)
        return fail(KV_EINVAL, "elem_bytes must be 1, 2 or 4 (got %d)", lay.elem_bytes);
    if (lay.chunk_tokens % lay.block_size != 0)
        return fail(KV_EINVAL, "chunk_tokens %d is not a whole number of %d-token blocks", lay.chunk_tokens,
                    lay.block_size);
    const int64_t row = static_cast<int64_t>(lay.head_dim) * lay.elem_bytes;
    if (row % 16 != 0)
        return fail(KV_EUNSUPPORTED, "head_dim*elem_bytes = %lld is not a multiple of 16 bytes",
                    static_cast<long long>(row));
    // Slabs (one block's K or V) are addressed with signed 32-bit byte offsets: at most 2 GiB
    // per block.
    const int64_t block_bytes = 2LL * lay.num_kv_heads * lay.block_size * row;
    if (block_bytes > (int64_t{1} << 31))
        return fail(KV_EUNSUPPORTED, "block of %lld bytes is too large (at most 2 GiB)",
                    static_cast<long long>(block_bytes));
    return KV_OK;
}

static bool same_layout(const kv_layout &a, const kv_layout &b) {
    return a.num_layers == b.num_layers && a.num_kv_heads == b.num_kv_heads && a.head_dim == b.head_dim &&
           a.elem_bytes == b.elem_bytes && a.block_size == b.block_size && a.chunk_tokens == b.chunk_tokens;
}

kv_status check_request(const kv_cache *cache, const kv_layout *pool_layout, int64_t pool_slots, int64_t n_tokens,
                        const int64_t *chunk_ids, int for_store) {
    if (!cache || !pool_layout)
        return fail(KV_EINVAL, "cache and pool layout must not be NULL");
    kv_status st = check_layout(cache->layout);
    if (st != KV_OK)
        return st;
    if (!same_layout(cache->layout, *pool_layout))
        return fail(KV_EINVAL,
                    "cache layout (L=%d H=%d D=%d E=%d BS=%d C=%d) differs from the pool's "
                    "(L=%d H=%d D=%d E=%d BS=%d C=%d)",
                    cache->layout.num_layers, cache->layout.num_kv_heads, cache->layout.head_dim,
                    cache->layout.elem_bytes, cache->layout.block_size, cache->layout.chunk_tokens,
                    pool_layout->num_layers, pool_layout->num_kv_heads, pool_layout->head_dim,
                    pool_layout->elem_bytes, pool_layout->block_size, pool_layout->chunk_tokens);
    if (cache->num_blocks <= 0)
        return fail(KV_EINVAL, "num_blocks must be positive (got %d)", cache->num_blocks);
    if (cache->block_order != KV_BLOCK_HND && cache->block_order != KV_BLOCK_NHD)
        return fail(KV_EINVAL, "block_order must be KV_BLOCK_HND or KV_BLOCK_NHD (got %d)", cache->block_order);
    if (cache->reserved != 0)
        return fail(KV_EINVAL, "kv_cache.reserved must be 0");
    const Geometry g = geometry(cache->layout, cache->block_stride_bytes);
    if (cache->block_stride_bytes != 0 && cache->block_stride_bytes < g.block_bytes)
        return fail(KV_EINVAL, "block_stride_bytes %lld is smaller than one block (%lld bytes)",
                    static_cast<long long>(cache->block_stride_bytes), static_cast<long long>(g.block_bytes));
    if (g.block_stride % 16 != 0)
        return fail(KV_EUNSUPPORTED, "block_stride_bytes %lld is not 16-byte aligned",
                    static_cast<long long>(g.block_stride));
    if (pool_slots > INT32_MAX)
        return fail(KV_EUNSUPPORTED, "more than 2^31-1 pool slots");
    if (n_tokens < 0)
        return fail(KV_EINVAL, "n_tokens must be >= 0 (got %lld)", static_cast<long long>(n_tokens));
    if (n_tokens == 0)
        return KV_OK;
    const int64_t blocks_needed = (n_tokens + g.BS - 1) / g.BS;
    if (blocks_needed > INT32_MAX)
        return fail(KV_EUNSUPPORTED, "prefix of %lld tokens needs more than 2^31-1 blocks",
                    static_cast<long long>(n_tokens));
    if (!cache->layer_ptrs)
        return fail(KV_EINVAL, "layer_ptrs must not be NULL");
    for (int l = 0; l < cache->layout.num_layers; ++l) {
        const uintptr_t p = reinterpret_cast<uintptr_t>(cache->layer_ptrs[l]);
        if (p == 0)
            return fail(KV_EINVAL, "layer_ptrs[%d] is NULL", l);
        if (p % 16 != 0)
            return fail(KV_EUNSUPPORTED, "layer_ptrs[%d] is not 16-byte aligned", l);
    }
    if (!chunk_ids)
        return fail(KV_EINVAL, "chunk_ids must not be NULL for n_tokens > 0");
    const int64_t nc = (n_tokens + g.C - 1) / g.C;
    for (int64_t i = 0; i < nc; ++i)
        if (chunk_ids[i] < 0 || chunk_ids[i] >= pool_slots)
            return fail(KV_EINVAL, "chunk_ids[%lld] = %lld is outside [0, %lld)", static_cast<long long>(i),
                        static_cast<long long>(chunk_ids[i]), static_cast<long long>(pool_slots));
    if (for_store) {
        std::unordered_set<int64_t> seen;
        seen.reserve(static_cast<size_t>(nc) * 2);
        for (int64_t i = 0; i < nc; ++i)
            if (!seen.insert(chunk_ids[i]).second)
                return fail(KV_EINVAL, "chunk id %lld appears twice in one store",
                            static_cast<long long>(chunk_ids[i]));
    }
    return KV_OK;
}

kv_status check_state_request(const kv_state *state, int64_t pool_state_slot_bytes, int64_t pool_state_slots,
                              int64_t n, const int64_t *pages, const int64_t *slot_ids, int for_store) {
    if (!state)
        return fail(KV_EINVAL, "state must not be NULL");
    const int64_t G = state->num_layers, pb = state->page_bytes;
    const int64_t stride = state->page_stride ? state->page_stride : pb;
    if (G < 1)
        return fail(KV_EINVAL, "state num_layers must be >= 1 (got %lld)", static_cast<long long>(G));
    if (pb < 1)
        return fail(KV_EINVAL, "page_bytes must be >= 1 (got %lld)", static_cast<long long>(pb));
    if (stride < pb)
        return fail(KV_EINVAL, "page_stride %lld is smaller than page_bytes %lld", static_cast<long long>(stride),
                    static_cast<long long>(pb));
    if (state->num_pages < 1)
        return fail(KV_EINVAL, "num_pages must be >= 1 (got %lld)", static_cast<long long>(state->num_pages));
    if (pb > INT64_MAX / G || G * pb != pool_state_slot_bytes)
        return fail(KV_EINVAL, "snapshot of %lld layers x %lld bytes differs from the pool's state slot of %lld bytes",
                    static_cast<long long>(G), static_cast<long long>(pb),
                    static_cast<long long>(pool_state_slot_bytes));
    if (G > kMaxStateLayers)
        return fail(KV_EUNSUPPORTED, "more than %d recurrent layers", kMaxStateLayers);
    if (pb % 16 != 0 || stride % 16 != 0)
        return fail(KV_EUNSUPPORTED, "page_bytes %lld and page_stride %lld must be multiples of 16",
                    static_cast<long long>(pb), static_cast<long long>(stride));
    if (state->num_pages > INT64_MAX / stride)
        return fail(KV_EUNSUPPORTED, "page buffer size overflows 64 bits");
    if (n < 0)
        return fail(KV_EINVAL, "n must be >= 0 (got %lld)", static_cast<long long>(n));
    if (n == 0)
        return KV_OK;
    if (!state->layer_ptrs)
        return fail(KV_EINVAL, "state layer_ptrs must not be NULL");
    for (int64_t g = 0; g < G; ++g) {
        const uintptr_t p = reinterpret_cast<uintptr_t>(state->layer_ptrs[g]);
        if (p == 0)
            return fail(KV_EINVAL, "state layer_ptrs[%lld] is NULL", static_cast<long long>(g));
        if (p % 16 != 0)
            return fail(KV_EUNSUPPORTED, "state layer_ptrs[%lld] is not 16-byte aligned", static_cast<long long>(g));
    }
    if (!pages || !slot_ids)
        return fail(KV_EINVAL, "pages and slot_ids must not be NULL for n > 0");
    for (int64_t k = 0; k < n; ++k) {
        if (pages[k] < 0 || pages[k] >= state->num_pages)
            return fail(KV_EINVAL, "pages[%lld] = %lld is outside [0, %lld)", static_cast<long long>(k),
                        static_cast<long long>(pages[k]), static_cast<long long>(state->num_pages));
        if (slot_ids[k] < 0 || slot_ids[k] >= pool_state_slots)
            return fail(KV_EINVAL, "slot_ids[%lld] = %lld is outside [0, %lld)", static_cast<long long>(k),
                        static_cast<long long>(slot_ids[k]), static_cast<long long>(pool_state_slots));
    }
    // The side this call writes must not be named twice.
    const int64_t *written = for_store ? slot_ids : pages;
    std::unordered_set<int64_t> seen;
    seen.reserve(static_cast<size_t>(n) * 2);
    for (int64_t k = 0; k < n; ++k)
        if (!seen.insert(written[k]).second)
            return fail(KV_EINVAL, "%s %lld appears twice in one %s", for_store ? "state slot" : "page",
                        static_cast<long long>(written[k]), for_store ? "store" : "load");
    return KV_OK;
}

}  // namespace kvx

extern "C" {

const char *kv_last_error(void) { return kvx::g_last_error.c_str(); }

const char *kv_status_name(kv_status status) {
    switch (status) {
    case KV_OK:
        return "KV_OK";
    case KV_EINVAL:
        return "KV_EINVAL";
    case KV_ENOMEM:
        return "KV_ENOMEM";
    case KV_EHIP:
        return "KV_EHIP";
    case KV_EUNSUPPORTED:
        return "KV_EUNSUPPORTED";
    case KV_EASYNC:
        return "KV_EASYNC";
    case KV_EBUSY:
        return "KV_EBUSY";
    default:
        return "KV_UNKNOWN";
    }
}

const char *kv_version(void) { return "kvx 0.1.0 (gfx950)"; }

kv_status kv_check(const kv_cache *cache, const kv_layout *pool_layout, int64_t pool_slots, int64_t n_tokens,
                   const int64_t *chunk_ids, int for_store) {
    return kvx::guarded([&]() -> kv_status {
        return kvx::check_request(cache, pool_layout, pool_slots, n_tokens, chunk_ids, for_store);
    });
}

kv_status kv_check_state(const kv_state *state, int64_t pool_state_slot_bytes, int64_t pool_state_slots, int64_t n,
                         const int64_t *pages, const int64_t *slot_ids, int for_store) {
    return kvx::guarded([&]() -> kv_status {
        return kvx::check_state_request(state, pool_state_slot_bytes, pool_state_slots, n, pages, slot_ids, for_store);
    });
}

}  // extern "C"

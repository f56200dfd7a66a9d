// Tier: one process owns the pinned pool; replicas in other processes store and load
// through it over a stream socket, passing their caches as HIP IPC handles.
//
// The paper's replicas share one host tier (Sec. 2, Fig. 1) and its fault is a consumer
// running before its producer completed (Sec. 3.2).  Here a pinned region cannot be
// registered in a second process, so the process that pinned the pool also runs every
// copy into and out of it; replicas hand over device memory instead.  Both ends complete
// on the host before handing over: the replica synchronises its stream before sending,
// and the tier synchronises its own stream before replying.  With an index the tier also
// chooses the slots: prefix requests name a prompt, and the tier stores the prompt's
// missing whole chunks or loads its longest whole-chunk hit.
//
// Frames are native-layout structs (both ends run on one host): a request header, the
// layers' IPC buffers, the block table, the chunk ids and the prompt's tokens; a reply
// header and a message.
#include <sys/socket.h>
#include <sys/types.h>
#include <sys/un.h>
#include <unistd.h>

#include <algorithm>
#include <array>
#include <cerrno>
#include <cstring>
#include <deque>
#include <map>
#include <string>
#include <thread>
#include <vector>

#include "kvx_internal.h"

namespace {

constexpr uint32_t kMagic = 0x5458564Bu;  // "KVXT"
enum Op : uint32_t { kOpStore = 1, kOpLoad = 2, kOpStorePrefix = 3, kOpLoadPrefix = 4 };
constexpr int32_t kMaxLayers = 4096;
constexpr int64_t kMaxPayload = int64_t(1) << 30;

struct RequestHeader {
    uint32_t magic;
    uint32_t op;
    kv_layout layout;
    int32_t num_blocks;
    int32_t block_order;
    int32_t num_layers;
    int32_t pad;
    int64_t block_stride_bytes;
    int64_t n_tokens;
    int64_t n_table;   // int32 block-table entries after the layers
    int64_t n_chunks;  // int64 chunk ids after the table (slot requests)
    int64_t n_ids;     // int32 token ids after the chunk ids (prefix requests)
    uint64_t salt;
    // Recurrent-state pages (prefix requests of hybrid models): state_layers IPC buffers follow
    // the cache's layers; the snapshot is page `page` of each.
    int32_t state_layers;  // 0 = no state
    int32_t pad2;
    int64_t page_bytes, page_stride, num_pages, page;
};

struct ReplyHeader {
    uint32_t magic;
    int32_t status;
    uint32_t msg_len;
    uint32_t pad;
    int64_t value;   // chunks stored (store prefix) or tokens hit (load prefix)
    int64_t value2;  // snapshots stored (store prefix)
};

// Whole-buffer socket I/O.  Returns false on EOF or error (errno kept); *eof set on a clean
// end before the first byte.
bool read_full(int fd, void *buf, size_t n, bool *eof = nullptr) {
    auto *p = static_cast<uint8_t *>(buf);
    size_t done = 0;
    if (eof)
        *eof = false;
    while (done < n) {
        const ssize_t r = recv(fd, p + done, n - done, 0);
        if (r == 0) {
            if (eof && done == 0)
                *eof = true;
            return false;
        }
        if (r < 0) {
            if (errno == EINTR)
                continue;
            return false;
        }
        done += static_cast<size_t>(r);
    }
    return true;
}

bool write_full(int fd, const void *buf, size_t n) {
    const auto *p = static_cast<const uint8_t *>(buf);
    size_t done = 0;
    while (done < n) {
        const ssize_t r = send(fd, p + done, n - done, MSG_NOSIGNAL);
        if (r < 0) {
            if (errno == EINTR)
                continue;
            return false;
        }
        done += static_cast<size_t>(r);
    }
    return true;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

kv_status check_ipc_buffer(const kv_ipc_buffer *buf, int64_t need);

// The tier end of one connection.
class Connection {
  public:
    Connection(kv_pool *pool, kv_index *index, int fd) : pool_(pool), index_(index), fd_(fd) {}

    ~Connection() {
        // Every request completed on the tier stream before its reply; the wait below only
        // guards the mappings against work a failed request might have left behind.
        if (!opened_.empty()) {
            std::lock_guard<std::mutex> lock(pool_->tier_mu);
            if (pool_->tier_stream)
                (void)hipStreamSynchronize(pool_->tier_stream);
            for (auto &kv : opened_)
                (void)hipIpcCloseMemHandle(kv.second.base);
        }
    }

    kv_status serve() {
        KVX_HIP(hipSetDevice(pool_->device));
        for (;;) {
            RequestHeader h;
            bool eof = false;
            if (!read_full(fd_, &h, sizeof(h), &eof)) {
                if (eof)
                    return KV_OK;
                return kvx::fail(KV_EINVAL, "tier: connection failed while reading a request (%s)",
                                 std::strerror(errno));
            }
            if (h.magic != kMagic || h.op < kOpStore || h.op > kOpLoadPrefix || h.num_layers < 1 ||
                h.num_layers > kMaxLayers || h.n_table < 0 || h.n_chunks < 0 || h.n_ids < 0 ||
                h.state_layers < 0 || h.state_layers > kMaxLayers || h.n_table > kMaxPayload ||
                h.n_chunks > kMaxPayload || h.n_ids > kMaxPayload)
                return kvx::fail(KV_EINVAL, "tier: malformed request header");
            const int64_t payload = static_cast<int64_t>(h.num_layers + h.state_layers) *
                                        int64_t(sizeof(kv_ipc_buffer)) +
                                    h.n_table * int64_t(sizeof(int32_t)) + h.n_chunks * int64_t(sizeof(int64_t)) +
                                    h.n_ids * int64_t(sizeof(int32_t));
            if (payload > kMaxPayload)
                return kvx::fail(KV_EINVAL, "tier: request payload of %lld bytes is too large",
                                 static_cast<long long>(payload));
            bufs_.resize(static_cast<size_t>(h.num_layers));
            state_bufs_.resize(static_cast<size_t>(h.state_layers));
            table_host_.resize(static_cast<size_t>(h.n_table));
            ids_.resize(static_cast<size_t>(h.n_chunks));
            tokens_.resize(static_cast<size_t>(h.n_ids));
            if (!read_full(fd_, bufs_.data(), bufs_.size() * sizeof(kv_ipc_buffer)) ||
                !read_full(fd_, state_bufs_.data(), state_bufs_.size() * sizeof(kv_ipc_buffer)) ||
                !read_full(fd_, table_host_.data(), table_host_.size() * sizeof(int32_t)) ||
                !read_full(fd_, ids_.data(), ids_.size() * sizeof(int64_t)) ||
                !read_full(fd_, tokens_.data(), tokens_.size() * sizeof(int32_t)))
                return kvx::fail(KV_EINVAL, "tier: connection failed while reading a request body");

            kv_status st;
            int64_t value = 0, value2 = 0;
            {
                std::lock_guard<std::mutex> lock(pool_->tier_mu);
                st = kvx::tier_resources(pool_, table_host_.size() * sizeof(int32_t));
                if (st == KV_OK) {
                    stream_ = pool_->tier_stream;
                    table_ = pool_->tier_table;
                    st = execute(h, &value, &value2);
                }
            }
            const std::string msg = st == KV_OK ? std::string() : std::string(kv_last_error());
            ReplyHeader r{kMagic, st, static_cast<uint32_t>(msg.size()), 0, value, value2};
            if (!write_full(fd_, &r, sizeof(r)) || !write_full(fd_, msg.data(), msg.size()))
                return kvx::fail(KV_EINVAL, "tier: connection failed while replying (%s)", std::strerror(errno));
        }
    }

  private:
    // Open (once per connection) the allocation behind an IPC buffer; *out = the buffer's address
    // in this process if [offset, offset + need) lies inside the mapping opened here.
    kv_status open_buffer(const kv_ipc_buffer &buf, int64_t need, const char *what, int32_t l, void **out) {
        std::array<uint8_t, 64> key;
        std::memcpy(key.data(), buf.handle, 64);
        auto it = opened_.find(key);
        if (it == opened_.end()) {
            // The declared allocation is checked before the open: opening one of 2 GiB or more has
            // not returned on the machines this library was measured on.
            kv_status st = check_ipc_buffer(&buf, need);
            if (st != KV_OK)
                return kvx::fail(st, "tier: %s %d: %s", what, l, kv_last_error());
            hipIpcMemHandle_t handle;
            static_assert(sizeof(handle) == 64, "IPC handle size");
            std::memcpy(&handle, buf.handle, 64);
            void *base = nullptr;
            KVX_HIP(hipIpcOpenMemHandle(&base, handle, hipIpcMemLazyEnablePeerAccess));
            // The mapping's own size bounds every access (the peer's word is not trusted).
            void *range_base = nullptr;
            size_t size = 0;
            const hipError_t e = hipMemGetAddressRange(&range_base, &size, base);
            if (e != hipSuccess) {
                (void)hipIpcCloseMemHandle(base);
                return kvx::hip_fail(e, "hipMemGetAddressRange(opened IPC buffer)", __FILE__, __LINE__);
            }
            it = opened_.emplace(key, Mapping{base, static_cast<int64_t>(size)}).first;
        }
        if (buf.offset < 0 || need < 0 || need > it->second.bytes || buf.offset > it->second.bytes - need)
            return kvx::fail(KV_EINVAL, "tier: %s %d (offset %lld, %lld bytes) exceeds its shared allocation of %lld "
                                        "bytes",
                             what, l, static_cast<long long>(buf.offset), static_cast<long long>(need),
                             static_cast<long long>(it->second.bytes));
        *out = static_cast<uint8_t *>(it->second.base) + buf.offset;
        return KV_OK;
    }

    // The replica's recurrent-state pages as this process sees them.
    kv_status map_state(const RequestHeader &h, kv_state *state) {
        const int64_t stride = h.page_stride ? h.page_stride : h.page_bytes;
        if (h.page_bytes < 1 || stride < h.page_bytes || h.num_pages < 1 || h.page < 0 || h.page >= h.num_pages ||
            h.num_pages > INT64_MAX / stride)
            return kvx::fail(KV_EINVAL, "tier: invalid recurrent-state pages");
        state_layers_.resize(static_cast<size_t>(h.state_layers));
        for (int32_t g = 0; g < h.state_layers; ++g) {
            kv_status st = open_buffer(state_bufs_[g], (h.num_pages - 1) * stride + h.page_bytes, "state layer", g,
                                       &state_layers_[static_cast<size_t>(g)]);
            if (st != KV_OK)
                return st;
        }
        std::memset(state, 0, sizeof(*state));
        state->num_layers = h.state_layers;
        state->device = pool_->device;
        state->page_bytes = h.page_bytes;
        state->page_stride = h.page_stride;
        state->num_pages = h.num_pages;
        state->layer_ptrs = state_layers_.data();
        return KV_OK;
    }

    // The replica's cache as this process sees it (layers mapped once per connection, each
    // bounded by the size of the mapping opened here), and its block table on the device.
    kv_status map_cache(const RequestHeader &h, kv_cache *cache) {
        const kv_layout &lay = h.layout;
        kv_status st = kvx::check_layout(lay);
        if (st != KV_OK)
            return st;
        if (h.block_stride_bytes < 0)
            return kvx::fail(KV_EINVAL, "tier: negative block stride");
        const kvx::Geometry g = kvx::geometry(lay, h.block_stride_bytes);
        if (h.num_blocks < 1)
            return kvx::fail(KV_EINVAL, "tier: num_blocks must be positive");
        layers_.resize(static_cast<size_t>(h.num_layers));
        for (int32_t l = 0; l < h.num_layers; ++l) {
            if (g.block_stride > INT64_MAX / h.num_blocks)
                return kvx::fail(KV_EINVAL, "tier: layer extent overflows 64 bits");
            st = open_buffer(bufs_[l], static_cast<int64_t>(h.num_blocks) * g.block_stride, "layer", l,
                             &layers_[static_cast<size_t>(l)]);
            if (st != KV_OK)
                return st;
        }

        // The block table into device memory on the tier stream, from pinned host memory (an
        // asynchronous copy from pageable memory would take the runtime's staged path).  The
        // previous request completed before its reply, so the staging is free.
        const size_t table_bytes = table_host_.size() * sizeof(int32_t);
        if (table_bytes) {
            std::memcpy(pool_->tier_table_pinned, table_host_.data(), table_bytes);
            KVX_HIP(hipMemcpyAsync(table_, pool_->tier_table_pinned, table_bytes, hipMemcpyHostToDevice, stream_));
        }

        std::memset(cache, 0, sizeof(*cache));
        cache->layout = lay;
        cache->num_blocks = h.num_blocks;
        cache->device = pool_->device;
        cache->block_order = h.block_order;
        cache->layer_ptrs = layers_.data();
        cache->block_stride_bytes = h.block_stride_bytes;
        return KV_OK;
    }

    // Complete everything enqueued on this connection's stream; then the request's own status
    // (an enqueue error, a failed synchronisation or a device-side fault, in that order).
    kv_status complete(kv_status enqueued) {
        const std::string enqueue_error = enqueued != KV_OK ? std::string(kv_last_error()) : std::string();
        const hipError_t e = hipStreamSynchronize(stream_);
        if (enqueued != KV_OK) {
            kvx::set_last_error(enqueue_error);
            return enqueued;
        }
        if (e != hipSuccess)
            return kvx::hip_fail(e, "hipStreamSynchronize(tier)", __FILE__, __LINE__);
        const int32_t async = kv_pool_async_error(pool_, 1);
        if (async != 0)
            return kvx::fail(KV_EASYNC, "tier: device-side fault 0x%x in this request (a block id was outside "
                                        "the cache)", static_cast<unsigned>(async));
        return KV_OK;
    }

    kv_status execute(const RequestHeader &h, int64_t *value, int64_t *value2) {
        const kv_layout &lay = h.layout;
        if (lay.block_size < 1 || lay.chunk_tokens < 1 || h.n_tokens < 0 || h.n_tokens > (int64_t{1} << 48) ||
            lay.num_layers != h.num_layers)
            return kvx::fail(KV_EINVAL, "tier: request layout or length is invalid");
        if (h.n_table != ceil_div(h.n_tokens, lay.block_size))
            return kvx::fail(KV_EINVAL, "tier: block table does not match n_tokens");
        const bool prefix = h.op == kOpStorePrefix || h.op == kOpLoadPrefix;
        if (!prefix && (h.n_chunks != ceil_div(h.n_tokens, lay.chunk_tokens) || h.n_ids != 0))
            return kvx::fail(KV_EINVAL, "tier: chunk ids do not match n_tokens");
        if (prefix && (h.n_ids != h.n_tokens || h.n_chunks != 0))
            return kvx::fail(KV_EINVAL, "tier: a prefix request carries its n_tokens token ids and no chunk ids");
        if (prefix && !index_)
            return kvx::fail(KV_EINVAL, "tier: this tier serves no index, so it takes no prefix requests");
        if (prefix && (kvx::index_chunk_tokens(index_) != lay.chunk_tokens ||
                       kvx::index_num_slots(index_) > pool_->num_slots ||
                       kvx::index_num_state_slots(index_) > pool_->num_state_slots))
            return kvx::fail(KV_EINVAL, "tier: the index does not match the pool (chunk length or slot counts)");
        if (h.state_layers && !prefix)
            return kvx::fail(KV_EINVAL, "tier: recurrent state travels with prefix requests only");
        if (h.n_tokens == 0)
            return KV_OK;

        kv_cache cache;
        kv_status st = map_cache(h, &cache);
        if (st != KV_OK)
            return complete(st);
        kv_state state;
        if (h.state_layers) {
            st = map_state(h, &state);
            if (st != KV_OK)
                return complete(st);
        }
        (void)kv_pool_async_error(pool_, 1);
        switch (h.op) {
        case kOpStore:
            return complete(kv_store(&cache, table_, h.n_tokens, pool_, ids_.data(), stream_));
        case kOpLoad:
            return complete(kv_load(&cache, table_, h.n_tokens, pool_, ids_.data(), stream_));
        case kOpStorePrefix:
            return store_prefix(h, cache, h.state_layers ? &state : nullptr, value, value2);
        default:
            return load_prefix(h, cache, h.state_layers ? &state : nullptr, value);
        }
    }

    kv_status store_prefix(const RequestHeader &h, const kv_cache &cache, const kv_state *state, int64_t *stored,
                           int64_t *stored_state) {
        const int64_t C = h.layout.chunk_tokens, bpc = C / h.layout.block_size;
        const int64_t nfull = h.n_tokens / C;
        slots_.resize(static_cast<size_t>(nfull));
        is_new_.resize(static_cast<size_t>(nfull));
        int64_t n_chunks = 0;
        kv_status st = kv_index_reserve(index_, h.salt, tokens_.data(), h.n_tokens, slots_.data(), is_new_.data(),
                                        &n_chunks);
        if (st != KV_OK)
            return complete(st);
        // Runs of consecutive new chunks, one store each (chunk i uses table entries from i*C/BS).
        int64_t count = 0;
        for (int64_t a = 0; a < n_chunks && st == KV_OK;) {
            if (!is_new_[a]) {
                ++a;
                continue;
            }
            int64_t b = a;
            while (b < n_chunks && is_new_[b])
                ++b;
            st = kv_store(&cache, table_ + a * bpc, (b - a) * C, pool_, slots_.data() + a, stream_);
            if (st == KV_OK)
                count += b - a;
            a = b;
        }
        // The snapshot at the boundary after the last whole chunk (Sec. 2.2), unless it has one.
        int64_t state_slot = -1;
        int32_t state_new = 0;
        if (st == KV_OK && state && n_chunks > 0) {
            st = kv_index_reserve_state(index_, slots_[n_chunks - 1], &state_slot, &state_new);
            if (st == KV_OK && state_new)
                st = kv_store_state(state, &h.page, 1, pool_, &state_slot, stream_);
        }
        st = complete(st);
        // Publish only what completed without fault (Sec. 3.2); otherwise abort it all.
        kv_status commit = KV_OK;
        if (state_new)
            commit = kv_index_commit_state(index_, slots_[n_chunks - 1], st == KV_OK);
        const kv_status commit_chunks =
            kv_index_commit(index_, slots_.data(), is_new_.data(), n_chunks, st == KV_OK);
        if (st != KV_OK)
            return st;
        if (commit != KV_OK)
            return commit;
        if (commit_chunks != KV_OK)
            return commit_chunks;
        *stored = count;
        *stored_state = state_new;
        return KV_OK;
    }

    kv_status load_prefix(const RequestHeader &h, const kv_cache &cache, const kv_state *state,
                          int64_t *hit_tokens) {
        const int64_t nfull = h.n_tokens / h.layout.chunk_tokens;
        slots_.resize(static_cast<size_t>(nfull));
        kv_lookup hit;
        const uint32_t flags = KV_LOOKUP_PIN | (state ? KV_LOOKUP_REQUIRE_STATE : 0u);
        kv_status st = kv_index_lookup(index_, h.salt, tokens_.data(), h.n_tokens, flags, slots_.data(), &hit);
        if (st != KV_OK)
            return complete(st);
        st = hit.hit_tokens ? kv_load(&cache, table_, hit.hit_tokens, pool_, slots_.data(), stream_) : KV_OK;
        // Aligned recovery: the snapshot at the hit's boundary (the pinned last hit chunk keeps it).
        if (st == KV_OK && state && hit.hit_chunks > 0)
            st = kv_load_state(state, &h.page, 1, pool_, &hit.state_slot, stream_);
        st = complete(st);
        const kv_status unpin = kv_index_unpin(index_, slots_.data(), hit.hit_chunks);
        if (st != KV_OK)
            return st;
        if (unpin != KV_OK)
            return unpin;
        *hit_tokens = hit.hit_tokens;
        return KV_OK;
    }

    kv_pool *pool_;
    kv_index *index_;
    int fd_;
    hipStream_t stream_ = nullptr;  // the pool's tier stream and table, set for each request
    int32_t *table_ = nullptr;
    struct Mapping {
        void *base;
        int64_t bytes;
    };
    std::map<std::array<uint8_t, 64>, Mapping> opened_;
    std::vector<kv_ipc_buffer> bufs_, state_bufs_;
    std::vector<int32_t> table_host_;
    std::vector<int64_t> ids_;
    std::vector<int32_t> tokens_;
    std::vector<int64_t> slots_;
    std::vector<uint8_t> is_new_;
    std::vector<void *> layers_, state_layers_;
};

}  // namespace

namespace kvx {

kv_status tier_resources(kv_pool *pool, size_t table_bytes) {
    if (!pool->tier_stream)
        KVX_HIP(hipStreamCreateWithFlags(&pool->tier_stream, hipStreamNonBlocking));
    if (table_bytes > pool->tier_table_cap) {
        // Grow both buffers (the previous request has completed: nothing reads them).
        const size_t cap = std::max<size_t>(table_bytes, size_t{1} << 20);
        if (pool->tier_table)
            KVX_HIP(hipFree(pool->tier_table));
        if (pool->tier_table_pinned)
            KVX_HIP(hipHostFree(pool->tier_table_pinned));
        pool->tier_table = nullptr;
        pool->tier_table_pinned = nullptr;
        pool->tier_table_cap = 0;
        KVX_HIP(hipMalloc(reinterpret_cast<void **>(&pool->tier_table), cap));
        KVX_HIP(hipHostMalloc(reinterpret_cast<void **>(&pool->tier_table_pinned), cap, hipHostMallocDefault));
        pool->tier_table_cap = cap;
    }
    return KV_OK;
}

}  // namespace kvx

namespace {

kv_status send_request(uint32_t op, int fd, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                       const int64_t *chunk_ids, uint64_t salt, const int32_t *tokens, const kv_state *state,
                       int64_t state_page, void *stream, int64_t *value, int64_t *value2) {
    if (!cache)
        return kvx::fail(KV_EINVAL, "cache must not be NULL");
    kv_status st = kvx::check_layout(cache->layout);
    if (st != KV_OK)
        return st;
    if (n_tokens < 0)
        return kvx::fail(KV_EINVAL, "n_tokens must be >= 0 (got %lld)", static_cast<long long>(n_tokens));
    const bool prefix = op == kOpStorePrefix || op == kOpLoadPrefix;
    if (n_tokens == 0)
        return KV_OK;
    if (!block_table || !cache->layer_ptrs || (prefix ? !tokens : !chunk_ids))
        return kvx::fail(KV_EINVAL, "block_table, layer_ptrs and %s must not be NULL for n_tokens > 0",
                         prefix ? "tokens" : "chunk_ids");
    const int32_t L = cache->layout.num_layers;
    if (L > kMaxLayers)
        return kvx::fail(KV_EUNSUPPORTED, "more than %d layers", kMaxLayers);
    if (state && (state->num_layers < 1 || state->num_layers > kvx::kMaxStateLayers || !state->layer_ptrs ||
                  state_page < 0 || state_page >= state->num_pages))
        return kvx::fail(KV_EINVAL, "state needs 1..%d layers, layer pointers and a page in [0, num_pages)",
                         kvx::kMaxStateLayers);

    // Host-side completion of everything enqueued before the call (Sec. 3.2).
    KVX_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));

    RequestHeader h;
    std::memset(&h, 0, sizeof(h));
    h.magic = kMagic;
    h.op = op;
    h.layout = cache->layout;
    h.num_blocks = cache->num_blocks;
    h.block_order = cache->block_order;
    h.num_layers = L;
    h.block_stride_bytes = cache->block_stride_bytes;
    h.n_tokens = n_tokens;
    h.n_table = ceil_div(n_tokens, cache->layout.block_size);
    h.n_chunks = prefix ? 0 : ceil_div(n_tokens, cache->layout.chunk_tokens);
    h.n_ids = prefix ? n_tokens : 0;
    h.salt = salt;
    const int32_t G = state ? state->num_layers : 0;
    if (state) {
        h.state_layers = G;
        h.page_bytes = state->page_bytes;
        h.page_stride = state->page_stride;
        h.num_pages = state->num_pages;
        h.page = state_page;
    }
    std::vector<kv_ipc_buffer> bufs(static_cast<size_t>(L + G));
    for (int32_t l = 0; l < L + G; ++l) {
        const void *ptr = l < L ? cache->layer_ptrs[l] : state->layer_ptrs[l - L];
        st = kv_ipc_export(ptr, &bufs[static_cast<size_t>(l)]);
        if (st != KV_OK)
            return st;
    }
    if (!write_full(fd, &h, sizeof(h)) || !write_full(fd, bufs.data(), bufs.size() * sizeof(kv_ipc_buffer)) ||
        !write_full(fd, block_table, static_cast<size_t>(h.n_table) * sizeof(int32_t)) ||
        (h.n_chunks && !write_full(fd, chunk_ids, static_cast<size_t>(h.n_chunks) * sizeof(int64_t))) ||
        (h.n_ids && !write_full(fd, tokens, static_cast<size_t>(h.n_ids) * sizeof(int32_t))))
        return kvx::fail(KV_EINVAL, "tier connection failed while sending (%s)", std::strerror(errno));
    ReplyHeader r;
    if (!read_full(fd, &r, sizeof(r)) || r.magic != kMagic || r.msg_len > (1u << 20))
        return kvx::fail(KV_EINVAL, "tier connection failed while waiting for the reply");
    std::string msg(r.msg_len, '\0');
    if (r.msg_len && !read_full(fd, &msg[0], r.msg_len))
        return kvx::fail(KV_EINVAL, "tier connection failed while reading the reply");
    if (r.status != KV_OK) {
        kvx::set_last_error("tier: " + msg);
        return r.status;
    }
    if (value)
        *value = r.value;
    if (value2)
        *value2 = r.value2;
    return KV_OK;
}

// The host-only check behind kv_ipc_check.
kv_status check_ipc_buffer(const kv_ipc_buffer *buf, int64_t need) {
    if (!buf)
        return kvx::fail(KV_EINVAL, "IPC buffer must not be NULL");
    if (buf->allocation_bytes <= 0)
        return kvx::fail(KV_EINVAL, "IPC buffer declares an allocation of %lld bytes",
                         static_cast<long long>(buf->allocation_bytes));
    if (buf->allocation_bytes >= KV_IPC_MAX_ALLOCATION_BYTES)
        return kvx::fail(KV_EUNSUPPORTED,
                         "IPC buffer declares an allocation of %lld bytes; shared allocations must be under %lld",
                         static_cast<long long>(buf->allocation_bytes),
                         static_cast<long long>(KV_IPC_MAX_ALLOCATION_BYTES));
    if (buf->offset < 0 || need < 0 || need > buf->allocation_bytes || buf->offset > buf->allocation_bytes - need)
        return kvx::fail(KV_EINVAL, "IPC buffer range (offset %lld, %lld bytes) exceeds its declared allocation of %lld",
                         static_cast<long long>(buf->offset), static_cast<long long>(need),
                         static_cast<long long>(buf->allocation_bytes));
    return KV_OK;
}

}  // namespace

extern "C" {

kv_status kv_ipc_check(const kv_ipc_buffer *buf, int64_t need) {
    return kvx::guarded([&]() -> kv_status { return check_ipc_buffer(buf, need); });
}


kv_status kv_ipc_export(const void *dev_ptr, kv_ipc_buffer *out) {
    return kvx::guarded([&]() -> kv_status {
        if (!dev_ptr || !out)
            return kvx::fail(KV_EINVAL, "dev_ptr and out must not be NULL");
        void *base = nullptr;
        size_t size = 0;
        KVX_HIP(hipMemGetAddressRange(&base, &size, const_cast<void *>(dev_ptr)));
        if (static_cast<int64_t>(size) >= KV_IPC_MAX_ALLOCATION_BYTES)
            return kvx::fail(KV_EUNSUPPORTED,
                             "allocation of %zu bytes is too large to share between processes (limit %lld); allocate "
                             "each shared buffer separately",
                             size, static_cast<long long>(KV_IPC_MAX_ALLOCATION_BYTES));
        hipIpcMemHandle_t handle;
        KVX_HIP(hipIpcGetMemHandle(&handle, base));
        static_assert(sizeof(handle) == sizeof(out->handle), "IPC handle size");
        std::memcpy(out->handle, &handle, sizeof(handle));
        out->offset = static_cast<const uint8_t *>(dev_ptr) - static_cast<uint8_t *>(base);
        out->allocation_bytes = static_cast<int64_t>(size);
        return KV_OK;
    });
}

kv_status kv_tier_serve(kv_pool *pool, kv_index *index, int fd) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool || fd < 0)
            return kvx::fail(KV_EINVAL, "pool must not be NULL and fd must be a connected socket");
        Connection c(pool, index, fd);
        return c.serve();
    });
}

kv_status kv_tier_listen(const char *path, int *listen_fd) {
    return kvx::guarded([&]() -> kv_status {
        if (!path || !listen_fd)
            return kvx::fail(KV_EINVAL, "path and listen_fd must not be NULL");
        sockaddr_un addr;
        std::memset(&addr, 0, sizeof(addr));
        addr.sun_family = AF_UNIX;
        if (std::strlen(path) >= sizeof(addr.sun_path))
            return kvx::fail(KV_EINVAL, "socket path longer than %zu bytes", sizeof(addr.sun_path) - 1);
        std::strncpy(addr.sun_path, path, sizeof(addr.sun_path) - 1);
        const int fd = socket(AF_UNIX, SOCK_STREAM, 0);
        if (fd < 0)
            return kvx::fail(KV_EINVAL, "socket: %s", std::strerror(errno));
        if (bind(fd, reinterpret_cast<sockaddr *>(&addr), sizeof(addr)) != 0 || listen(fd, 64) != 0) {
            const int err = errno;
            close(fd);
            return kvx::fail(KV_EINVAL, "cannot listen at %s: %s", path, std::strerror(err));
        }
        *listen_fd = fd;
        return KV_OK;
    });
}

kv_status kv_tier_run(kv_pool *pool, kv_index *index, int listen_fd, int32_t connections) {
    return kvx::guarded([&]() -> kv_status {
        if (!pool || listen_fd < 0 || connections < 0)
            return kvx::fail(KV_EINVAL, "pool must not be NULL, listen_fd a listening socket, connections >= 0");
        struct Result {
            kv_status status = KV_OK;
            std::string message;
        };
        // The tier stream and table buffers before the first connection, with one small copy on the
        // stream: otherwise the first request pays for making them (tens of ms measured).
        {
            int prev = -1;
            KVX_HIP(hipGetDevice(&prev));
            KVX_HIP(hipSetDevice(pool->device));
            kv_status st;
            {
                std::lock_guard<std::mutex> lock(pool->tier_mu);
                st = kvx::tier_resources(pool, sizeof(int32_t));
                hipError_t e = hipSuccess;
                if (st == KV_OK)
                    e = hipMemcpyAsync(pool->tier_table, pool->tier_table_pinned, sizeof(int32_t),
                                       hipMemcpyHostToDevice, pool->tier_stream);
                if (st == KV_OK && e == hipSuccess)
                    e = hipStreamSynchronize(pool->tier_stream);
                if (st == KV_OK && e != hipSuccess)
                    st = kvx::hip_fail(e, "tier warm-up copy", __FILE__, __LINE__);
            }
            const hipError_t e = hipSetDevice(prev);  // the caller's device, whatever happened above
            if (st != KV_OK)
                return st;
            if (e != hipSuccess)
                return kvx::hip_fail(e, "hipSetDevice(caller's device)", __FILE__, __LINE__);
        }
        std::deque<Result> results;  // push_back keeps references to earlier elements valid
        std::vector<std::thread> threads;
        kv_status accept_error = KV_OK;
        std::string accept_message;
        for (int32_t k = 0; connections == 0 || k < connections;) {
            const int fd = accept(listen_fd, nullptr, nullptr);
            if (fd < 0) {
                if (errno == EINTR)
                    continue;
                accept_error = KV_EINVAL;
                accept_message = std::string("accept: ") + std::strerror(errno);
                break;
            }
            ++k;
            try {
                results.emplace_back();
                Result *r = &results.back();
                threads.emplace_back([pool, index, fd, r] {
                    r->status = kv_tier_serve(pool, index, fd);
                    if (r->status != KV_OK) {
                        try {
                            r->message = kv_last_error();
                        } catch (...) {
                        }
                    }
                    close(fd);
                });
            } catch (const std::exception &e) {
                // No thread took this connection: refuse it, stop accepting, and still join the
                // threads already serving (a joinable thread must never be destroyed).
                close(fd);
                accept_error = KV_ENOMEM;
                accept_message = std::string("cannot serve another connection: ") + e.what();
                break;
            }
        }
        for (std::thread &t : threads)
            t.join();
        for (const Result &r : results)
            if (r.status != KV_OK) {
                kvx::set_last_error(r.message);
                return r.status;
            }
        if (accept_error != KV_OK)
            return kvx::fail(accept_error, "%s", accept_message.c_str());
        return KV_OK;
    });
}

kv_status kv_tier_store(int fd, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                        const int64_t *chunk_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return send_request(kOpStore, fd, cache, block_table, n_tokens, chunk_ids, 0, nullptr, nullptr, 0, stream,
                            nullptr, nullptr);
    });
}

kv_status kv_tier_load(int fd, const kv_cache *cache, const int32_t *block_table, int64_t n_tokens,
                       const int64_t *chunk_ids, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        return send_request(kOpLoad, fd, cache, block_table, n_tokens, chunk_ids, 0, nullptr, nullptr, 0, stream,
                            nullptr, nullptr);
    });
}

kv_status kv_tier_store_prefix(int fd, const kv_cache *cache, const int32_t *block_table, const kv_state *state,
                               int64_t state_page, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                               int64_t *stored_chunks, int32_t *stored_state, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        int64_t v = 0, v2 = 0;
        const kv_status st = send_request(kOpStorePrefix, fd, cache, block_table, n_tokens, nullptr, salt, tokens,
                                          state, state_page, stream, &v, &v2);
        if (stored_chunks)
            *stored_chunks = st == KV_OK ? v : 0;
        if (stored_state)
            *stored_state = st == KV_OK ? static_cast<int32_t>(v2) : 0;
        return st;
    });
}

kv_status kv_tier_load_prefix(int fd, const kv_cache *cache, const int32_t *block_table, const kv_state *state,
                              int64_t state_page, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                              int64_t *hit_tokens, void *stream) {
    return kvx::guarded([&]() -> kv_status {
        int64_t v = 0;
        const kv_status st = send_request(kOpLoadPrefix, fd, cache, block_table, n_tokens, nullptr, salt, tokens, state,
                                          state_page, stream, &v, nullptr);
        if (hit_tokens)
            *hit_tokens = st == KV_OK ? v : 0;
        return st;
    });
}

}  // extern "C"

// Pool index: prefix-keyed chunk slots with LRU eviction, whole-chunk hits, aligned
// recovery and two-phase stores, over the slots of a kv_pool.  Host only: no HIP call.
//
// The shared tier of the paper keeps a fixed RAM budget of chunks with LRU eviction
// (Table 1); a chunk is reused only as a whole (Sec. 3.1-3.2), and a hybrid prefix is
// restorable only with the recurrent snapshot at its boundary (Sec. 2.2).  The rules where
// the paper is silent are stated in kvx.h and are the same as the oracle's model.
#include <cstring>
#include <memory>
#include <mutex>
#include <set>
#include <unordered_map>
#include <vector>

#include "kvx_internal.h"

namespace {

struct Key {
    uint64_t a, b;
    bool operator==(const Key &o) const { return a == o.a && b == o.b; }
};

struct KeyHash {
    size_t operator()(const Key &k) const { return static_cast<size_t>(k.a ^ (k.b >> 7)); }
};

// Finaliser of SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014): a bijective 64-bit avalanche.
inline uint64_t avalanche(uint64_t x) {
    x ^= x >> 30;
    x *= 0xBF58476D1CE4E5B9ull;
    x ^= x >> 27;
    x *= 0x94D049BB133111EBull;
    x ^= x >> 31;
    return x;
}

inline uint64_t rotl(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }

// Chained chunk keys.  Two 64-bit lanes start from the salt and the chunk length and absorb
// every token in order with an odd-multiply/rotate round (a bijection of the lane for each
// token); the key of chunk i is the avalanched lane pair after token (i+1)*C - 1, so it
// names the salt and the whole prefix the chunk completes.
class KeyChain {
  public:
    KeyChain(uint64_t salt, int32_t C)
        : a_(avalanche(salt ^ 0x6A09E667F3BCC909ull) ^ static_cast<uint32_t>(C)),
          b_(avalanche(~salt ^ 0xBB67AE8584CAA73Bull) + static_cast<uint32_t>(C)) {}

    void absorb(const int32_t *t, int64_t n) {
        for (int64_t i = 0; i < n; ++i) {
            const uint64_t w = static_cast<uint32_t>(t[i]);
            a_ = rotl(a_ ^ (w * 0x9E3779B97F4A7C15ull), 29) * 0xD6E8FEB86659FD93ull;
            b_ = rotl(b_ + (w * 0xC2B2AE3D27D4EB4Full), 31) * 0xFF51AFD7ED558CCDull;
        }
    }

    Key key() const { return {avalanche(a_), avalanche(b_ ^ 0x510E527FADE682D1ull)}; }

  private:
    uint64_t a_, b_;
};

// Intrusive least-recently-used list over node indices (head = least recent).
template <class Node>
struct Lru {
    int64_t head = -1, tail = -1;

    void push_back(std::vector<Node> &v, int64_t s) {
        v[s].prev = tail;
        v[s].next = -1;
        if (tail >= 0)
            v[tail].next = s;
        else
            head = s;
        tail = s;
        v[s].in_lru = true;
    }
    void remove(std::vector<Node> &v, int64_t s) {
        if (v[s].prev >= 0)
            v[v[s].prev].next = v[s].next;
        else
            head = v[s].next;
        if (v[s].next >= 0)
            v[v[s].next].prev = v[s].prev;
        else
            tail = v[s].prev;
        v[s].prev = v[s].next = -1;
        v[s].in_lru = false;
    }
    void touch(std::vector<Node> &v, int64_t s) {
        if (v[s].in_lru) {
            remove(v, s);
            push_back(v, s);
        }
    }
};

struct Entry {
    Key key{};
    int64_t state = -1;  // snapshot slot of the boundary after this chunk
    int64_t prev = -1, next = -1;
    int32_t pins = 0;
    bool used = false, pending = false, aborted = false, state_pending = false, in_lru = false;
};

struct StateEntry {
    int64_t owner = -1;  // chunk slot the snapshot belongs to
    int64_t prev = -1, next = -1;
    bool in_lru = false;
};

}  // namespace

struct kv_index {
    int32_t C = 0;
    int64_t num_slots = 0, num_state_slots = 0;
    std::vector<Entry> e;
    std::vector<StateEntry> se;
    std::unordered_map<Key, int64_t, KeyHash> by_key;
    std::set<int64_t> free_slots, free_state;
    Lru<Entry> lru;
    Lru<StateEntry> slru;
    int64_t evictions = 0, state_evictions = 0;
    std::mutex mu;

    void free_state_of(int64_t s) {
        Entry &x = e[s];
        if (x.state < 0)
            return;
        const int64_t ss = x.state;
        if (se[ss].in_lru)
            slru.remove(se, ss);
        se[ss].owner = -1;
        free_state.insert(ss);
        x.state = -1;
        x.state_pending = false;
    }

    void drop(int64_t s) {
        free_state_of(s);
        auto it = by_key.find(e[s].key);
        if (it != by_key.end() && it->second == s)
            by_key.erase(it);
        if (e[s].in_lru)
            lru.remove(e, s);
        e[s] = Entry{};
        free_slots.insert(s);
    }

    void release(int64_t s) {
        e[s].pins -= 1;
        if (e[s].aborted && e[s].pins == 0)
            drop(s);
    }

    bool evict_one() {
        for (int64_t s = lru.head; s >= 0; s = e[s].next)
            if (e[s].pins == 0) {
                drop(s);
                ++evictions;
                return true;
            }
        return false;
    }

    int64_t alloc() {
        if (free_slots.empty() && !evict_one())
            return -1;
        const int64_t s = *free_slots.begin();
        free_slots.erase(free_slots.begin());
        return s;
    }

    int64_t alloc_state() {
        if (free_state.empty()) {
            for (int64_t ss = slru.head; ss >= 0; ss = se[ss].next) {
                const int64_t owner = se[ss].owner;
                if (e[owner].pins == 0 && !e[owner].pending) {
                    free_state_of(owner);
                    ++state_evictions;
                    break;
                }
            }
            if (free_state.empty())
                return -1;
        }
        const int64_t ss = *free_state.begin();
        free_state.erase(free_state.begin());
        return ss;
    }

    // Touch a prefix's chunks from last to first (the head ends most recent).
    void touch_prefix(const int64_t *slots, int64_t n) {
        for (int64_t j = n - 1; j >= 0; --j)
            lru.touch(e, slots[j]);
    }

    bool valid_slot(int64_t s) const { return s >= 0 && s < num_slots && e[s].used; }

    // Every listed slot is used and pinned at least as often as it is listed.
    bool pins_cover(const int64_t *slots, int64_t n) const {
        std::unordered_map<int64_t, int32_t> count;
        for (int64_t i = 0; i < n; ++i) {
            if (!valid_slot(slots[i]))
                return false;
            if (++count[slots[i]] > e[slots[i]].pins)
                return false;
        }
        return true;
    }
};

namespace kvx {

int32_t index_chunk_tokens(const kv_index *index) { return index->C; }
int64_t index_num_slots(const kv_index *index) { return index->num_slots; }
int64_t index_num_state_slots(const kv_index *index) { return index->num_state_slots; }

}  // namespace kvx

namespace {

kv_status check_tokens(const kv_index *x, const int32_t *tokens, int64_t n_tokens) {
    if (!x)
        return kvx::fail(KV_EINVAL, "index must not be NULL");
    if (n_tokens < 0)
        return kvx::fail(KV_EINVAL, "n_tokens must be >= 0 (got %lld)", static_cast<long long>(n_tokens));
    if (n_tokens >= x->C && !tokens)
        return kvx::fail(KV_EINVAL, "tokens must not be NULL");
    return KV_OK;
}

}  // namespace

extern "C" {

kv_status kv_index_create(int32_t chunk_tokens, int64_t num_slots, int64_t num_state_slots, kv_index **out) {
    return kvx::guarded([&]() -> kv_status {
        if (!out)
            return kvx::fail(KV_EINVAL, "out must not be NULL");
        *out = nullptr;
        if (chunk_tokens < 1 || num_slots < 1 || num_state_slots < 0)
            return kvx::fail(KV_EINVAL,
                             "need chunk_tokens >= 1, num_slots >= 1, num_state_slots >= 0 (got %d, %lld, %lld)",
                             chunk_tokens, static_cast<long long>(num_slots), static_cast<long long>(num_state_slots));
        std::unique_ptr<kv_index> x(new kv_index());  // freed if a container below throws
        x->C = chunk_tokens;
        x->num_slots = num_slots;
        x->num_state_slots = num_state_slots;
        x->e.resize(static_cast<size_t>(num_slots));
        x->se.resize(static_cast<size_t>(num_state_slots));
        for (int64_t s = 0; s < num_slots; ++s)
            x->free_slots.insert(x->free_slots.end(), s);
        for (int64_t s = 0; s < num_state_slots; ++s)
            x->free_state.insert(x->free_state.end(), s);
        x->by_key.reserve(static_cast<size_t>(num_slots) * 2);
        *out = x.release();
        return KV_OK;
    });
}

kv_status kv_index_destroy(kv_index *index) {
    return kvx::guarded([&]() -> kv_status {
        delete index;
        return KV_OK;
    });
}

kv_status kv_index_keys(const kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens,
                        uint64_t *keys) {
    return kvx::guarded([&]() -> kv_status {
        kv_status st = check_tokens(index, tokens, n_tokens);
        if (st != KV_OK)
            return st;
        const int64_t nfull = n_tokens / index->C;
        if (nfull > 0 && !keys)
            return kvx::fail(KV_EINVAL, "keys must not be NULL");
        KeyChain kc(salt, index->C);
        for (int64_t i = 0; i < nfull; ++i) {
            kc.absorb(tokens + i * index->C, index->C);
            const Key k = kc.key();
            keys[2 * i] = k.a;
            keys[2 * i + 1] = k.b;
        }
        return KV_OK;
    });
}

kv_status kv_index_lookup(kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens, uint32_t flags,
                          int64_t *slots, kv_lookup *out) {
    return kvx::guarded([&]() -> kv_status {
        kv_status st = check_tokens(index, tokens, n_tokens);
        if (st != KV_OK)
            return st;
        if (!out)
            return kvx::fail(KV_EINVAL, "out must not be NULL");
        if (flags & ~(KV_LOOKUP_REQUIRE_STATE | KV_LOOKUP_PIN))
            return kvx::fail(KV_EINVAL, "unknown lookup flags 0x%x", flags);
        kv_index &x = *index;
        std::lock_guard<std::mutex> lock(x.mu);
        const int64_t nfull = n_tokens / x.C;
        if (nfull > 0 && !slots)
            return kvx::fail(KV_EINVAL, "slots must not be NULL");
        KeyChain kc(salt, x.C);
        int64_t kv = 0;
        for (; kv < nfull; ++kv) {
            kc.absorb(tokens + kv * x.C, x.C);
            auto it = x.by_key.find(kc.key());
            if (it == x.by_key.end() || x.e[it->second].pending)
                break;
            slots[kv] = it->second;
        }
        auto has_state = [&](int64_t s) { return x.e[s].state >= 0 && !x.e[s].state_pending; };
        int64_t hit = kv;
        if (flags & KV_LOOKUP_REQUIRE_STATE)
            while (hit > 0 && !has_state(slots[hit - 1]))
                --hit;
        int64_t state_slot = -1;
        if (hit > 0 && has_state(slots[hit - 1])) {
            state_slot = x.e[slots[hit - 1]].state;
            x.slru.touch(x.se, state_slot);
        }
        x.touch_prefix(slots, hit);
        if (flags & KV_LOOKUP_PIN)
            for (int64_t j = 0; j < hit; ++j)
                x.e[slots[j]].pins += 1;
        out->kv_chunks = kv;
        out->hit_chunks = hit;
        out->hit_tokens = hit * x.C;
        out->state_slot = state_slot;
        return KV_OK;
    });
}

kv_status kv_index_unpin(kv_index *index, const int64_t *slots, int64_t n) {
    return kvx::guarded([&]() -> kv_status {
        if (!index || n < 0 || (n > 0 && !slots))
            return kvx::fail(KV_EINVAL, "index and slots must not be NULL, n >= 0");
        std::lock_guard<std::mutex> lock(index->mu);
        if (!index->pins_cover(slots, n))
            return kvx::fail(KV_EINVAL, "a listed slot is not pinned (that often)");
        for (int64_t i = 0; i < n; ++i)
            index->release(slots[i]);
        return KV_OK;
    });
}

kv_status kv_index_reserve(kv_index *index, uint64_t salt, const int32_t *tokens, int64_t n_tokens, int64_t *slots,
                           uint8_t *is_new, int64_t *n_chunks) {
    return kvx::guarded([&]() -> kv_status {
        kv_status st = check_tokens(index, tokens, n_tokens);
        if (st != KV_OK)
            return st;
        kv_index &x = *index;
        const int64_t nfull = n_tokens / x.C;
        if (!n_chunks || (nfull > 0 && (!slots || !is_new)))
            return kvx::fail(KV_EINVAL, "slots, is_new and n_chunks must not be NULL");
        std::lock_guard<std::mutex> lock(x.mu);
        *n_chunks = nfull;
        KeyChain kc(salt, x.C);
        for (int64_t i = 0; i < nfull; ++i) {
            kc.absorb(tokens + i * x.C, x.C);
            const Key key = kc.key();
            auto it = x.by_key.find(key);
            if (it != x.by_key.end()) {
                x.e[it->second].pins += 1;
                slots[i] = it->second;
                is_new[i] = 0;
                continue;
            }
            const int64_t s = x.alloc();
            if (s < 0) {
                for (int64_t j = 0; j < i; ++j) {  // undo this call; evictions stand
                    if (is_new[j])
                        x.drop(slots[j]);
                    else
                        x.release(slots[j]);
                }
                *n_chunks = 0;
                return kvx::fail(KV_EBUSY, "no slot can be freed for chunk %lld: all %lld slots are pinned or pending",
                                 static_cast<long long>(i), static_cast<long long>(x.num_slots));
            }
            Entry &en = x.e[s];
            en = Entry{};
            en.key = key;
            en.used = true;
            en.pending = true;
            en.pins = 1;
            x.by_key.emplace(key, s);
            slots[i] = s;
            is_new[i] = 1;
        }
        return KV_OK;
    });
}

kv_status kv_index_commit(kv_index *index, const int64_t *slots, const uint8_t *is_new, int64_t n, int ok) {
    return kvx::guarded([&]() -> kv_status {
        if (!index || n < 0 || (n > 0 && (!slots || !is_new)))
            return kvx::fail(KV_EINVAL, "index, slots and is_new must not be NULL, n >= 0");
        kv_index &x = *index;
        std::lock_guard<std::mutex> lock(x.mu);
        std::set<int64_t> seen;
        for (int64_t i = 0; i < n; ++i) {
            const int64_t s = slots[i];
            if (!x.valid_slot(s) || x.e[s].pins == 0 || !seen.insert(s).second)
                return kvx::fail(KV_EINVAL, "slot %lld is not a distinct pinned entry of this reservation",
                                 static_cast<long long>(s));
            if (is_new[i] && (!x.e[s].pending || x.e[s].aborted))
                return kvx::fail(KV_EINVAL, "slot %lld is not a pending entry", static_cast<long long>(s));
        }
        for (int64_t i = 0; i < n; ++i) {
            const int64_t s = slots[i];
            Entry &en = x.e[s];
            if (is_new[i]) {
                if (ok) {
                    en.pending = false;
                    x.lru.push_back(x.e, s);
                } else {
                    en.aborted = true;
                    x.free_state_of(s);
                    auto it = x.by_key.find(en.key);
                    if (it != x.by_key.end() && it->second == s)
                        x.by_key.erase(it);
                }
            }
            x.release(s);
        }
        std::vector<int64_t> live;
        live.reserve(static_cast<size_t>(n));
        for (int64_t i = 0; i < n; ++i)
            if (x.e[slots[i]].used && !x.e[slots[i]].pending)
                live.push_back(slots[i]);
        x.touch_prefix(live.data(), static_cast<int64_t>(live.size()));
        return KV_OK;
    });
}

kv_status kv_index_reserve_state(kv_index *index, int64_t slot, int64_t *state_slot, int32_t *is_new) {
    return kvx::guarded([&]() -> kv_status {
        if (!index || !state_slot || !is_new)
            return kvx::fail(KV_EINVAL, "index, state_slot and is_new must not be NULL");
        kv_index &x = *index;
        std::lock_guard<std::mutex> lock(x.mu);
        if (!x.valid_slot(slot) || x.e[slot].pins == 0 || x.e[slot].aborted)
            return kvx::fail(KV_EINVAL, "slot %lld is not a pinned entry", static_cast<long long>(slot));
        Entry &en = x.e[slot];
        if (en.state >= 0) {
            *state_slot = en.state;
            *is_new = 0;
            return KV_OK;
        }
        const int64_t ss = x.alloc_state();
        if (ss < 0)
            return kvx::fail(KV_EBUSY, "no snapshot slot can be freed");
        en.state = ss;
        en.state_pending = true;
        x.se[ss].owner = slot;
        *state_slot = ss;
        *is_new = 1;
        return KV_OK;
    });
}

kv_status kv_index_commit_state(kv_index *index, int64_t slot, int ok) {
    return kvx::guarded([&]() -> kv_status {
        if (!index)
            return kvx::fail(KV_EINVAL, "index must not be NULL");
        kv_index &x = *index;
        std::lock_guard<std::mutex> lock(x.mu);
        if (!x.valid_slot(slot) || x.e[slot].state < 0 || !x.e[slot].state_pending)
            return kvx::fail(KV_EINVAL, "slot %lld has no pending snapshot", static_cast<long long>(slot));
        Entry &en = x.e[slot];
        if (ok) {
            en.state_pending = false;
            x.slru.push_back(x.se, en.state);
        } else {
            x.se[en.state].owner = -1;
            x.free_state.insert(en.state);
            en.state = -1;
            en.state_pending = false;
        }
        return KV_OK;
    });
}

kv_status kv_index_get_stats(kv_index *index, kv_index_stats *out) {
    return kvx::guarded([&]() -> kv_status {
        if (!index || !out)
            return kvx::fail(KV_EINVAL, "index and out must not be NULL");
        kv_index &x = *index;
        std::lock_guard<std::mutex> lock(x.mu);
        std::memset(out, 0, sizeof(*out));
        for (const Entry &en : x.e) {
            if (!en.used)
                continue;
            if (!en.pending)
                out->entries += 1;
            else if (!en.aborted)
                out->pending += 1;
        }
        for (const StateEntry &s : x.se)
            out->state_entries += s.in_lru ? 1 : 0;
        out->free_slots = static_cast<int64_t>(x.free_slots.size());
        out->free_state_slots = static_cast<int64_t>(x.free_state.size());
        out->evictions = x.evictions;
        out->state_evictions = x.state_evictions;
        return KV_OK;
    });
}

}  // extern "C"

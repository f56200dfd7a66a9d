// Pack (store) and unpack (load) kernels for gfx950.
//
// A workgroup moves one slab at a time: the (layer l, K/V, block j) piece of chunk i, i.e. the
// bs <= BS tokens of one paged block for one layer and one of K/V.  On the cache side the
// slab is the contiguous [H][BS][D] region of that block (HND, the paper's replica layout,
// Table 1); on the chunk side it is the contiguous [bs][H][D] run of token-major rows
// inside plane (l, kv) of the chunk.  The slab is therefore contiguous on both sides and
// differs only by a permutation of D*E-byte rows: cache row (h, s) <-> chunk row (s, h).
//
// Token-major (NHD) cache blocks hold the slab's rows already in chunk order: the slab
// is then a straight contiguous copy.  For HND blocks, lanes walk the chunk side in order
// in both directions: the pool/staging side (host memory over PCIe in zero-copy mode) is
// read or written in contiguous 1 KiB-per-wave runs, and the cache side in whole-row runs
// (256 bytes at D*E = 256) spread over the slab's H head regions.  Measured on MI355X with
// both orders running on the same cache allocations, this order is 3-4% faster for unpack
// than walking the cache side (whose writes are then contiguous) on every allocation, and
// 1-2% faster for pack.  Rows are >= 16 bytes and moved as 16-byte vectors, so no LDS
// transpose is needed for coalescing (staging through LDS was measured slower).
// Values are moved as integers only: no float register ever holds them (NaN payloads, -0
// and subnormals survive).
//
// Index math is one division at thread start; afterwards every step is an addition with
// carry.  Streaming data is read and written nontemporally.  Device-side (staged) launches
// run one workgroup per slab and cap residency at 5 workgroups per CU (KVX_LDS_RESERVE).
// Host-side (zero-copy) launches run a few dozen workgroups that stride over the slabs
// (KVX_HOST_WGS_*): the link bounds them, and the rest of the chip stays free.
#include <algorithm>

#include "kvx_internal.h"

namespace kvx {

namespace {

// One 16-byte vector as a native 128-bit register tuple (kept in VGPRs; never a float).
typedef uint32_t vec16 __attribute__((ext_vector_type(4)));

// Compile-time tuning knobs: vectors each thread loads before storing (a full tile of
// kThreads*U vectors; 1 measured best) and streaming (nontemporal) access on the read and
// write side.
#ifndef KVX_UNROLL
#define KVX_UNROLL 1
#endif
#ifndef KVX_NT_LOAD
#define KVX_NT_LOAD 1
#endif
#ifndef KVX_NT_STORE
#define KVX_NT_STORE 1
#endif
// Dynamic LDS reserved per workgroup to cap the workgroups resident per CU (only the unpack of
// token-major slabs uses it, as a slab buffer):
// 32 KiB of the CU's 160 KiB allows 5 (20 waves per CU).  Measured on MI355X with the
// 27B-class layout, variants alternating on the same cache allocations in one process: 5
// resident workgroups moved 4.2-4.6% more than 4 on two machines and the same on two others,
// while 6, 7 and 8 lose on unpack (-2% to -5% against 4), as does an uncapped launch: fewer
// concurrent 32 KiB streams per CU keep the HBM read/write mix efficient, too few leave HBM idle.
#ifndef KVX_LDS_RESERVE
#define KVX_LDS_RESERVE 32768
#endif
// Workgroups of a host-side (zero-copy) pack / unpack launch; each strides over the
// launch's slabs (0: one workgroup per slab).  Measured on MI355X at the 27B-class layout
// (one workgroup per slab: store 54.5, load 55.9 GB/s): 64 for pack gives 55.9 GB/s (16:
// 49.8, 256: 54.7); 32 for unpack gives 57.0 GB/s (16: 44, 64 to 256: 57.5) and, with
// a staged store running at the same time, lets both directions share the link.
#ifndef KVX_HOST_WGS_PACK
#define KVX_HOST_WGS_PACK 64
#endif
#ifndef KVX_HOST_WGS_UNPACK
#define KVX_HOST_WGS_UNPACK 32
#endif

__device__ __forceinline__ vec16 load16(const vec16 *p) {
#if KVX_NT_LOAD
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}

__device__ __forceinline__ void store16(vec16 *p, vec16 v) {
#if KVX_NT_STORE
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

// Cache-side stores of unpack go through a buffer resource spanning the slab, with cache
// policy "nt sc1" (nontemporal, agent scope).  Paired on six destination allocations of the
// 27B-class layout, this moved 0.1-2.3% more than plain nontemporal stores on every one of
// them (about 1% on average); "sc1" without "nt" varied by allocation, stores without either
// lost 2-7%, and pack's stores and either kernel's loads gained nothing from other policies.
constexpr int kCachePolicyNtSc1 = 2 | 16;  // CDNA3/4 cache-policy bits: NT = 2, SC1 = 16
constexpr int kRawBufferFlags = 0x00020000;  // descriptor word 3 of a raw (untyped) buffer

__device__ __forceinline__ __amdgpu_buffer_rsrc_t slab_buffer(uint8_t *slab, int64_t bytes) {
    // bytes < 2^31: validation caps a block at 2 GiB, so a K or V slab at 1 GiB.
    return __builtin_amdgcn_make_buffer_rsrc(slab, 0, static_cast<int>(bytes), kRawBufferFlags);
}

__device__ __forceinline__ void store16_cache(__amdgpu_buffer_rsrc_t slab, int vec, vec16 v) {
    __builtin_amdgcn_raw_buffer_store_b128(v, slab, vec * 16, 0, kCachePolicyNtSc1);
}

// Chunk-side stores of pack.  Into mapped pinned host memory (zero-copy) they take the same
// "nt sc1" policy, which moved 57.1 GB/s over the link against 55.7-55.9 with plain nontemporal
// stores (56.8 without either bit); into device staging plain nontemporal stores measured the same
// as any policy.
template <bool HOST_SIDE>
__device__ __forceinline__ void store16_chunk(vec16 *base, __amdgpu_buffer_rsrc_t slab, int vec, vec16 v) {
    if constexpr (HOST_SIDE)
        __builtin_amdgcn_raw_buffer_store_b128(v, slab, vec * 16, 0, kCachePolicyNtSc1);
    else
        store16(base + vec, v);
}

// Walks chunk-order vector indices v = t, t + kThreads, t + 2*kThreads, ... of one slab,
// maintaining (s, h, col) with v = (s*H + h)*VR + col.
struct RowWalker {
    int s, h, col;
    int VR, H;
    int dcol, ds0, dh0, ds1, dh1;  // per-step increments (without / with a column carry)

    __device__ RowWalker(int v, int vec_per_row, int heads) : VR(vec_per_row), H(heads) {
        int q = v / VR;
        col = v - q * VR;
        s = q / H;
        h = q - s * H;
        int dq = kThreads / VR;
        dcol = kThreads - dq * VR;
        ds0 = dq / H;
        dh0 = dq - ds0 * H;
        ds1 = (dq + 1) / H;
        dh1 = (dq + 1) - ds1 * H;
    }

    __device__ void advance() {
        col += dcol;
        int ds = ds0, dh = dh0;
        if (col >= VR) {
            col -= VR;
            ds = ds1;
            dh = dh1;
        }
        h += dh;
        s += ds;
        if (h >= H) {
            h -= H;
            s += 1;
        }
    }

    // 16-byte-vector offset of the current element inside the cache-side [H][BS][D] slab.
    __device__ int cache_vec(int BS) const { return (h * BS + s) * VR + col; }
};

template <int DIR, int U, bool HOST_SIDE>
__device__ __forceinline__ void move_slab(const GatherArgs &a, int c, int ll, int kv, int j);

// HOST_SIDE marks launches whose chunk side is mapped pinned host memory (zero-copy mode);
// the body is the same, the instantiation (and launch occupancy) is separate.
template <int DIR, int U, bool HOST_SIDE>
__device__ __forceinline__ void move_slab_id(const GatherArgs &a, int64_t id) {
    // Slab id -> (chunk c, layer ll, kv, block j); j varies fastest so consecutive ids
    // touch consecutive chunk-side regions.
    const int bpc = a.blocks_per_chunk;
    const int j = static_cast<int>(id % bpc);
    int64_t rest = id / bpc;
    const int kv = static_cast<int>(rest & 1);
    rest >>= 1;
    const int ll = static_cast<int>(rest % a.nlayers);
    const int c = static_cast<int>(rest / a.nlayers);
    move_slab<DIR, U, HOST_SIDE>(a, c, ll, kv, j);
}

template <int DIR, int U, bool HOST_SIDE>
__global__ __launch_bounds__(kThreads) void gather_kernel(const GatherArgs a) {
    if constexpr (HOST_SIDE) {
        // A capped grid strides over the slabs: the link, not the number of waves in flight,
        // bounds these launches, and the CUs they leave free run other streams' kernels.
        const int64_t total = static_cast<int64_t>(a.nchunks) * a.nlayers * 2 * a.blocks_per_chunk;
        for (int64_t id = blockIdx.x; id < total; id += gridDim.x)
            move_slab_id<DIR, U, HOST_SIDE>(a, id);
    } else {
        move_slab_id<DIR, U, HOST_SIDE>(a, blockIdx.x);  // one workgroup per slab
    }
}

template <int DIR, int U, bool HOST_SIDE>
__device__ __forceinline__ void move_slab(const GatherArgs &a, int c, int ll, int kv, int j) {
    const int bpc = a.blocks_per_chunk;

    const int64_t i = a.chunk0 + c;  // global chunk index
    const int64_t remaining = a.n_tokens - i * a.C;
    const int64_t r = remaining < a.C ? remaining : a.C;  // tokens in chunk i
    const int64_t tok0 = static_cast<int64_t>(j) * a.BS;  // first token of the slab in the chunk
    if (tok0 >= r)
        return;
    const int bs = static_cast<int>((r - tok0) < a.BS ? (r - tok0) : a.BS);

    const int l = a.layer0 + ll;
    const int64_t row_bytes = static_cast<int64_t>(a.vec_per_row) * 16;
    uint8_t *chunk_slab = a.chunk_base + static_cast<int64_t>(a.slot[c]) * a.slot_stride +
                          ((static_cast<int64_t>(l) * 2 + kv) * r + tok0) * a.H * row_bytes;
    vec16 *chunk_v = reinterpret_cast<vec16 *>(chunk_slab);
    const int nvec = bs * a.H * a.vec_per_row;

    const int32_t b = a.block_table[i * bpc + j];
    if (b < 0 || b >= a.num_blocks) {
        // A block id outside the cache: flag it, touch no cache byte, and on a store write
        // zeros for the slab's chunk rows so that no stale staging or pool bytes (another
        // request's state) are passed on as this chunk's contents.
        if (threadIdx.x == 0)
            __hip_atomic_store(a.err, KV_ASYNC_BAD_BLOCK, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        if (DIR == kPack) {
            const vec16 zero = {0u, 0u, 0u, 0u};
            for (int v = static_cast<int>(threadIdx.x); v < nvec; v += kThreads)
                chunk_v[v] = zero;
        }
        return;
    }

    const __amdgpu_buffer_rsrc_t chunk_buf = slab_buffer(chunk_slab, static_cast<int64_t>(nvec) * 16);
    const int64_t slab_bytes = static_cast<int64_t>(a.H) * a.BS * row_bytes;
    uint8_t *cache_slab = a.layer[ll] + static_cast<int64_t>(b) * a.block_stride + kv * slab_bytes;
    vec16 *cache_v = reinterpret_cast<vec16 *>(cache_slab);
    const __amdgpu_buffer_rsrc_t cache_buf = slab_buffer(cache_slab, slab_bytes);

    const int tid = static_cast<int>(threadIdx.x);
    if (a.nhd) {
        // Token-major block: the slab's first bs*H rows are already in chunk row order.
        if constexpr (DIR == kUnpack && !HOST_SIDE) {
            // Device-side unpack: read the whole slab contiguously into the workgroup's reserved LDS,
            // then write it with each pass spread over 8 segments of the slab (512 B each).  Paired
            // on the paper's attention layout, this moved 3.0% more than the straight copy; 4, 16 or
            // 32 segments measured the same as 8.  Host-side launches reserve no LDS.
            constexpr int kSeg = 8, kPer = kThreads / kSeg;
            if (nvec * 16 <= KVX_LDS_RESERVE && nvec % (kSeg * kPer) == 0) {
                extern __shared__ vec16 lds_slab[];
                for (int v = tid; v < nvec; v += kThreads)
                    lds_slab[v] = load16(chunk_v + v);
                __syncthreads();
                const int seg = nvec / kSeg;
                const int sg = tid / kPer, off = tid % kPer;
                for (int i = 0; i * kPer < seg; ++i) {
                    const int v = sg * seg + i * kPer + off;
                    store16_cache(cache_buf, v, lds_slab[v]);
                }
                return;
            }
        }
        for (int v = tid; v < nvec; v += kThreads) {
            if (DIR == kPack)
                store16_chunk<HOST_SIDE>(chunk_v, chunk_buf, v, load16(cache_v + v));
            else
                store16_cache(cache_buf, v, load16(chunk_v + v));
        }
        return;
    }
    RowWalker w(threadIdx.x, a.vec_per_row, a.H);
    int base = 0;  // first chunk-side vector of the current tile (uniform across the workgroup)
    // Full tiles: every thread has U in-range vectors; all U loads issue before any store.
    for (; base + kThreads * U <= nvec; base += kThreads * U) {
        const int v = base + tid;
        int cache_off[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            cache_off[u] = w.cache_vec(a.BS);
            w.advance();
        }
        vec16 buf[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (DIR == kPack)
                buf[u] = load16(cache_v + cache_off[u]);
            else
                buf[u] = load16(chunk_v + v + u * kThreads);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (DIR == kPack)
                store16_chunk<HOST_SIDE>(chunk_v, chunk_buf, v + u * kThreads, buf[u]);
            else
                store16_cache(cache_buf, cache_off[u], buf[u]);
        }
    }
    // Tail: one vector at a time.
    for (int v = base + tid; v < nvec; v += kThreads) {
        const int co = w.cache_vec(a.BS);
        w.advance();
        if (DIR == kPack)
            store16_chunk<HOST_SIDE>(chunk_v, chunk_buf, v, load16(cache_v + co));
        else
            store16_cache(cache_buf, co, load16(chunk_v + v));
    }
}

constexpr int kUnroll = KVX_UNROLL;

}  // namespace

int max_chunks_per_launch(const Geometry &g, int nlayers) {
    const int64_t wgs_per_chunk = static_cast<int64_t>(nlayers) * 2 * g.blocks_per_chunk;
    const int64_t max_wgs = (int64_t{1} << 31) / kThreads - 1;
    int64_t m = max_wgs / wgs_per_chunk;
    if (m > kMaxLaunchChunks)
        m = kMaxLaunchChunks;
    return static_cast<int>(m < 1 ? 1 : m);
}

hipError_t launch_gather(const GatherArgs &args, Direction dir, bool host_side, hipStream_t stream) {
    const int64_t slabs = static_cast<int64_t>(args.nchunks) * args.nlayers * 2 * args.blocks_per_chunk;
    if (slabs <= 0)
        return hipSuccess;
    const int64_t host_wgs = dir == kPack ? KVX_HOST_WGS_PACK : KVX_HOST_WGS_UNPACK;
    const int64_t grid = host_side && host_wgs > 0 ? std::min<int64_t>(slabs, host_wgs) : slabs;
    const void *fn;
    if (host_side)
        fn = dir == kPack ? reinterpret_cast<const void *>(&gather_kernel<kPack, kUnroll, true>)
                          : reinterpret_cast<const void *>(&gather_kernel<kUnpack, kUnroll, true>);
    else
        fn = dir == kPack ? reinterpret_cast<const void *>(&gather_kernel<kPack, kUnroll, false>)
                          : reinterpret_cast<const void *>(&gather_kernel<kUnpack, kUnroll, false>);
    // Device-side (staged) launches cap residency with reserved LDS; host-side launches are
    // already few workgroups and reserve none.
    const unsigned lds = host_side ? 0u : static_cast<unsigned>(KVX_LDS_RESERVE);
    void *kargs[] = {const_cast<GatherArgs *>(&args)};
    // hipLaunchKernel reports launch failures directly (no sticky last-error state).
    return hipLaunchKernel(fn, dim3(static_cast<uint32_t>(grid)), dim3(kThreads), kargs, lds, stream);
}

}  // namespace kvx

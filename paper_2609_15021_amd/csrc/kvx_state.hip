// State-snapshot kernels for gfx950: move the recurrent layers' boundary snapshots
// (convolution state, recurrent state and padding as opaque pages, Sec. 2.2) between
// their device page buffers and the packed state slots, [G][page_bytes] per snapshot.
//
// Each page is contiguous on both sides, so the move is a batched copy: a workgroup moves
// one piece (up to kStatePiece = 16 KiB) of one page at a time with 16-byte vectors.
// Device-side launches run one workgroup per piece and pass it through LDS; host-side
// (zero-copy) launches run a few workgroups that stride over the pieces and copy directly.
// This work is bound by HBM (staging) or by
// the host link (zero-copy); there is no arithmetic to put on the matrix cores.  Bytes
// never pass through a float register.
#include <algorithm>

#include "kvx_internal.h"

namespace kvx {

namespace {

typedef uint32_t svec16 __attribute__((ext_vector_type(4)));

// Vectors each lane keeps in flight before storing (host-side launches).
constexpr int kStateUnroll = 4;
// LDS of a device-side workgroup: the buffer the piece passes through, 32 KiB at a time.
constexpr int kStateLds = 32768;

// Workgroups of a host-side (zero-copy) launch, striding over its pieces (0: one per piece).
// Measured on MI355X with 16 x 48 pages of 3.06 MiB (store / load GB/s): one per piece
// 54.4 / 55.7, 8: 54.3 / 56.6, 16: 55.4 / 57.2, 32: 55.5 / 56.6, 64: 54.9 / 57.3.
#ifndef KVX_STATE_HOST_WGS
#define KVX_STATE_HOST_WGS 16
#endif

// Piece q of the launch's snapshots: [snapshot k][layer g][piece of the page].
template <int DIR, bool HOST_SIDE>
__device__ __forceinline__ void move_piece(const StateArgs &a, int64_t q) {
    const int64_t per_snap = static_cast<int64_t>(a.G) * a.ppp;
    const int k = static_cast<int>(q / per_snap);
    const int64_t rem = q - k * per_snap;
    const int g = static_cast<int>(rem / a.ppp);
    const int64_t start = (rem - static_cast<int64_t>(g) * a.ppp) * a.piece;
    const int64_t len = min(a.piece, a.page_bytes - start);

    uint8_t *page = a.layer[g] + a.page[k] * a.page_stride + start;
    uint8_t *packed = a.base + a.off[k] + static_cast<int64_t>(g) * a.page_bytes + start;
    const svec16 *src = reinterpret_cast<const svec16 *>(DIR == kPack ? page : packed);
    svec16 *dst = reinterpret_cast<svec16 *>(DIR == kPack ? packed : page);
    const int nv = static_cast<int>(len >> 4);  // len <= piece <= kStatePiece
    // Zero-copy stores into mapped pinned host memory use cache policy "nt sc1" (NT = 2, SC1 = 16),
    // as the gather kernels' do: over the link it moved more than plain nontemporal stores.
    const __amdgpu_buffer_rsrc_t dst_buf =
        __builtin_amdgcn_make_buffer_rsrc(dst, 0, static_cast<int>(len), 0x00020000);

    if constexpr (!HOST_SIDE) {
        // Device-side launches move the piece through LDS, at most 32 KiB at a time: contiguous
        // reads into LDS, then writes with each pass spread over 8 segments of what LDS holds.
        // Paired on 48 x 3.06 MiB pages (then in 64 KiB pieces), this moved 2.8-4.5% more (pack)
        // and 3.9-4.0% more (unpack) than the direct copy with 4 vectors in flight; the LDS
        // reservation alone changed nothing.
        extern __shared__ svec16 lds_half[];
        constexpr int kHalf = kStateLds / 16, kPer = kThreads / 8;
        const int tid = static_cast<int>(threadIdx.x);
        for (int h0 = 0; h0 < nv; h0 += kHalf) {
            const int hn = min(kHalf, nv - h0);
            if (hn % (8 * kPer) != 0) {  // a short tail: straight copy
                for (int v = h0 + tid; v < h0 + hn; v += kThreads)
                    __builtin_nontemporal_store(__builtin_nontemporal_load(src + v), dst + v);
                continue;
            }
            for (int v = tid; v < hn; v += kThreads)
                lds_half[v] = __builtin_nontemporal_load(src + h0 + v);
            __syncthreads();
            const int seg = hn / 8, sg = tid / kPer, off = tid % kPer;
            for (int i = 0; i * kPer < seg; ++i) {
                const int v = sg * seg + i * kPer + off;
                __builtin_nontemporal_store(lds_half[v], dst + h0 + v);
            }
            __syncthreads();  // the next half overwrites the buffer
        }
        return;
    }
    for (int v0 = static_cast<int>(threadIdx.x); v0 < nv; v0 += kThreads * kStateUnroll) {
        svec16 buf[kStateUnroll];
#pragma unroll
        for (int u = 0; u < kStateUnroll; ++u) {
            const int v = v0 + u * kThreads;
            if (v < nv)
                buf[u] = __builtin_nontemporal_load(src + v);
        }
#pragma unroll
        for (int u = 0; u < kStateUnroll; ++u) {
            const int v = v0 + u * kThreads;
            if (v < nv) {
                if constexpr (HOST_SIDE && DIR == kPack)
                    __builtin_amdgcn_raw_buffer_store_b128(buf[u], dst_buf, v * 16, 0, 2 | 16);
                else
                    __builtin_nontemporal_store(buf[u], dst + v);
            }
        }
    }
}

template <int DIR, bool HOST_SIDE>
__global__ __launch_bounds__(kThreads) void state_kernel(const StateArgs a) {
    if constexpr (HOST_SIDE) {
        // A capped grid strides over the pieces: the link bounds these launches.
        for (int64_t i = blockIdx.x; i < a.npieces; i += gridDim.x)
            move_piece<DIR, HOST_SIDE>(a, a.q0 + i);
    } else {
        move_piece<DIR, HOST_SIDE>(a, a.q0 + static_cast<int64_t>(blockIdx.x));  // one workgroup per piece
    }
}

}  // namespace

hipError_t launch_state(const StateArgs &args, int64_t pieces, Direction dir, bool host_side,
                        hipStream_t stream) {
    if (pieces <= 0)
        return hipSuccess;
    const void *fn;
    if (host_side)
        fn = dir == kPack ? reinterpret_cast<const void *>(&state_kernel<kPack, true>)
                          : reinterpret_cast<const void *>(&state_kernel<kUnpack, true>);
    else
        fn = dir == kPack ? reinterpret_cast<const void *>(&state_kernel<kPack, false>)
                          : reinterpret_cast<const void *>(&state_kernel<kUnpack, false>);
    StateArgs a = args;
    a.npieces = pieces;
    const int64_t grid = host_side && KVX_STATE_HOST_WGS > 0 ? std::min<int64_t>(pieces, KVX_STATE_HOST_WGS) : pieces;
    void *kargs[] = {&a};
    return hipLaunchKernel(fn, dim3(static_cast<uint32_t>(grid)), dim3(kThreads), kargs, host_side ? 0u : kStateLds,
                           stream);
}

}  // namespace kvx

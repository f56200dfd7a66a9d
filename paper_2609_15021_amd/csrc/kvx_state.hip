// State-snapshot kernels for gfx950: move the recurrent layers' boundary snapshots
// (convolution state, recurrent state and padding as opaque pages, Sec. 2.2) between
// their device page buffers and the packed state slots, [G][page_bytes] per snapshot.
//
// Each page is contiguous on both sides, so the move is a batched copy: one workgroup
// moves one piece (up to 64 KiB) of one page with 16-byte vectors, every lane of a wave
// touching consecutive vectors on both sides.  This work is bound by HBM (staging) or by
// the host link (zero-copy); there is no arithmetic to put on the matrix cores.  Bytes
// never pass through a float register.
#include "kvx_internal.h"

namespace kvx {

namespace {

typedef uint32_t svec16 __attribute__((ext_vector_type(4)));

// Vectors each lane keeps in flight before storing.
constexpr int kStateUnroll = 4;

template <int DIR, bool HOST_SIDE>
__global__ __launch_bounds__(kThreads) void state_kernel(const StateArgs a) {
    const int64_t q = a.q0 + static_cast<int64_t>(blockIdx.x);
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
    const int nv = static_cast<int>(len >> 4);  // len <= piece = 64 KiB

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
            if (v < nv)
                __builtin_nontemporal_store(buf[u], dst + v);
        }
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
    void *kargs[] = {const_cast<StateArgs *>(&args)};
    return hipLaunchKernel(fn, dim3(static_cast<uint32_t>(pieces)), dim3(kThreads), kargs, 0, stream);
}

}  // namespace kvx

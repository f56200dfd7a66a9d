// Test and benchmark harness kernels (not part of the kvx library):
//  * kvh_fill_values: the device twin of harness/__init__.py's seeded value generator
//    (counter-based SplitMix64; u11 / n01 bf16 and raw-bit distributions);
//  * kvh_spin: a producer delay that spins on the constant-rate wall clock;
//  * kvh_fill_u8 / kvh_copy_u8: byte fill and same-stream device copy kernels (the
//    delayed producer and consumer of the paper's byte probes);
//  * kvh_copy_raw / kvh_copy_sync_then_raw / kvh_copy_async: the host-side copy
//    variants of the paper's ordering controls (Sec. 3.2) -- a raw synchronous copy that
//    names no stream, the same after waiting for the stream, and an async copy on it.
// Nothing here implements any part of the store/load arithmetic.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>

namespace {

thread_local std::string g_err;

int fail(hipError_t e, const char *what) {
    char buf[512];
    snprintf(buf, sizeof(buf), "%s: %s (%s)", what, hipGetErrorName(e), hipGetErrorString(e));
    g_err = buf;
    return -1;
}

#define KVH_HIP(expr)                   \
    do {                                \
        hipError_t e_ = (expr);         \
        if (e_ != hipSuccess)           \
            return fail(e_, #expr);     \
    } while (0)

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

// SplitMix64 finaliser, written on explicit 32-bit halves.  The equivalent expression on
// uint64_t values was compiled into code that dropped the last shift-xor for the 1- and
// 4-byte fill instantiations on gfx950 (checked against the host generator with a
// standalone build); the 32-bit form computes the published function exactly.
struct u64h {
    uint32_t lo, hi;
};
__device__ __forceinline__ u64h shr(u64h a, int s) { return {(a.lo >> s) | (a.hi << (32 - s)), a.hi >> s}; }
__device__ __forceinline__ u64h xr(u64h a, u64h b) { return {a.lo ^ b.lo, a.hi ^ b.hi}; }
// Low 64 bits of a * (chi:clo).
__device__ __forceinline__ u64h mulc(u64h a, uint32_t clo, uint32_t chi) {
    return {a.lo * clo, __umulhi(a.lo, clo) + a.lo * chi + a.hi * clo};
}
__device__ __forceinline__ uint64_t mix64(uint64_t z64) {
    u64h z{static_cast<uint32_t>(z64), static_cast<uint32_t>(z64 >> 32)};
    z = xr(z, shr(z, 30));
    z = mulc(z, 0x1CE4E5B9u, 0xBF58476Du);
    z = xr(z, shr(z, 27));
    z = mulc(z, 0x133111EBu, 0x94D049BBu);
    z = xr(z, shr(z, 31));
    return (static_cast<uint64_t>(z.hi) << 32) | z.lo;
}

__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// dist: 0 = u11, 1 = n01, 2 = raw.  Returns the element's low elem_bytes*8 bits.
__device__ __forceinline__ uint32_t value_of(uint64_t seed, uint64_t counter, int dist) {
    const uint64_t z = mix64(seed + (counter + 1) * kGamma);
    if (dist == 0) {
        const int32_t k = static_cast<int32_t>(z >> 40) - (1 << 23);
        return bf16_rne(static_cast<float>(k) * 0x1p-23f);
    }
    if (dist == 1) {
        const int32_t s = static_cast<int32_t>((z & 0xFFFF) + ((z >> 16) & 0xFFFF) + ((z >> 32) & 0xFFFF) +
                                               ((z >> 48) & 0xFFFF)) -
                          131070;
        // fp32 sqrt(3)/65536 rounded to nearest: bits 0x37ddb3d7.
        return bf16_rne(static_cast<float>(s) * __uint_as_float(0x37ddb3d7u));
    }
    return static_cast<uint32_t>(z);
}

// Each work-item writes one 16-byte vector of 16/E elements, grid-stride.
template <int E>
__global__ __launch_bounds__(256) void fill_values_kernel(uint4 *dst, int64_t nvec, uint64_t counter0, uint64_t seed,
                                                          int dist) {
    constexpr int per = 16 / E;
    for (int64_t v = blockIdx.x * 256ll + threadIdx.x; v < nvec; v += static_cast<int64_t>(gridDim.x) * 256) {
        uint32_t w[4] = {0, 0, 0, 0};
        const uint64_t c0 = counter0 + static_cast<uint64_t>(v) * per;
#pragma unroll
        for (int k = 0; k < per; ++k) {
            const uint32_t x = value_of(seed, c0 + k, dist);
            if (E == 4)
                w[k] = x;
            else if (E == 2)
                w[k / 2] |= (x & 0xFFFFu) << (16 * (k % 2));
            else
                w[k / 4] |= (x & 0xFFu) << (8 * (k % 4));
        }
        dst[v] = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

__global__ void spin_kernel(uint64_t ticks) {
    const uint64_t t0 = wall_clock64();
    while (wall_clock64() - t0 < ticks)
        __builtin_amdgcn_s_sleep(64);
}

__global__ __launch_bounds__(256) void fill_u8_kernel(uint8_t *dst, int64_t n, uint8_t value) {
    for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256)
        dst[i] = value;
}

__global__ __launch_bounds__(256) void copy_u8_kernel(uint8_t *dst, const uint8_t *src, int64_t n) {
    for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256)
        dst[i] = src[i];
}

unsigned grid_for(int64_t work) {
    int64_t g = (work + 255) / 256;
    if (g > 65536)
        g = 65536;
    return static_cast<unsigned>(g < 1 ? 1 : g);
}

}  // namespace

extern "C" {

const char *kvh_last_error(void) { return g_err.c_str(); }

// Fill n_elems elements of elem_bytes at dst with the generator's values for counters
// counter0 .. counter0 + n_elems - 1.  n_elems*elem_bytes must be a multiple of 16 and
// dst 16-byte aligned.
int kvh_fill_values(void *dst, uint64_t counter0, int64_t n_elems, int elem_bytes, uint64_t seed, int dist,
                    void *stream) {
    if (!dst || n_elems < 0 || (elem_bytes != 1 && elem_bytes != 2 && elem_bytes != 4) || dist < 0 || dist > 2 ||
        (n_elems * elem_bytes) % 16 != 0 || reinterpret_cast<uintptr_t>(dst) % 16 != 0) {
        g_err = "kvh_fill_values: bad arguments";
        return -1;
    }
    if ((dist == 0 || dist == 1) && elem_bytes != 2) {
        g_err = "kvh_fill_values: u11/n01 are bf16 (elem_bytes 2)";
        return -1;
    }
    const int64_t nvec = n_elems * elem_bytes / 16;
    if (nvec == 0)
        return 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint4 *d = static_cast<uint4 *>(dst);
    const unsigned grid = grid_for(nvec);
    if (elem_bytes == 1)
        hipLaunchKernelGGL(fill_values_kernel<1>, dim3(grid), dim3(256), 0, s, d, nvec, counter0, seed, dist);
    else if (elem_bytes == 2)
        hipLaunchKernelGGL(fill_values_kernel<2>, dim3(grid), dim3(256), 0, s, d, nvec, counter0, seed, dist);
    else
        hipLaunchKernelGGL(fill_values_kernel<4>, dim3(grid), dim3(256), 0, s, d, nvec, counter0, seed, dist);
    KVH_HIP(hipGetLastError());
    return 0;
}

// Enqueue a single-wave kernel that spins for `ms` milliseconds of wall-clock time
// (0 <= ms <= 10000), measured on the device's constant-rate counter.
int kvh_spin(void *stream, double ms) {
    if (!(ms >= 0.0 && ms <= 10000.0)) {
        g_err = "kvh_spin: ms must be in [0, 10000]";
        return -1;
    }
    int dev = 0, khz = 0;
    KVH_HIP(hipGetDevice(&dev));
    KVH_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    const uint64_t ticks = static_cast<uint64_t>(ms * static_cast<double>(khz));
    hipLaunchKernelGGL(spin_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream), ticks);
    KVH_HIP(hipGetLastError());
    return 0;
}

int kvh_wall_clock_khz(void) {
    int dev = 0, khz = 0;
    KVH_HIP(hipGetDevice(&dev));
    KVH_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    return khz;
}

int kvh_fill_u8(void *dst, int64_t n, int value, void *stream) {
    if (!dst || n < 0 || value < 0 || value > 255) {
        g_err = "kvh_fill_u8: bad arguments";
        return -1;
    }
    if (n == 0)
        return 0;
    hipLaunchKernelGGL(fill_u8_kernel, dim3(grid_for(n)), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<uint8_t *>(dst), n, static_cast<uint8_t>(value));
    KVH_HIP(hipGetLastError());
    return 0;
}

// Same-stream device copy by a kernel (the paper's third ordered control, a tensor copy).
int kvh_copy_u8(void *dst, const void *src, int64_t n, void *stream) {
    if (!dst || !src || n < 0) {
        g_err = "kvh_copy_u8: bad arguments";
        return -1;
    }
    if (n == 0)
        return 0;
    hipLaunchKernelGGL(copy_u8_kernel, dim3(grid_for(n)), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<uint8_t *>(dst), static_cast<const uint8_t *>(src), n);
    KVH_HIP(hipGetLastError());
    return 0;
}

// The faulty branch of the paper (Sec. 3.2): a synchronous raw copy that names no stream.
int kvh_copy_raw(void *dst, const void *src, int64_t n) {
    KVH_HIP(hipMemcpy(dst, src, static_cast<size_t>(n), hipMemcpyDefault));
    return 0;
}

// Ordered control 1: wait for the preceding stream work, then the same raw copy.
int kvh_copy_sync_then_raw(void *dst, const void *src, int64_t n, void *stream) {
    KVH_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    KVH_HIP(hipMemcpy(dst, src, static_cast<size_t>(n), hipMemcpyDefault));
    return 0;
}

// Ordered control 2: an asynchronous copy on the current stream.
int kvh_copy_async(void *dst, const void *src, int64_t n, void *stream) {
    KVH_HIP(hipMemcpyAsync(dst, src, static_cast<size_t>(n), hipMemcpyDefault, static_cast<hipStream_t>(stream)));
    return 0;
}

// Streams with explicit flags for the ordering tests (0 = blocking, 1 = non-blocking).
// Default priority only.
int kvh_stream_create(int non_blocking, void **out) {
    hipStream_t s = nullptr;
    KVH_HIP(hipStreamCreateWithFlags(&s, non_blocking ? hipStreamNonBlocking : hipStreamDefault));
    *out = s;
    return 0;
}

int kvh_stream_destroy(void *stream) {
    KVH_HIP(hipStreamDestroy(static_cast<hipStream_t>(stream)));
    return 0;
}

int kvh_stream_sync(void *stream) {
    KVH_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    return 0;
}

// Pinned host buffers for probes (never pageable; cf. Sec. 3.3).
int kvh_host_alloc(int64_t n, void **out) {
    KVH_HIP(hipHostMalloc(out, static_cast<size_t>(n), hipHostMallocMapped | hipHostMallocPortable));
    return 0;
}

// Device-side address of pinned host memory from kvh_host_alloc (for same-stream kernel copies).
int kvh_host_device_ptr(void *host, void **out) {
    KVH_HIP(hipHostGetDevicePointer(out, host, 0));
    return 0;
}

int kvh_host_free(void *p) {
    KVH_HIP(hipHostFree(p));
    return 0;
}

}  // extern "C"

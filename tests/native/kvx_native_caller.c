/*
 * A native C caller of the kvx C ABI: no Python, no torch.  It reads a host cache, two block
 * tables and chunk ids from files, copies the cache to device memory it allocates itself,
 * stores the prefix into a pool and loads it into a second device cache on a stream it
 * created, then writes the pool bytes and the second cache back to files.  The calling test
 * compares them with the CPU oracle.
 *
 * usage: kvx_native_caller MODE L H D E BS C NB N NSLOTS DIR
 *   MODE: staged | zero_copy; DIR holds a.bin, bta.bin, btb.bin, ids.bin (inputs) and
 *   receives pool.bin and b.bin.  Exit status 0 on success; errors name the failing call.
 */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "kvx.h"

static int read_file(const char *dir, const char *name, void *buf, size_t n) {
    char path[4096];
    snprintf(path, sizeof(path), "%s/%s", dir, name);
    FILE *f = fopen(path, "rb");
    if (!f)
        return -1;
    size_t got = fread(buf, 1, n, f);
    fclose(f);
    return got == n ? 0 : -1;
}

static int write_file(const char *dir, const char *name, const void *buf, size_t n) {
    char path[4096];
    snprintf(path, sizeof(path), "%s/%s", dir, name);
    FILE *f = fopen(path, "wb");
    if (!f)
        return -1;
    size_t put = fwrite(buf, 1, n, f);
    return (fclose(f) == 0 && put == n) ? 0 : -1;
}

#define CHECK_HIP(x)                                                             \
    do {                                                                         \
        hipError_t e_ = (x);                                                     \
        if (e_ != hipSuccess) {                                                  \
            fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorName(e_));         \
            return 1;                                                            \
        }                                                                        \
    } while (0)

#define CHECK_KV(x)                                                              \
    do {                                                                         \
        kv_status s_ = (x);                                                      \
        if (s_ != KV_OK) {                                                       \
            fprintf(stderr, "%s failed: %s\n", #x, kv_last_error());             \
            return 1;                                                            \
        }                                                                        \
    } while (0)

int main(int argc, char **argv) {
    if (argc != 12) {
        fprintf(stderr, "usage: %s MODE L H D E BS C NB N NSLOTS DIR\n", argv[0]);
        return 2;
    }
    const int staged = strcmp(argv[1], "staged") == 0;
    kv_layout lay = {atoi(argv[2]), atoi(argv[3]), atoi(argv[4]), atoi(argv[5]), atoi(argv[6]), atoi(argv[7])};
    const int32_t nb = atoi(argv[8]);
    const int64_t n = atoll(argv[9]), nslots = atoll(argv[10]);
    const char *dir = argv[11];
    const int64_t nblk = (n + lay.block_size - 1) / lay.block_size;
    const int64_t nc = (n + lay.chunk_tokens - 1) / lay.chunk_tokens;
    const size_t layer_bytes = (size_t)nb * 2 * lay.num_kv_heads * lay.block_size * lay.head_dim * lay.elem_bytes;
    const size_t cache_bytes = layer_bytes * (size_t)lay.num_layers;

    unsigned char *host_a = malloc(cache_bytes), *host_b = malloc(cache_bytes);
    int32_t *bta = malloc((size_t)nblk * 4), *btb = malloc((size_t)nblk * 4);
    int64_t *ids = malloc((size_t)nc * 8);
    void **layers_a = malloc(sizeof(void *) * (size_t)lay.num_layers);
    void **layers_b = malloc(sizeof(void *) * (size_t)lay.num_layers);
    if (!host_a || !host_b || !bta || !btb || !ids || !layers_a || !layers_b)
        return 1;
    if (read_file(dir, "a.bin", host_a, cache_bytes) || read_file(dir, "bta.bin", bta, (size_t)nblk * 4) ||
        read_file(dir, "btb.bin", btb, (size_t)nblk * 4) || read_file(dir, "ids.bin", ids, (size_t)nc * 8)) {
        fprintf(stderr, "cannot read the inputs in %s\n", dir);
        return 1;
    }

    int device = 0;
    CHECK_HIP(hipSetDevice(device));
    unsigned char *dev_a = NULL, *dev_b = NULL;
    int32_t *dev_bta = NULL, *dev_btb = NULL;
    CHECK_HIP(hipMalloc((void **)&dev_a, cache_bytes));
    CHECK_HIP(hipMalloc((void **)&dev_b, cache_bytes));
    CHECK_HIP(hipMalloc((void **)&dev_bta, (size_t)nblk * 4));
    CHECK_HIP(hipMalloc((void **)&dev_btb, (size_t)nblk * 4));
    CHECK_HIP(hipMemcpy(dev_a, host_a, cache_bytes, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemset(dev_b, 0x5A, cache_bytes));
    CHECK_HIP(hipMemcpy(dev_bta, bta, (size_t)nblk * 4, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(dev_btb, btb, (size_t)nblk * 4, hipMemcpyHostToDevice));
    /* The work below runs on a non-blocking stream: finish the set-up copies and fill first. */
    CHECK_HIP(hipDeviceSynchronize());
    for (int l = 0; l < lay.num_layers; ++l) {
        layers_a[l] = dev_a + (size_t)l * layer_bytes;
        layers_b[l] = dev_b + (size_t)l * layer_bytes;
    }
    kv_cache cache_a, cache_b;
    memset(&cache_a, 0, sizeof(cache_a));
    cache_a.layout = lay;
    cache_a.num_blocks = nb;
    cache_a.device = device;
    cache_a.block_order = KV_BLOCK_HND;
    cache_a.layer_ptrs = (void *const *)layers_a;
    cache_b = cache_a;
    cache_b.layer_ptrs = (void *const *)layers_b;

    kv_pool_options opts;
    memset(&opts, 0, sizeof(opts));
    opts.mode = staged ? KV_MODE_STAGED : KV_MODE_ZERO_COPY;
    opts.staging_slots = staged ? 2 : 0;
    opts.chunks_per_batch = staged ? 2 : 0;
    kv_pool *pool = NULL;
    CHECK_KV(kv_pool_create(&lay, nslots, &opts, &pool));
    const int64_t slot_bytes = kv_pool_slot_bytes(pool);
    memset(kv_pool_slot(pool, 0), 0xA5, (size_t)(slot_bytes * nslots));

    hipStream_t stream;
    CHECK_HIP(hipStreamCreateWithFlags(&stream, hipStreamNonBlocking));
    CHECK_KV(kv_store(&cache_a, dev_bta, n, pool, ids, stream));
    CHECK_KV(kv_load(&cache_b, dev_btb, n, pool, ids, stream));
    CHECK_HIP(hipStreamSynchronize(stream)); /* host completion before reading the pool */
    if (kv_pool_async_error(pool, 0) != 0) {
        fprintf(stderr, "device-side fault reported\n");
        return 1;
    }
    CHECK_HIP(hipMemcpy(host_b, dev_b, cache_bytes, hipMemcpyDeviceToHost));
    if (write_file(dir, "pool.bin", kv_pool_slot(pool, 0), (size_t)(slot_bytes * nslots)) ||
        write_file(dir, "b.bin", host_b, cache_bytes)) {
        fprintf(stderr, "cannot write the outputs in %s\n", dir);
        return 1;
    }
    CHECK_KV(kv_pool_destroy(pool));
    CHECK_HIP(hipStreamDestroy(stream));
    CHECK_HIP(hipFree(dev_a));
    CHECK_HIP(hipFree(dev_b));
    CHECK_HIP(hipFree(dev_bta));
    CHECK_HIP(hipFree(dev_btb));
    free(host_a);
    free(host_b);
    free(bta);
    free(btb);
    free(ids);
    free(layers_a);
    free(layers_b);
    printf("NATIVE OK %s %lld tokens\n", argv[1], (long long)n);
    return 0;
}

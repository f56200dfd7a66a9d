// kvx_tierd: the shared host tier as a standalone process (the paper's host tier that replicas
// share, Sec. 2 and Fig. 1).  It pins one pool and a pool index over its slots, listens on a Unix
// stream socket and serves replica processes through the C ABI's tier calls: by slot
// (kv_tier_store / kv_tier_load) and by prompt (kv_tier_store_prefix / kv_tier_load_prefix, the
// index choosing the slots).  It runs until the given number of connections has ended, or until
// SIGINT or SIGTERM shuts the listening socket down; connections in progress finish first.
//
// usage: kvx_tierd --socket PATH --layout L,H,D,E,BS,C --slots N [--mode M] [--device D]
//                  [--staging-slots K] [--chunks-per-batch B] [--state-slots S --state-bytes SB]
//                  [--index-slots I] [--connections K] [--fill BYTE] [--dump FILE] [--hip-runtime SO]
//   M: staged, zero_copy, or STORE+LOAD (e.g. staged+zero_copy: stores staged, loads zero-copy)
//   I: slots the index manages (default N; 0 = no index, slot requests only)
//   SO: the HIP runtime library to use.  The replicas hand over their caches as HIP IPC handles,
//       which open only in a process running the same runtime build as theirs (a replica in a
//       torch process uses the runtime torch ships).  The daemon loads SO (default: the system's
//       libamdhip64.so.7) before libkvx.so, so that the library binds to it.
// Prints "READY <path>" once listening, then "STATS ..." (with an index) and "TIER ok" or
// "TIER <error>" at the end; exit status 0 on success.
#include <dlfcn.h>
#include <sys/socket.h>
#include <unistd.h>

#include <climits>
#include <csignal>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

#include "kvx.h"

namespace {

// The C ABI entry points the daemon calls, resolved from libkvx.so after the HIP runtime is loaded.
struct Api {
    decltype(&kv_pool_create) pool_create;
    decltype(&kv_pool_set_modes) pool_set_modes;
    decltype(&kv_pool_slot) pool_slot;
    decltype(&kv_pool_slot_bytes) pool_slot_bytes;
    decltype(&kv_pool_destroy) pool_destroy;
    decltype(&kv_index_create) index_create;
    decltype(&kv_index_get_stats) index_get_stats;
    decltype(&kv_index_destroy) index_destroy;
    decltype(&kv_tier_listen) tier_listen;
    decltype(&kv_tier_run) tier_run;
    decltype(&kv_last_error) last_error;
    int (*set_device)(int);  // hipSetDevice
};

template <class F>
bool resolve(void *lib, const char *name, F *out) {
    *out = reinterpret_cast<F>(dlsym(lib, name));
    if (!*out)
        std::fprintf(stderr, "kvx_tierd: %s not found: %s\n", name, dlerror());
    return *out != nullptr;
}

bool load_api(const std::string &hip_runtime, Api *api) {
    void *hip = dlopen(hip_runtime.c_str(), RTLD_NOW | RTLD_GLOBAL);
    if (!hip) {
        std::fprintf(stderr, "kvx_tierd: cannot load the HIP runtime %s: %s\n", hip_runtime.c_str(), dlerror());
        return false;
    }
    char exe[PATH_MAX];
    const ssize_t len = readlink("/proc/self/exe", exe, sizeof(exe) - 1);
    if (len <= 0)
        return false;
    exe[len] = '\0';
    std::string dir(exe);
    dir = dir.substr(0, dir.rfind('/'));
    void *lib = dlopen((dir + "/libkvx.so").c_str(), RTLD_NOW | RTLD_LOCAL);
    if (!lib) {
        std::fprintf(stderr, "kvx_tierd: cannot load %s/libkvx.so: %s\n", dir.c_str(), dlerror());
        return false;
    }
    return resolve(lib, "kv_pool_create", &api->pool_create) &&
           resolve(lib, "kv_pool_set_modes", &api->pool_set_modes) &&
           resolve(lib, "kv_pool_slot", &api->pool_slot) && resolve(lib, "kv_pool_slot_bytes", &api->pool_slot_bytes) &&
           resolve(lib, "kv_pool_destroy", &api->pool_destroy) && resolve(lib, "kv_index_create", &api->index_create) &&
           resolve(lib, "kv_index_get_stats", &api->index_get_stats) &&
           resolve(lib, "kv_index_destroy", &api->index_destroy) && resolve(lib, "kv_tier_listen", &api->tier_listen) &&
           resolve(lib, "kv_tier_run", &api->tier_run) && resolve(lib, "kv_last_error", &api->last_error) &&
           resolve(hip, "hipSetDevice", &api->set_device);
}

volatile sig_atomic_t g_listen_fd = -1;
volatile sig_atomic_t g_stopped = 0;

void on_signal(int) {
    g_stopped = 1;
    // Async-signal-safe: the (restarted) accept on the listening socket then fails, and the accept
    // loop stops taking connections and waits for those in progress.  close() would not wake it.
    if (g_listen_fd >= 0)
        shutdown(g_listen_fd, SHUT_RDWR);
}

int usage(const char *msg) {
    std::fprintf(stderr, "kvx_tierd: %s\n", msg);
    std::fprintf(stderr,
                 "usage: kvx_tierd --socket PATH --layout L,H,D,E,BS,C --slots N [--mode M] [--device D]\n"
                 "                 [--staging-slots K] [--chunks-per-batch B] [--state-slots S --state-bytes SB]\n"
                 "                 [--index-slots I] [--connections K] [--fill BYTE] [--dump FILE]\n"
                 "                 [--hip-runtime SO]\n");
    return 2;
}

bool parse_mode(const std::string &s, uint32_t *mode) {
    if (s == "staged")
        *mode = KV_MODE_STAGED;
    else if (s == "zero_copy")
        *mode = KV_MODE_ZERO_COPY;
    else
        return false;
    return true;
}

Api g_api;

int fail(const char *what) {
    std::printf("TIER %s failed: %s\n", what, g_api.last_error());
    std::fflush(stdout);
    return 1;
}

}  // namespace

int main(int argc, char **argv) {
    std::string sock, layout_s, mode_s = "staged", dump, hip_runtime = "libamdhip64.so.7";
    long long slots = 0, state_slots = 0, state_bytes = 0, index_slots = -1;
    int device = 0, staging_slots = 3, cpb = 0, connections = 0, fill = -1;
    for (int i = 1; i < argc; ++i) {
        const std::string a = argv[i];
        if (i + 1 >= argc)
            return usage(("missing value after " + a).c_str());
        const char *v = argv[++i];
        if (a == "--socket") sock = v;
        else if (a == "--layout") layout_s = v;
        else if (a == "--slots") slots = std::atoll(v);
        else if (a == "--mode") mode_s = v;
        else if (a == "--device") device = std::atoi(v);
        else if (a == "--staging-slots") staging_slots = std::atoi(v);
        else if (a == "--chunks-per-batch") cpb = std::atoi(v);
        else if (a == "--state-slots") state_slots = std::atoll(v);
        else if (a == "--state-bytes") state_bytes = std::atoll(v);
        else if (a == "--index-slots") index_slots = std::atoll(v);
        else if (a == "--connections") connections = std::atoi(v);
        else if (a == "--fill") fill = std::atoi(v);
        else if (a == "--dump") dump = v;
        else if (a == "--hip-runtime") hip_runtime = v;
        else return usage(("unknown option " + a).c_str());
    }
    kv_layout lay;
    if (sock.empty() || slots < 1 ||
        std::sscanf(layout_s.c_str(), "%d,%d,%d,%d,%d,%d", &lay.num_layers, &lay.num_kv_heads, &lay.head_dim,
                    &lay.elem_bytes, &lay.block_size, &lay.chunk_tokens) != 6)
        return usage("--socket, --layout L,H,D,E,BS,C and --slots N >= 1 are required");
    uint32_t store_mode = 0, load_mode = 0;
    const size_t plus = mode_s.find('+');
    if (!parse_mode(mode_s.substr(0, plus), &store_mode) ||
        !parse_mode(plus == std::string::npos ? mode_s : mode_s.substr(plus + 1), &load_mode))
        return usage("--mode must be staged, zero_copy or STORE+LOAD of those");
    if (index_slots < 0)
        index_slots = slots;

    if (!load_api(hip_runtime, &g_api))
        return 1;
    const Api &k = g_api;
    if (k.set_device(device) != 0)
        return usage("cannot select the device");
    kv_pool_options opts;
    std::memset(&opts, 0, sizeof(opts));
    opts.mode = store_mode;
    opts.staging_slots = (store_mode == KV_MODE_STAGED || load_mode == KV_MODE_STAGED) ? staging_slots : 0;
    opts.chunks_per_batch = cpb;
    opts.num_state_slots = state_slots;
    opts.state_slot_bytes = state_bytes;
    kv_pool *pool = nullptr;
    if (k.pool_create(&lay, slots, &opts, &pool) != KV_OK)
        return fail("kv_pool_create");
    if (k.pool_set_modes(pool, store_mode, load_mode) != KV_OK)
        return fail("kv_pool_set_modes");
    if (fill >= 0)
        std::memset(k.pool_slot(pool, 0), fill & 0xFF, static_cast<size_t>(slots * k.pool_slot_bytes(pool)));
    kv_index *index = nullptr;
    if (index_slots > 0 && k.index_create(lay.chunk_tokens, index_slots, state_slots, &index) != KV_OK)
        return fail("kv_index_create");

    int fd = -1;
    if (k.tier_listen(sock.c_str(), &fd) != KV_OK)
        return fail("kv_tier_listen");
    g_listen_fd = fd;
    std::signal(SIGINT, on_signal);
    std::signal(SIGTERM, on_signal);
    std::printf("READY %s\n", sock.c_str());
    std::fflush(stdout);

    const kv_status st = k.tier_run(pool, index, fd, connections);
    const std::string err = st == KV_OK ? std::string() : std::string(k.last_error());
    g_listen_fd = -1;
    close(fd);
    unlink(sock.c_str());
    if (index) {
        kv_index_stats s;
        if (k.index_get_stats(index, &s) == KV_OK)
            std::printf("STATS entries=%lld pending=%lld free_slots=%lld state_entries=%lld evictions=%lld "
                        "state_evictions=%lld\n",
                        static_cast<long long>(s.entries), static_cast<long long>(s.pending),
                        static_cast<long long>(s.free_slots), static_cast<long long>(s.state_entries),
                        static_cast<long long>(s.evictions), static_cast<long long>(s.state_evictions));
        k.index_destroy(index);
    }
    if (!dump.empty()) {
        FILE *f = std::fopen(dump.c_str(), "wb");
        const size_t n = static_cast<size_t>(slots * k.pool_slot_bytes(pool));
        if (!f || std::fwrite(k.pool_slot(pool, 0), 1, n, f) != n || std::fclose(f) != 0) {
            std::printf("TIER cannot write %s\n", dump.c_str());
            return 1;
        }
    }
    k.pool_destroy(pool);
    // A stop by signal shuts the listening socket down under the accept loop: that is a clean end.
    if (st != KV_OK && !g_stopped) {
        std::printf("TIER %s\n", err.c_str());
        return 1;
    }
    std::printf("TIER ok\n");
    return 0;
}

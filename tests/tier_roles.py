"""Process roles for the tier tests (run as separate processes by tests/test_gpu_tier.py).

  tier  SOCK L H D E BS C SLOTS MODE NCONN DUMP   own the pool, serve NCONN replica connections
                                                  (one Python thread each), then save the pool bytes
                                                  to DUMP
  tier-native  (same arguments) INDEX_SLOTS        the same with the library's own listener and threads,
                                                  and a pool index over INDEX_SLOTS slots
  store SOCK L H D E BS C NB N SEED DELAY_MS      replica A: its cache from the seeded generator
                                                  (DELAY_MS > 0: zeros, then a delayed producer
                                                  writes byte 37 on its stream), stored through the tier
  store-prefix SOCK L H D E BS C NB N SEED SALT    replica A stores the prompt harness.prompt_tokens(SEED, N)
                                                  by prefix; prints the chunks it stored
  store-hybrid (store-prefix arguments) G PB NPAGES PAGE
                                                  the same plus recurrent-state pages (state_pages(SEED, ...))
                                                  whose page PAGE is the snapshot after the last whole chunk
"""
import os
import socket
import sys
import threading

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import harness  # noqa: E402
from harness import gpu as hg  # noqa: E402
from paper_2609_15021_amd import kvx  # noqa: E402

POOL_SENT = 0xA5


def _pool(lay, slots, mode, **kw):
    """mode: zero_copy, staged, or staged+zero_copy (staged stores, zero-copy loads)."""
    store_mode, _, load_mode = mode.partition("+")
    pool = kvx.kv_pool_create(lay, slots, store_mode, staging_slots=2, chunks_per_batch=2, **kw)
    if load_mode:
        kvx.kv_pool_set_modes(pool, store_mode, load_mode)
    return pool


def tier(sock, L, H, D, E, BS, C, slots, mode, nconn, dump):
    lay = kvx.make_layout(L, H, D, E, BS, C)
    pool = _pool(lay, slots, mode)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    srv = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    srv.bind(sock)
    srv.listen(8)
    srv.settimeout(90)
    print("READY", flush=True)
    results = []

    def serve(conn):
        try:
            kvx.kv_tier_serve(pool, conn.fileno())
            results.append("ok")
        except Exception as e:  # reported to the test through stdout
            results.append(repr(e))
        finally:
            conn.close()

    threads = []
    for _ in range(nconn):
        conn, _ = srv.accept()
        t = threading.Thread(target=serve, args=(conn,))
        t.start()
        threads.append(t)
    for t in threads:
        t.join(timeout=90)
    np.save(dump, view.copy())
    print("TIER", ";".join(results), flush=True)
    kvx.kv_pool_destroy(pool)


def state_pages(seed, G, npages, pb):
    """Seeded recurrent-state pages [G][npages][pb] (uint8)."""
    return np.random.default_rng(seed + 77).integers(0, 256, size=(G, npages, pb), dtype=np.uint8)


def tier_native(sock, L, H, D, E, BS, C, slots, mode, nconn, dump, index_slots, state_slots=0, state_bytes=0):
    lay = kvx.make_layout(L, H, D, E, BS, C)
    pool = _pool(lay, slots, mode, num_state_slots=state_slots, state_slot_bytes=state_bytes)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    index = kvx.kv_index_create(C, index_slots, state_slots) if index_slots else None
    fd = kvx.kv_tier_listen(sock)
    print("READY", flush=True)
    try:
        kvx.kv_tier_run(pool, fd, nconn, index)
        result = "ok"
    except kvx.KvError as e:
        result = repr(e)
    os.close(fd)
    np.save(dump, view.copy())
    if index is not None:
        print("INDEX", kvx.kv_index_get_stats(index), flush=True)
    print("TIER", result, flush=True)
    kvx.kv_pool_destroy(pool)


def replica_cache(L, H, D, E, BS, C, NB, seed):
    lay = kvx.make_layout(L, H, D, E, BS, C)
    A = harness.gen_cache(seed, "raw", L, NB, H, BS, D, E)
    dA = torch.from_numpy(A.view({1: np.uint8, 2: np.int16, 4: np.int32}[E])).to("cuda:0")
    torch.cuda.synchronize()
    return dA, kvx.Cache(dA, lay, NB)


def store_prefix(sock, L, H, D, E, BS, C, NB, n, seed, salt):
    dA, cache = replica_cache(L, H, D, E, BS, C, NB, seed)
    bt = harness.block_table(seed + 1, NB, -(-n // BS))
    c = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    c.connect(sock)
    stored, _ = kvx.kv_tier_store_prefix(c.fileno(), cache, bt, salt, harness.prompt_tokens(seed, n))
    c.close()
    print("STORED", stored, flush=True)


def store_hybrid(sock, L, H, D, E, BS, C, NB, n, seed, salt, G, pb, npages, page):
    dA, cache = replica_cache(L, H, D, E, BS, C, NB, seed)
    dS = torch.from_numpy(state_pages(seed, G, npages, pb)).to("cuda:0")
    torch.cuda.synchronize()
    bt = harness.block_table(seed + 1, NB, -(-n // BS))
    c = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    c.connect(sock)
    stored, stored_state = kvx.kv_tier_store_prefix(c.fileno(), cache, bt, salt, harness.prompt_tokens(seed, n),
                                                    state=kvx.State(dS, pb, npages), state_page=page)
    c.close()
    print("STORED", stored, stored_state, flush=True)


def store(sock, L, H, D, E, BS, C, NB, n, seed, delay_ms):
    lay = kvx.make_layout(L, H, D, E, BS, C)
    A = harness.gen_cache(seed, "raw", L, NB, H, BS, D, E)
    dA = torch.from_numpy(A.view({1: np.uint8, 2: np.int16, 4: np.int32}[E])).to("cuda:0")
    bt = harness.block_table(seed + 1, NB, -(-n // BS))
    ids = np.arange(-(-n // C))
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    if delay_ms > 0:
        dA.zero_()
        torch.cuda.synchronize()
        hg.spin(float(delay_ms), s)
        hg.fill_u8(dA, dA.numel() * dA.element_size(), 37, s)
    c = socket.socket(socket.AF_UNIX, socket.SOCK_STREAM)
    c.connect(sock)
    kvx.kv_tier_store(c.fileno(), kvx.Cache(dA, lay, NB), bt, n, ids, s)
    c.close()
    print("STORED", flush=True)


if __name__ == "__main__":
    role, args = sys.argv[1], sys.argv[2:]
    if role == "tier":
        tier(args[0], *map(int, args[1:8]), args[8], int(args[9]), args[10])
    elif role == "tier-native":
        tier_native(args[0], *map(int, args[1:8]), args[8], int(args[9]), args[10], *map(int, args[11:]))
    elif role == "store":
        store(args[0], *map(int, args[1:12]))
    elif role == "store-prefix":
        store_prefix(args[0], *map(int, args[1:12]))
    elif role == "store-hybrid":
        store_hybrid(args[0], *map(int, args[1:16]))
    else:
        raise SystemExit(f"unknown role {role}")

"""kv_load_noalloc through the C ABI: the restore that allocates nothing (static device scratch,
every copy and kernel on the caller's stream) must give exactly kv_load's result on the same inputs,
on two calls in a row, the second with a smaller input.  Bit-exact (the path moves opaque bytes); the
tiny case and 24 seeded random layouts are also compared with the CPU oracle."""
import ctypes

import numpy as np
import pytest
import torch

import harness
import oracle
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import (B27, DEV, TINY, bt_tensor, first_mismatch, host_cache, oracle_pool,
                               oracle_unpack_into, to_device, to_host)

pytestmark = pytest.mark.gpu

SENT = 0x5A


def _noalloc(cache, block_table, n, pool, chunk_ids, stream):
    """The entry point called directly through the C ABI (ctypes), as a C caller would."""
    ids = np.ascontiguousarray(np.asarray(chunk_ids, dtype=np.int64))
    assert ids.size >= -(-n // cache.layout.chunk_tokens) and block_table.numel() >= -(-n // cache.layout.block_size)
    fn = kvx._lib.kv_load_noalloc
    fn.argtypes = [ctypes.POINTER(kvx.KvCache), ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_void_p]
    fn.restype = ctypes.c_int32
    st = fn(ctypes.byref(cache.struct), ctypes.c_void_p(block_table.data_ptr()), int(n), pool.handle,
            ctypes.c_void_p(ids.ctypes.data), ctypes.c_void_p(stream.cuda_stream))
    if st != kvx.KV_OK:
        raise kvx.KvError(st, kvx.kv_last_error())


@pytest.mark.parametrize("mode", ["staged", "zero_copy"])
def test_noalloc_matches_kv_load_tiny(mode):
    """Tiny layout: a 17-chunk restore with a partial chunk and shuffled slots, then a smaller
    4-chunk restore into other blocks; both equal kv_load's result and the oracle's."""
    lay, NB = TINY, 512
    seed = harness.sub_seed("noalloc", "tiny")
    A = host_cache(lay, NB, seed, "raw")
    n_store = 4096 + 192
    nc = lay.nc(n_store)
    cid = harness.chunk_ids(nc, nc + 3, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, nc + 3, mode)
    kvx.pool_view(pool)[:] = 0xA5
    dA = to_device(A)
    s = torch.cuda.Stream()
    btA = harness.block_table(seed + 1, NB, lay.nblk(n_store))
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), bt_tensor(btA), n_store, pool, cid, s)
    s.synchronize()
    want_pool = oracle_pool(lay, A, btA, n_store, cid, nc + 3, 0xA5)
    for call, n in enumerate((n_store, 1000)):
        btB = harness.block_table(seed + 10 + call, NB, lay.nblk(n))
        tB = bt_tensor(btB)
        ids = cid[:lay.nc(n)]
        ref = torch.empty_like(dA)
        got = torch.empty_like(dA)
        ref.view(torch.uint8).fill_(SENT)
        got.view(torch.uint8).fill_(SENT)
        torch.cuda.synchronize()
        kvx.kv_load(kvx.Cache(ref, lay.kv, NB), tB, n, pool, ids, s)
        _noalloc(kvx.Cache(got, lay.kv, NB), tB, n, pool, ids, s)
        s.synchronize()
        assert torch.equal(got, ref), f"call {call} (n={n}): kv_load_noalloc differs from kv_load"
        B0 = np.zeros_like(A)
        B0.view(np.uint8)[:] = SENT
        want = oracle_unpack_into(lay, B0, btB, n, want_pool[:], ids)
        g = to_host(got, A)
        assert np.array_equal(g, want), f"call {call}: " + first_mismatch(g, want)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


def test_noalloc_matches_kv_load_27b():
    """27B-class layout (one 64 MiB chunk fills the scratch): a 33-chunk restore with a 192-token
    partial chunk, then a 9-chunk restore into another block set; both equal kv_load's result."""
    lay, NB = B27, 1024
    seed = harness.sub_seed("noalloc", "27b")
    n_store = 32 * 256 + 192
    nc = lay.nc(n_store)
    A = torch.empty((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
    hg.fill_values(A, 0, seed, "n01", 2)
    pool = kvx.kv_pool_create(lay.kv, nc, "staged")
    ids = harness.chunk_ids(nc, nc, seed + 3)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(A, lay.kv, NB), bt_tensor(harness.block_table(seed + 1, NB, lay.nblk(n_store))), n_store,
                 pool, ids, s)
    s.synchronize()
    for call, n in enumerate((n_store, 8 * 256 + 100)):
        tB = bt_tensor(harness.block_table(seed + 10 + call, NB, lay.nblk(n)))
        ref = torch.full_like(A, 0x5A5A)
        got = torch.full_like(A, 0x5A5A)
        torch.cuda.synchronize()
        kvx.kv_load(kvx.Cache(ref, lay.kv, NB), tB, n, pool, ids[:lay.nc(n)], s)
        _noalloc(kvx.Cache(got, lay.kv, NB), tB, n, pool, ids[:lay.nc(n)], s)
        s.synchronize()
        assert torch.equal(got, ref), f"call {call} (n={n}): kv_load_noalloc differs from kv_load"
        del ref, got
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("i", range(24))
def test_noalloc_random_layouts(i):
    """Seeded random layouts (the random-layout parity cases' generator: 1-5 layers, 1-8 heads,
    16-128-byte rows of 1-, 2- and 4-byte elements, 1-32-token blocks, packed and padded strides,
    both block orders, partial chunks, shuffled ids), the pool filled with the CPU oracle's packed
    bytes: a restore of the whole prefix, then a shorter one into another cache; each equals the
    oracle's cache bytes, sentinels included."""
    from tests.test_gpu_fuzz import ORDERS, _case
    lay, n, NB, stride, order, num_slots, _ = _case(i)
    mode = ("staged", "zero_copy")[i % 2]
    print(f"[noalloc] case {i} {mode}: L{lay.L} H{lay.H} D{lay.D} E{lay.E} BS{lay.BS} C{lay.C} n={n} NB={NB} "
          f"stride={stride} order={order} slots={num_slots}", flush=True)
    seed = harness.sub_seed("noalloc-fuzz", i)
    rng = np.random.default_rng(seed)
    A = [rng.integers(0, 256, NB * stride, dtype=np.uint8) for _ in range(lay.L)]
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    ids = harness.chunk_ids(lay.nc(n), num_slots, seed + 3)
    want_pool = np.full(num_slots * lay.slot_bytes, 0xA5, dtype=np.uint8)
    assert oracle.pack(lay.orc, A, stride, NB, btA, n, want_pool, ids, 4, block_order=ORDERS[order]) == oracle.OK
    pool = kvx.kv_pool_create(lay.kv, num_slots, mode)
    kvx.pool_view(pool)[:] = want_pool
    s = torch.cuda.Stream()
    for call, m in enumerate((n, max(1, n // 3))):
        btB = harness.block_table(seed + 10 + call, NB, lay.nblk(m))
        want = [np.full(NB * stride, SENT, dtype=np.uint8) for _ in range(lay.L)]
        assert oracle.unpack(lay.orc, want, stride, NB, btB, m, want_pool, ids[:lay.nc(m)], 4,
                             block_order=ORDERS[order]) == oracle.OK
        dB = [torch.full((NB * stride,), SENT, dtype=torch.uint8, device=DEV) for _ in range(lay.L)]
        torch.cuda.synchronize()
        _noalloc(kvx.Cache(dB, lay.kv, NB, stride, order), bt_tensor(btB), m, pool, ids[:lay.nc(m)], s)
        s.synchronize()
        for l in range(lay.L):
            got = dB[l].cpu().numpy()
            assert np.array_equal(got, want[l]), f"call {call} (n={m}) layer {l}: " + first_mismatch(got, want[l])
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


def test_noalloc_refuses_what_it_cannot_do():
    """A chunk larger than the static scratch is KV_EUNSUPPORTED; a device pool is KV_EINVAL; both
    before anything is enqueued."""
    big = kvx.make_layout(64, 8, 128, 2, 16, 512)        # 128 MiB chunks
    pool = kvx.kv_pool_create(big, 1, "zero_copy")
    t = torch.zeros((1, 2, 8, 16, 128), dtype=torch.int16, device=DEV)
    cache = kvx.Cache([t] * 64, big, 1)
    s = torch.cuda.Stream()
    with pytest.raises(kvx.KvError) as e:
        _noalloc(cache, torch.zeros(32, dtype=torch.int32, device=DEV), 16, pool, [0], s)
    assert e.value.status == kvx.KV_EUNSUPPORTED
    kvx.kv_pool_destroy(pool)
    dpool = kvx.kv_pool_create(TINY.kv, 2, "zero_copy", host_kind=kvx.KV_POOL_DEVICE)
    c = kvx.Cache(torch.zeros((2, 8, 2, 2, 16, 64), dtype=torch.int16, device=DEV), TINY.kv, 8)
    with pytest.raises(kvx.KvError) as e:
        _noalloc(c, torch.zeros(8, dtype=torch.int32, device=DEV), 16, dpool, [0], s)
    assert e.value.status == kvx.KV_EINVAL
    kvx.kv_pool_destroy(dpool)


def test_noalloc_replays_under_graph_capture():
    """The callers this entry point is for include code under graph capture: the restore is captured
    into a HIP graph and replayed three times, with eager work and synchronisation between the
    replays; every replay must leave exactly kv_load's result (checked after each replay)."""
    lay, NB = TINY, 512
    seed = harness.sub_seed("noalloc", "graph")
    A = host_cache(lay, NB, seed, "raw")
    n = 4096 + 192
    nc = lay.nc(n)
    cid = harness.chunk_ids(nc, nc + 2, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, nc + 2, "staged")
    dA = to_device(A)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), bt_tensor(harness.block_table(seed + 1, NB, lay.nblk(n))), n, pool, cid, s)
    tB = bt_tensor(harness.block_table(seed + 2, NB, lay.nblk(n)))
    ref = torch.empty_like(dA)
    ref.view(torch.uint8).fill_(SENT)
    got = torch.empty_like(dA)
    other = torch.empty_like(dA)
    cache_got = kvx.Cache(got, lay.kv, NB)
    torch.cuda.synchronize()
    kvx.kv_load(kvx.Cache(ref, lay.kv, NB), tB, n, pool, cid, s)
    _noalloc(cache_got, tB, n, pool, cid, s)  # first call on the device (address lookup) outside the capture
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        _noalloc(cache_got, tB, n, pool, cid, s)
    t_other = bt_tensor(harness.block_table(seed + 4, NB, lay.nblk(n)))
    for rep in range(3):
        got.view(torch.uint8).fill_(SENT)
        # Eager work of the program between replays: a restore of the same chunks elsewhere.
        kvx.kv_load(kvx.Cache(other, lay.kv, NB), t_other, n, pool, cid, s)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"replay {rep}: the captured restore differs from kv_load"
    assert kvx.kv_pool_async_error(pool) == 0
    del g
    kvx.kv_pool_destroy(pool)

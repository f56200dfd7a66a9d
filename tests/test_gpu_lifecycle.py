"""Pool lifecycle and concurrency on the GPU.

* kv_pool_destroy waits for every store/load still queued on caller streams (they
  write the pool or its staging), so freeing the pool never races with the device; and
  creating and destroying pools leaves later allocations of the process intact.
* Two host threads, each with its own stream and cache, use one pool at the same
  time (both storing, or one storing while the other loads): the pool serialises
  enqueues and its staging ring stays ordered across streams.
"""
import threading
import time

import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import (DEV, TINY, bt_tensor, device_cache, first_mismatch, host_cache, oracle_pool,
                               oracle_unpack_into, to_device, to_host)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_destroy_waits_for_queued_work(mode):
    lay, NB, n = TINY, 512, 4096
    seed = harness.sub_seed("destroy", mode)
    A = host_cache(lay, NB, seed, "u11")
    bt = bt_tensor(harness.block_table(seed + 1, NB, lay.nblk(n)))
    dA = to_device(A)
    pool = kvx.kv_pool_create(lay.kv, 16, mode, staging_slots=2, chunks_per_batch=2)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    hg.spin(300.0, s)
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), bt, n, pool, np.arange(16), s)
    t0 = time.perf_counter()
    kvx.kv_pool_destroy(pool)
    waited = time.perf_counter() - t0
    assert s.query(), "the store was still queued after the pool was destroyed"
    assert waited > 0.15, f"destroy returned after {waited:.3f} s, before the queued store ran"


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_two_threads_share_one_pool(mode):
    """Thread k stores chunks [8k, 8k+8) of its own prefix copy into one pool; afterwards the pool
    holds exactly what the oracle stores for the whole prefix."""
    lay, NB, n = TINY, 512, 4096
    seed = harness.sub_seed("threads", mode)
    A = host_cache(lay, NB, seed, "raw")
    bt = harness.block_table(seed + 1, NB, lay.nblk(n))
    pool = kvx.kv_pool_create(lay.kv, 16, mode, staging_slots=2, chunks_per_batch=1)
    view = kvx.pool_view(pool)
    view[:] = 0
    dA = [to_device(A), to_device(A)]
    caches = [kvx.Cache(d, lay.kv, NB) for d in dA]
    half = n // 2
    tables = [bt_tensor(bt[:half // lay.BS]), bt_tensor(bt[half // lay.BS:])]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    errors = []

    def worker(k):
        try:
            for _ in range(5):
                hg.spin(2.0, streams[k])
                kvx.kv_store(caches[k], tables[k], half, pool, np.arange(8 * k, 8 * k + 8), streams[k])
            streams[k].synchronize()
        except Exception as e:  # surfaced below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    want = oracle_pool(lay, A, bt, n, np.arange(16), 16, 0)
    assert np.array_equal(view, want)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged", "staged+zero_copy"])
def test_one_thread_stores_while_another_loads(mode):
    """Thread 0 stores chunks 0-7 of replica A's prefix again and again while thread 1 restores
    chunks 8-15 (stored beforehand) into replica B, each on its own stream, through one pool with a
    two-slot ring of one chunk per batch.  Afterwards the pool and B equal the oracle's bytes."""
    store_mode, load_mode = (mode.split("+") * 2)[:2]
    lay, NB, n = TINY, 512, 4096
    seed = harness.sub_seed("store-while-load", mode)
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    pool = kvx.kv_pool_create(lay.kv, 16, "staged", staging_slots=2, chunks_per_batch=1)
    kvx.kv_pool_set_modes(pool, store_mode, load_mode)
    view = kvx.pool_view(pool)
    view[:] = 0
    dA, dB = to_device(A), device_cache(lay, NB, fill=0x5A)
    cA, cB = kvx.Cache(dA, lay.kv, NB), kvx.Cache(dB, lay.kv, NB)
    half, hb = n // 2, n // 2 // lay.BS
    tA_lo, tA_hi, tB_hi = bt_tensor(btA[:hb]), bt_tensor(btA[hb:]), bt_tensor(btB[hb:])
    torch.cuda.synchronize()
    kvx.kv_store(cA, tA_hi, half, pool, np.arange(8, 16))  # the chunks thread 1 restores
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    errors = []

    def worker(k):
        try:
            for _ in range(8):
                hg.spin(1.0, streams[k])
                if k == 0:
                    kvx.kv_store(cA, tA_lo, half, pool, np.arange(8), streams[0])
                else:
                    kvx.kv_load(cB, tB_hi, half, pool, np.arange(8, 16), streams[1])
            streams[k].synchronize()
        except Exception as e:  # surfaced below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    want_pool = oracle_pool(lay, A, btA, n, np.arange(16), 16, 0)
    assert np.array_equal(view, want_pool), "pool: " + first_mismatch(view, want_pool)
    B0 = np.full_like(A, 0).view(np.uint8)
    B0[:] = 0x5A
    want_B = oracle_unpack_into(lay, B0.view(A.dtype).reshape(A.shape), btB[hb:], half, want_pool[8 * lay.slot_bytes:],
                                np.arange(8))
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


def test_pool_churn_leaves_later_allocations_intact():
    """Staged pools of varying staging size are created and destroyed 40 times, with fresh tensors
    allocated between them.  Every fresh tensor reads back the value just written to it, and every
    round trip equals the oracle's bytes.  Freeing a physically contiguous staging allocation once
    corrupted later allocations of the process; staging is plain device memory now."""
    lay, NB = TINY, 96
    for it in range(40):
        seed = harness.sub_seed("churn", it)
        n = 256 * (1 + it % 3) + 7 * it
        A = host_cache(lay, NB, seed, "raw")
        btA = harness.block_table(seed + 1, NB, lay.nblk(n))
        btB = harness.block_table(seed + 2, NB, lay.nblk(n))
        ids = harness.chunk_ids(lay.nc(n), lay.nc(n) + 1, seed + 3)
        pool = kvx.kv_pool_create(lay.kv, lay.nc(n) + 1, "staged", staging_slots=2, chunks_per_batch=1 + it % 3)
        view = kvx.pool_view(pool)
        view[:] = 0xA5
        probe = torch.full((1 << 20,), it % 251, dtype=torch.uint8, device=DEV)
        dA, dB = to_device(A), device_cache(lay, NB, fill=0x5A)
        tA, tB = bt_tensor(btA), bt_tensor(btB)
        torch.cuda.synchronize()
        assert bool((probe == it % 251).all()) and int(probe.cpu().numpy().min()) == it % 251, f"iteration {it}"
        s = torch.cuda.Stream()
        torch.cuda.synchronize()
        kvx.kv_store(kvx.Cache(dA, lay.kv, NB), tA, n, pool, ids, s)
        kvx.kv_load(kvx.Cache(dB, lay.kv, NB), tB, n, pool, ids, s)
        s.synchronize()
        want_pool = oracle_pool(lay, A, btA, n, ids, lay.nc(n) + 1, 0xA5)
        assert np.array_equal(view, want_pool), f"iteration {it}, pool: " + first_mismatch(view, want_pool)
        B0 = np.full_like(A, 0).view(np.uint8)
        B0[:] = 0x5A
        want_B = oracle_unpack_into(lay, B0.view(A.dtype).reshape(A.shape), btB, n, want_pool, ids)
        got_B = to_host(dB, A)
        assert np.array_equal(got_B, want_B), f"iteration {it}, cache B: " + first_mismatch(got_B, want_B)
        kvx.kv_pool_destroy(pool)
        del dA, dB, tA, tB, probe


def test_many_short_lived_streams():
    """A store on each of 40 fresh streams: every one is ordered and the pool stays usable; streams
    whose work completed do not accumulate in the pool."""
    lay, NB, n = TINY, 512, 1024
    seed = harness.sub_seed("streams")
    A = host_cache(lay, NB, seed, "raw")
    bt = harness.block_table(seed + 1, NB, lay.nblk(n))
    pool = kvx.kv_pool_create(lay.kv, lay.nc(n), "staged", staging_slots=2, chunks_per_batch=2)
    view = kvx.pool_view(pool)
    dA = to_device(A)
    cache = kvx.Cache(dA, lay.kv, NB)
    tb = bt_tensor(bt)
    torch.cuda.synchronize()
    for _ in range(40):
        s = torch.cuda.Stream()
        view[:] = 0
        kvx.kv_store(cache, tb, n, pool, np.arange(lay.nc(n)), s)
        s.synchronize()
        del s
    want = oracle_pool(lay, A, bt, n, np.arange(lay.nc(n)), lay.nc(n), 0)
    assert np.array_equal(view, want)
    kvx.kv_pool_destroy(pool)

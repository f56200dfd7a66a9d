"""Pool lifecycle and concurrency on the GPU.

* kv_pool_destroy waits for every store/load still queued on caller streams (they
  write the pool or its staging), so freeing the pool never races with the device.
* Two host threads, each with its own stream and cache, use one pool at the same
  time: the pool serialises enqueues and its staging ring stays ordered across streams.
"""
import threading
import time

import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import TINY, bt_tensor, host_cache, oracle_pool, to_device

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

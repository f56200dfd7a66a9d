"""Stream ordering through kv_store / kv_load: the paper's byte probes (Sec. 3.2).

Store: a delayed producer on the caller's stream writes byte 37 into the cache,
then kv_store runs on that stream; after the host synchronises the stream, every
stored byte must be 37 (the unordered fault delivers the old 0).  Load: a
delayed consumer on the stream reads the destination cache's old value 0, then
kv_load writes 53 from the pool; the consumer must still see 0.  Sizes follow
the paper's 4 KiB / 1 MiB / 16 MiB objects (4 / 1,024 / 16,384 tokens of the
1 KiB-per-token tiny layout), with no delay and with a seeded 5-50 ms delay.
"""
import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import DEV, TINY, bt_tensor, device_cache

pytestmark = pytest.mark.gpu

SIZES_TOKENS = (4, 1024, 16384)
TRIALS = 10


def _make_stream(kind):
    if kind == "torch":
        return torch.cuda.Stream(), None
    if kind == "nonblocking":
        s = hg.RawStream(True)
        return int(s), s
    if kind == "blocking":
        s = hg.RawStream(False)
        return int(s), s
    return 0, None  # the null stream


def _sync(stream):
    if isinstance(stream, torch.cuda.Stream):
        stream.synchronize()
    else:
        torch.cuda.synchronize()


def _named_slot_mask(lay, NB, bt, n):
    m = np.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=bool)
    t = np.arange(n)
    m[:, bt[t // lay.BS], :, :, t % lay.BS, :] = True
    return m


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("stream_kind", ["torch", "nonblocking", "blocking", "null"])
def test_store_probe_37(mode, stream_kind):
    lay = TINY
    delays = harness.spin_delays_ms(harness.sub_seed("order-store", mode, stream_kind), 100)
    stream, owner = _make_stream(stream_kind)
    k = 0
    fails = []
    for n in SIZES_TOKENS:
        NB = lay.nblk(n) + 8
        bt = harness.block_table(harness.sub_seed("bt", n), NB, lay.nblk(n))
        tb = bt_tensor(bt)
        nc = lay.nc(n)
        pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=4)
        view = kvx.pool_view(pool)
        dA = device_cache(lay, NB, fill=0)
        cA = kvx.Cache(dA, lay.kv, NB)
        payload = n * lay.token_bytes
        for delayed in (False, True):
            for _ in range(TRIALS):
                dA.zero_()
                view[:] = 0
                torch.cuda.synchronize()
                if delayed:
                    hg.spin(float(delays[k]), stream)
                    k += 1
                hg.fill_u8(dA, dA.numel() * dA.element_size(), 37, stream)
                kvx.kv_store(cA, tb, n, pool, np.arange(nc), stream)
                _sync(stream)
                got = np.concatenate([view[i * lay.slot_bytes:i * lay.slot_bytes + min(lay.C, n - i * lay.C)
                                           * lay.token_bytes] for i in range(nc)])
                assert got.size == payload
                fails.append((n, delayed, int(np.count_nonzero(got != 37))))
        kvx.kv_pool_destroy(pool)
    if owner is not None:
        owner.close()
    bad = [f for f in fails if f[2]]
    assert not bad, f"{len(bad)} of {len(fails)} store probes saw stale bytes: {bad[:5]}"
    assert len(fails) == len(SIZES_TOKENS) * 2 * TRIALS


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("stream_kind", ["torch", "nonblocking", "blocking", "null"])
def test_load_probe_53(mode, stream_kind):
    lay = TINY
    delays = harness.spin_delays_ms(harness.sub_seed("order-load", mode, stream_kind), 100)
    stream, owner = _make_stream(stream_kind)
    k = 0
    fails = []
    for n in SIZES_TOKENS:
        NB = lay.nblk(n) + 8
        bt = harness.block_table(harness.sub_seed("btB", n), NB, lay.nblk(n))
        tb = bt_tensor(bt)
        nc = lay.nc(n)
        pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=4)
        view = kvx.pool_view(pool)
        dB = device_cache(lay, NB, fill=0)
        probe = torch.empty_like(dB)
        cB = kvx.Cache(dB, lay.kv, NB)
        mask = _named_slot_mask(lay, NB, bt, n).reshape(-1)
        nbytes = dB.numel() * dB.element_size()
        for delayed in (False, True):
            for _ in range(TRIALS):
                dB.zero_()
                probe.view(torch.uint8).fill_(0xEE)
                view[:] = 53
                torch.cuda.synchronize()
                if delayed:
                    hg.spin(float(delays[k]), stream)
                    k += 1
                hg.copy_u8(probe, dB, nbytes, stream)  # delayed consumer of the old value
                kvx.kv_load(cB, tb, n, pool, np.arange(nc), stream)
                _sync(stream)
                seen = probe.view(torch.uint8).cpu().numpy().reshape(-1)
                after = dB.view(torch.uint8).cpu().numpy().reshape(-1)
                elem_mask = np.repeat(mask, lay.E)
                stale = int(np.count_nonzero(seen != 0))
                wrong = int(np.count_nonzero(after[elem_mask] != 53)) + int(np.count_nonzero(after[~elem_mask]))
                fails.append((n, delayed, stale, wrong))
        kvx.kv_pool_destroy(pool)
    if owner is not None:
        owner.close()
    bad = [f for f in fails if f[2] or f[3]]
    assert not bad, f"{len(bad)} of {len(fails)} load probes failed: {bad[:5]}"


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_store_then_load_same_stream_no_host_sync(mode):
    """A store followed by a load on one stream, with a delayed producer before the store and no
    host synchronisation in between: the load must see the stored bytes (pool RAW across the
    staged mode's side streams)."""
    lay, n = TINY, 4096 + 64
    NB = 600
    btA = harness.block_table(harness.sub_seed("rawA"), NB, lay.nblk(n))
    btB = harness.block_table(harness.sub_seed("rawB"), NB, lay.nblk(n))
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    nc = lay.nc(n)
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=2)
    dA = device_cache(lay, NB, fill=0)
    dB = device_cache(lay, NB, fill=0)
    cA, cB = kvx.Cache(dA, lay.kv, NB), kvx.Cache(dB, lay.kv, NB)
    s = torch.cuda.Stream()
    delays = harness.spin_delays_ms(harness.sub_seed("raw-delay", mode), 10)
    mask = np.repeat(_named_slot_mask(lay, NB, btB, n).reshape(-1), lay.E)
    for trial in range(10):
        value = 100 + trial
        hg.spin(float(delays[trial]), s)
        hg.fill_u8(dA, dA.numel() * dA.element_size(), value, s)
        kvx.kv_store(cA, tA, n, pool, np.arange(nc), s)
        kvx.kv_load(cB, tB, n, pool, np.arange(nc), s)
        s.synchronize()
        after = dB.view(torch.uint8).cpu().numpy().reshape(-1)
        assert np.all(after[mask] == value), f"trial {trial}: load did not see the store"
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_cross_stream_store_then_load_ordered_by_event(mode):
    """Replica A stores on its stream, replica B loads on another; the caller orders them with an
    event (the host-side completion handling of Sec. 3.2 / Fig. 2, done on the device)."""
    lay, n = TINY, 2048
    NB = 300
    btA = harness.block_table(harness.sub_seed("xA"), NB, lay.nblk(n))
    btB = harness.block_table(harness.sub_seed("xB"), NB, lay.nblk(n))
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    nc = lay.nc(n)
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=2)
    dA = device_cache(lay, NB, fill=0)
    dB = device_cache(lay, NB, fill=0)
    cA, cB = kvx.Cache(dA, lay.kv, NB), kvx.Cache(dB, lay.kv, NB)
    sA, sB = torch.cuda.Stream(), torch.cuda.Stream()
    mask = np.repeat(_named_slot_mask(lay, NB, btB, n).reshape(-1), lay.E)
    for trial in range(5):
        hg.spin(20.0, sA)
        hg.fill_u8(dA, dA.numel() * dA.element_size(), 7 + trial, sA)
        kvx.kv_store(cA, tA, n, pool, np.arange(nc), sA)
        ev = torch.cuda.Event()
        ev.record(sA)
        sB.wait_event(ev)
        kvx.kv_load(cB, tB, n, pool, np.arange(nc), sB)
        sB.synchronize()
        after = dB.view(torch.uint8).cpu().numpy().reshape(-1)
        assert np.all(after[mask] == 7 + trial)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_random_interleavings_keep_each_stream_ordered(mode):
    """Three streams share one pool whose staging ring has two one-chunk slots, so their batches
    reuse each other's staging.  Each round, in a seeded order with seeded 0-4 ms delays, every
    stream fills its own source cache with a new byte, stores it into its own slots, restores them
    into its own destination, and copies the destination aside, all on that stream.  Every copy
    must hold that round's byte in every named slot and the sentinel elsewhere: each stream's
    fill -> store -> load -> read chain stays ordered whatever the other streams do."""
    lay, NB, n, rounds = TINY, 64, 3 * TINY.C, 12
    rng = np.random.default_rng(harness.sub_seed("interleave", mode))
    nc = lay.nc(n)
    pool = kvx.kv_pool_create(lay.kv, 3 * nc, mode, staging_slots=2, chunks_per_batch=1)
    streams = [torch.cuda.Stream() for _ in range(3)]
    A = [device_cache(lay, NB, fill=0) for _ in range(3)]
    B = [device_cache(lay, NB, fill=0xEE) for _ in range(3)]
    bts = [(harness.block_table(int(rng.integers(1 << 30)), NB, lay.nblk(n)),
            harness.block_table(int(rng.integers(1 << 30)), NB, lay.nblk(n))) for _ in range(3)]
    tabs = [(bt_tensor(a), bt_tensor(b)) for a, b in bts]
    slots = [np.arange(k * nc, (k + 1) * nc) for k in range(3)]
    nbytes = A[0].numel() * A[0].element_size()
    snaps = {}
    torch.cuda.synchronize()
    for r in range(rounds):
        for k in rng.permutation(3):
            s, v = streams[k], int(1 + (r * 3 + k) % 200)
            hg.spin(float(rng.uniform(0, 4)), s)
            hg.fill_u8(A[k], nbytes, v, s)
            kvx.kv_store(kvx.Cache(A[k], lay.kv, NB), tabs[k][0], n, pool, slots[k], s)
            hg.spin(float(rng.uniform(0, 2)), s)
            kvx.kv_load(kvx.Cache(B[k], lay.kv, NB), tabs[k][1], n, pool, slots[k], s)
            snap = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
            hg.copy_u8(snap, B[k], nbytes, s)
            snaps[(r, k)] = (snap, v)
    for s in streams:
        s.synchronize()
    masks = [_named_slot_mask(lay, NB, bts[k][1], n).reshape(-1) for k in range(3)]
    for (r, k), (snap, v) in sorted(snaps.items()):
        got = snap.cpu().numpy().view(np.uint8).reshape(-1)
        m = np.repeat(masks[k], lay.E)
        assert (got[m] == v).all(), f"round {r} stream {k}: {int((got[m] != v).sum())} named bytes not {v}"
        assert (got[~m] == 0xEE).all(), f"round {r} stream {k}: bytes outside the named slots changed"
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)

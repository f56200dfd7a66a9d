"""GPU parity for recurrent-state snapshot pages (Sec. 2.2) and their ordering.

Expected bytes come from the oracle's state pack/unpack applied to the same host-generated
pages.  Cases cover snapshots smaller and larger than one staging slot, pages that are not a
whole number of 16 KiB pieces, more snapshots than one launch carries, the maximum layer count,
and a page geometry of a 27B-class hybrid model's recurrent layer.
"""
import numpy as np
import pytest
import torch

import harness
import oracle
from harness import gpu as hg
from oracle.recovery import KV, STATE, restorable_chunks
from paper_2609_15021_amd import kvx
from tests.gpu_support import DEV, TINY, bt_tensor, first_mismatch, host_cache, layers_of, oracle_pool, \
    oracle_unpack_into, to_device, to_host

pytestmark = pytest.mark.gpu

STATE_SENT, CHUNK_SENT, PAGE_SENT = 0xA5, 0x11, 0x5A
# Recurrent page of a GDN layer with 48 value heads of 128x128 fp32 state plus a 3-step
# convolution state over 10,240 bf16 channels: 3 MiB + 60 KiB (the paper gives no sizes).
GDN_PAGE = 3 * 1024 * 1024 + 3 * 10240 * 2

CASES = {  # G, page_bytes, page_stride, num_pages, n, chunks_per_batch
    "small": (3, 4096, 4096 + 256, 10, 4, 2),
    "split-snapshot": (5, 100 * 1024, 100 * 1024 + 64, 6, 3, 1),
    "many-snapshots": (2, 256, 256, 400, 300, 1),
    "max-layers-16B-pages": (64, 16, 48, 5, 5, 1),
    "gdn-27b-class": (48, GDN_PAGE, GDN_PAGE, 3, 2, 16),
}


def _pages(seed, G, num_pages, stride):
    return np.random.default_rng(seed).integers(0, 256, size=(G, num_pages, stride), dtype=np.uint8)


def _layers(A):
    return [np.ascontiguousarray(A[g]).reshape(-1) for g in range(A.shape[0])]


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_state_round_trip(mode, case):
    G, pb, stride, npages, n, cpb = CASES[case]
    seed = harness.sub_seed("state", case, mode)
    rng = np.random.default_rng(seed + 1)
    A = _pages(seed, G, npages, stride)
    pagesA = rng.permutation(npages)[:n]
    pagesB = rng.permutation(npages)[:n]
    nslots = n + 2
    slots = rng.permutation(nslots)[:n]
    pool = kvx.kv_pool_create(TINY.kv, 2, mode, staging_slots=2, chunks_per_batch=cpb, num_state_slots=nslots,
                              state_slot_bytes=G * pb)
    sview, cview = kvx.state_view(pool), kvx.pool_view(pool)
    sview[:] = STATE_SENT
    cview[:] = CHUNK_SENT
    dA = torch.from_numpy(A).to(DEV)
    dB = torch.full_like(dA, PAGE_SENT)
    stA = kvx.State(dA, pb, npages, stride)
    stB = kvx.State(dB, pb, npages, stride)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store_state(stA, pagesA, pool, slots, s)
    kvx.kv_load_state(stB, pagesB, pool, slots, s)
    s.synchronize()
    want_pool = np.full(nslots * G * pb, STATE_SENT, dtype=np.uint8)
    assert oracle.state_pack(_layers(A), pb, stride, pagesA, want_pool, slots) == oracle.OK
    assert np.array_equal(sview, want_pool), first_mismatch(sview, want_pool)
    assert (cview == CHUNK_SENT).all(), "a state transfer wrote into the chunk slots"
    B = np.full_like(A, PAGE_SENT)
    layersB = _layers(B)
    assert oracle.state_unpack(layersB, pb, stride, pagesB, want_pool, slots) == oracle.OK
    want_B = np.stack([x.reshape(npages, stride) for x in layersB])
    got_B = dB.cpu().numpy()
    assert np.array_equal(got_B, want_B), first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_state_store_probe_37_and_load_probe_53(mode):
    """Sec. 3.2's probes on snapshot pages: a delayed producer writes 37 before the store, and a
    delayed consumer reads the old 0 before the load writes 53."""
    G, pb, npages = 4, 256 * 1024, 2  # 1 MiB per snapshot, the paper's mid-size probe
    delays = harness.spin_delays_ms(harness.sub_seed("state-order", mode), 20)
    pool = kvx.kv_pool_create(TINY.kv, 1, mode, staging_slots=2, chunks_per_batch=1, num_state_slots=1,
                              state_slot_bytes=G * pb)
    sview = kvx.state_view(pool)
    dS = torch.zeros((G, npages, pb), dtype=torch.uint8, device=DEV)
    probe = torch.empty_like(dS)
    st = kvx.State(dS, pb, npages)
    s = torch.cuda.Stream()
    fails = []
    for trial in range(10):
        dS.zero_()
        sview[:] = 0
        torch.cuda.synchronize()
        hg.spin(float(delays[2 * trial]), s)
        hg.fill_u8(dS, dS.numel(), 37, s)
        kvx.kv_store_state(st, [1], pool, [0], s)
        s.synchronize()
        fails.append(("store", trial, int(np.count_nonzero(sview != 37))))

        dS.zero_()
        probe.fill_(0xEE)
        sview[:] = 53
        torch.cuda.synchronize()
        hg.spin(float(delays[2 * trial + 1]), s)
        hg.copy_u8(probe, dS, dS.numel(), s)
        kvx.kv_load_state(st, [0], pool, [0], s)
        s.synchronize()
        seen, after = probe.cpu().numpy(), dS.cpu().numpy()
        fails.append(("load", trial, int(np.count_nonzero(seen != 0)) + int(np.count_nonzero(after[:, 0] != 53)) +
                      int(np.count_nonzero(after[:, 1]))))
    kvx.kv_pool_destroy(pool)
    bad = [f for f in fails if f[2]]
    assert not bad, f"{len(bad)} of {len(fails)} probes failed: {bad[:5]}"


def test_state_calls_need_a_state_area():
    pool = kvx.kv_pool_create(TINY.kv, 2, "staged")
    d = torch.zeros((1, 2, 64), dtype=torch.uint8, device=DEV)
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_store_state(kvx.State(d, 64, 2), [0], pool, [0])
    assert e.value.status == kvx.KV_EINVAL and "state area" in str(e.value)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_hybrid_session_aligned_recovery(mode):
    """Replica A stores all chunks of a prefix but snapshots only at two chunk boundaries.  Under
    aligned recovery (Sec. 2.2) replica B restores the longest prefix that has both -- here 4 of
    the 6 chunks -- loading those chunks and the snapshot at their boundary, and gets A's bytes."""
    lay = TINY
    n = 5 * lay.C + 100
    nc = lay.nc(n)
    G, pb, npages = 3, 8192, 8
    seed = harness.sub_seed("hybrid", mode)
    NB = lay.nblk(n) + 7
    A = host_cache(lay, NB, seed, "raw")
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    SA = _pages(seed + 3, G, npages, pb)
    snap_page_after = {1: 5, 3: 2}   # chunk index -> A's page holding the snapshot after it
    state_slot_of = {1: 0, 3: 1}
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=2, num_state_slots=2,
                              state_slot_bytes=G * pb)
    dA, dSA = to_device(A), torch.from_numpy(SA).to(DEV)
    dB = torch.zeros_like(dA)
    dSB = torch.zeros_like(dSA)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), bt_tensor(btA), n, pool, np.arange(nc), s)
    chunks = sorted(snap_page_after)
    kvx.kv_store_state(kvx.State(dSA, pb, npages), [snap_page_after[i] for i in chunks], pool,
                       [state_slot_of[i] for i in chunks], s)
    s.synchronize()  # host-side completion before the pool is published (Sec. 3.2)

    flags = [KV | (STATE if i in snap_page_after else 0) for i in range(nc)]
    k = restorable_chunks(flags, require_state=True)
    assert k == 4
    n_restore = k * lay.C
    page_B = 6
    kvx.kv_load(kvx.Cache(dB, lay.kv, NB), bt_tensor(btB[:lay.nblk(n_restore)]), n_restore, pool, np.arange(k), s)
    kvx.kv_load_state(kvx.State(dSB, pb, npages), [page_B], pool, [state_slot_of[k - 1]], s)
    s.synchronize()

    want_pool = oracle_pool(lay, A, btA, n, np.arange(nc), nc, 0)
    want_B = oracle_unpack_into(lay, np.zeros_like(A), btB[:lay.nblk(n_restore)], n_restore, want_pool,
                                np.arange(k))
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), first_mismatch(got_B, want_B)
    got_S = dSB.cpu().numpy()
    assert np.array_equal(got_S[:, page_B], SA[:, snap_page_after[k - 1]])
    assert not got_S[:, [p for p in range(npages) if p != page_B]].any()
    kvx.kv_pool_destroy(pool)


def test_state_area_options_are_validated():
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(TINY.kv, 2, "staged", num_state_slots=2, state_slot_bytes=0)
    assert e.value.status == kvx.KV_EINVAL
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(TINY.kv, 2, "staged", num_state_slots=0, state_slot_bytes=4096)
    assert e.value.status == kvx.KV_EINVAL
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(TINY.kv, 2, "staged", num_state_slots=2, state_slot_bytes=4104)
    assert e.value.status == kvx.KV_EUNSUPPORTED
    pool = kvx.kv_pool_create(TINY.kv, 3, "zero_copy", num_state_slots=2, state_slot_bytes=4096)
    info = kvx.kv_pool_get_info(pool)
    assert info["num_state_slots"] == 2 and info["state_slot_bytes"] == 4096
    # The state area follows the chunk slots in the same pinned region, 4 KiB aligned.
    assert info["state_host_base"] >= info["host_base"] + info["pool_bytes"]
    assert info["state_host_base"] % 4096 == 0
    assert kvx.kv_pool_state_slot(pool, 1) == info["state_host_base"] + 4096
    assert kvx.kv_pool_state_slot(pool, 2) == 0
    kvx.kv_pool_destroy(pool)

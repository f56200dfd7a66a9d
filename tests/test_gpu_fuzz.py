"""Seeded random layouts (and snapshot geometries) through the C ABI, bit-exact against the CPU
oracle.

Each case draws a layout (1-5 layers; 1, 2, 3, 4, 5 or 8 KV heads; 16-128-byte rows of 1-, 2-
or 4-byte elements; 1-32-token blocks; chunks of 1-8 blocks), a packed or padded block stride,
token-major or head-major blocks, a prefix length with partial chunks and blocks, shuffled chunk
ids, a spare slot or two, and a staging ring of 2-3 slots of 1-3 chunks.  Cache bytes are raw
random bytes, one device allocation per layer.  Pool and destination cache must equal the
oracle's bytes, sentinels included.  Non-power-of-two head counts and row widths exercise the
kernels' carry-based index walk; small rings and strided zero-copy grids exercise the engine.

Pools are created and destroyed per case, with tensors allocated in between: this sequence found
that freeing physically contiguous staging corrupted later allocations (now plain device memory).
"""
import numpy as np
import pytest
import torch

import harness
import oracle
from paper_2609_15021_amd import kvx
from tests.gpu_support import DEV, TINY, Layout, bt_tensor, first_mismatch

pytestmark = pytest.mark.gpu

POOL_SENT, CACHE_SENT = 0xA5, 0x5A
ORDERS = {kvx.KV_BLOCK_HND: oracle.BLOCK_HND, kvx.KV_BLOCK_NHD: oracle.BLOCK_NHD}


def _case(i):
    rng = np.random.default_rng(harness.sub_seed("fuzz", i))
    L = int(rng.integers(1, 6))
    H = int(rng.choice([1, 2, 3, 4, 5, 8]))
    E = int(rng.choice([1, 2, 4]))
    row = 16 * int(rng.integers(1, 9))
    BS = int(rng.choice([1, 2, 4, 8, 16, 32]))
    C = BS * int(rng.integers(1, 9))
    lay = Layout(L, H, row // E, E, BS, C)
    n = int(rng.integers(1, 4 * C + 1)) if rng.random() < 0.8 else C * int(rng.integers(1, 5))
    NB = lay.nblk(n) + int(rng.integers(0, 40))
    stride = lay.block_bytes + 16 * int(rng.integers(0, 3))
    order = int(rng.choice([kvx.KV_BLOCK_HND, kvx.KV_BLOCK_NHD]))
    nc = lay.nc(n)
    slots = nc + int(rng.integers(0, 3))
    ring = (int(rng.integers(2, 4)), int(rng.integers(1, 4)))
    return lay, n, NB, stride, order, slots, ring


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("i", range(120))
def test_random_layout_round_trip(i, mode):
    lay, n, NB, stride, order, num_slots, (K, cpb) = _case(i)
    print(f"[fuzz] case {i} {mode}: L{lay.L} H{lay.H} D{lay.D} E{lay.E} BS{lay.BS} C{lay.C} n={n} NB={NB} "
          f"stride={stride} order={order} slots={num_slots} ring={K}x{cpb}", flush=True)
    seed = harness.sub_seed("fuzz-data", i, mode)
    rng = np.random.default_rng(seed)
    A = [rng.integers(0, 256, NB * stride, dtype=np.uint8) for _ in range(lay.L)]
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    ids = harness.chunk_ids(lay.nc(n), num_slots, seed + 3)

    want_pool = np.full(num_slots * lay.slot_bytes, POOL_SENT, dtype=np.uint8)
    assert oracle.pack(lay.orc, A, stride, NB, btA, n, want_pool, ids, 4, block_order=ORDERS[order]) == oracle.OK
    want_B = [np.full(NB * stride, CACHE_SENT, dtype=np.uint8) for _ in range(lay.L)]
    assert oracle.unpack(lay.orc, want_B, stride, NB, btB, n, want_pool, ids, 4,
                         block_order=ORDERS[order]) == oracle.OK

    pool = kvx.kv_pool_create(lay.kv, num_slots, mode, staging_slots=K, chunks_per_batch=cpb)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = [torch.from_numpy(a).to(DEV) for a in A]
    dB = [torch.full((NB * stride,), CACHE_SENT, dtype=torch.uint8, device=DEV) for _ in range(lay.L)]
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB, stride, order), tA, n, pool, ids, s)
    kvx.kv_load(kvx.Cache(dB, lay.kv, NB, stride, order), tB, n, pool, ids, s)
    s.synchronize()
    assert np.array_equal(view, want_pool), "pool: " + first_mismatch(view, want_pool)
    for l in range(lay.L):
        got = dB[l].cpu().numpy()
        assert np.array_equal(got, want_B[l]), f"cache B layer {l}: " + first_mismatch(got, want_B[l])
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


def _state_case(i):
    rng = np.random.default_rng(harness.sub_seed("fuzz-state", i))
    G = int(rng.integers(1, 9)) if rng.random() < 0.85 else 64
    pb = 16 * int(rng.integers(1, 12001)) if rng.random() < 0.7 else 16 * int(rng.integers(1, 9))
    stride = pb + 16 * int(rng.integers(0, 4))
    n = int(rng.integers(1, 41))
    npages = n + int(rng.integers(0, 5))
    nslots = n + int(rng.integers(0, 3))
    cpb = int(rng.integers(1, 4))
    return G, pb, stride, n, npages, nslots, cpb


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("i", range(60))
def test_random_snapshot_round_trip(i, mode):
    """Seeded snapshot geometries (1-8 or 64 recurrent layers, 16-byte to 187.5 KiB pages, padded
    strides, 1-40 snapshots, spare slots): a store that reads some pages twice into distinct slots,
    then a load that reads some slots twice into distinct pages.  State slots, chunk slots and
    destination pages equal the oracle's bytes."""
    G, pb, stride, n, npages, nslots, cpb = _state_case(i)
    print(f"[fuzz-state] case {i} {mode}: G{G} page {pb} stride {stride} n={n} pages={npages} slots={nslots} "
          f"cpb={cpb}", flush=True)
    seed = harness.sub_seed("fuzz-state-data", i, mode)
    rng = np.random.default_rng(seed)
    A = rng.integers(0, 256, size=(G, npages, stride), dtype=np.uint8)
    pages_s = rng.integers(0, npages, n)            # a store may read a page twice
    slots_s = rng.permutation(nslots)[:n]          # ... into distinct slots
    pages_l = rng.permutation(npages)[:n]          # a load writes distinct pages
    slots_l = rng.choice(slots_s, n)               # ... and may read a slot twice
    want_state = np.full(nslots * G * pb, POOL_SENT, dtype=np.uint8)
    assert oracle.state_pack([np.ascontiguousarray(A[g]).reshape(-1) for g in range(G)], pb, stride, pages_s,
                             want_state, slots_s) == oracle.OK
    B = np.full_like(A, CACHE_SENT)
    layers_b = [np.ascontiguousarray(B[g]).reshape(-1) for g in range(G)]
    assert oracle.state_unpack(layers_b, pb, stride, pages_l, want_state, slots_l) == oracle.OK
    want_B = np.stack([x.reshape(npages, stride) for x in layers_b])

    pool = kvx.kv_pool_create(TINY.kv, 1, mode, staging_slots=2, chunks_per_batch=cpb, num_state_slots=nslots,
                              state_slot_bytes=G * pb)
    sview, cview = kvx.state_view(pool), kvx.pool_view(pool)
    sview[:] = POOL_SENT
    cview[:] = 0x11
    dA = torch.from_numpy(A).to(DEV)
    dB = torch.full_like(dA, CACHE_SENT)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store_state(kvx.State(dA, pb, npages, stride), pages_s, pool, slots_s, s)
    kvx.kv_load_state(kvx.State(dB, pb, npages, stride), pages_l, pool, slots_l, s)
    s.synchronize()
    assert np.array_equal(sview, want_state), "state slots: " + first_mismatch(sview, want_state)
    assert (cview == 0x11).all(), "a state transfer wrote into the chunk slots"
    got_B = dB.cpu().numpy()
    assert np.array_equal(got_B, want_B), "pages: " + first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)

"""GPU parity of a device-resident pool (KV_POOL_DEVICE): kv_store packs into device memory and
kv_load unpacks from it, with no host link in the path.  The pool's bytes are read back with a
plain device copy and compared with the CPU oracle's store of the same host-generated inputs;
the restored cache with the oracle's load.  Bit-exact, as for the host pool."""
import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import (B27, DEV, TINY, Layout, bt_tensor, device_cache, first_mismatch, host_cache,
                               oracle_pool, oracle_unpack_into, to_device, to_host)
from tests.test_gpu_fullsize import _oracle_slot

pytestmark = pytest.mark.gpu

POOL_SENT = 0xA5
CACHE_SENT = 0x5A


def _read(ptr: int, nbytes: int, stream) -> np.ndarray:
    out = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    hg.copy_async(out, ptr, nbytes, stream)
    stream.synchronize()
    return out.cpu().numpy()


def _device_round_trip(lay: Layout, NB: int, n: int, seed_tag: str, dist="u11", order=kvx.KV_BLOCK_HND,
                       chunks_per_batch=0, extra_slots=2):
    seed = harness.sub_seed("device-pool", seed_tag, n, lay.L, lay.H, lay.D, lay.E, lay.BS, lay.C)
    A = host_cache(lay, NB, seed, dist)
    if order == kvx.KV_BLOCK_NHD:  # the same tokens in token-major blocks: [L][NB][2][BS][H][D]
        A = np.ascontiguousarray(A.transpose(0, 1, 2, 4, 3, 5))
    nblk, nc = lay.nblk(n), lay.nc(n)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    num_slots = nc + extra_slots
    cid = harness.chunk_ids(nc, num_slots, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, num_slots, "zero_copy", host_kind=kvx.KV_POOL_DEVICE,
                              chunks_per_batch=chunks_per_batch)
    info = kvx.kv_pool_get_info(pool)
    assert info["host_base"] is None and info["is_pinned"] == 0 and kvx.kv_pool_slot(pool, 0) == 0
    s = torch.cuda.Stream()
    hg.fill_u8(info["device_base"], info["pool_bytes"], POOL_SENT, s)
    dA = to_device(A)
    dB = torch.empty_like(dA)
    dB.view(torch.uint8).fill_(CACHE_SENT)
    cA = kvx.Cache(dA, lay.kv, NB, block_order=order)
    cB = kvx.Cache(dB, lay.kv, NB, block_order=order)
    torch.cuda.synchronize()  # dB was filled on the default stream; s is non-blocking
    kvx.kv_store(cA, bt_tensor(btA), n, pool, cid, s)
    got_pool = _read(info["device_base"], info["pool_bytes"], s)
    A_hnd = A if order == kvx.KV_BLOCK_HND else np.ascontiguousarray(A.transpose(0, 1, 2, 4, 3, 5))
    want_pool = oracle_pool(lay, A_hnd, btA, n, cid, num_slots, POOL_SENT)
    assert np.array_equal(got_pool, want_pool), "device pool: " + first_mismatch(got_pool, want_pool)
    kvx.kv_load(cB, bt_tensor(btB), n, pool, cid, s)
    s.synchronize()
    B0 = np.full(A_hnd.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0, btB, n, want_pool, cid)
    if order == kvx.KV_BLOCK_NHD:
        want_B = np.ascontiguousarray(want_B.transpose(0, 1, 2, 4, 3, 5))
    got_B = to_host(dB, want_B)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("n", [4096, 4096 + 192, 4096 + 1, 17, 1])
def test_device_pool_tiny(n):
    """The tiny configuration (and partial chunks/blocks) through a device pool, shuffled slots."""
    _device_round_trip(TINY, 512, n, "tiny")


@pytest.mark.parametrize("dims,order", [
    ((16, 4, 256, 1, 32, 1568), kvx.KV_BLOCK_NHD),   # the paper's FP8 attention geometry, NHD pages
    ((3, 3, 24, 2, 16, 256), kvx.KV_BLOCK_HND),      # 3-vector rows, 3 heads
    ((2, 2, 4, 4, 1, 8), kvx.KV_BLOCK_HND),          # E = 4, one-token blocks
])
def test_device_pool_layouts(dims, order):
    lay = Layout(*dims)
    n = 2 * lay.C + lay.BS + 1
    _device_round_trip(lay, lay.nblk(n) + 7, n, "layouts", dist="raw", order=order, chunks_per_batch=2)


def test_device_pool_rejects_staged_and_staging():
    lay = TINY
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(lay.kv, 4, "staged", host_kind=kvx.KV_POOL_DEVICE)
    assert e.value.status == kvx.KV_EINVAL
    with pytest.raises(kvx.KvError):
        kvx.kv_pool_create(lay.kv, 4, "zero_copy", host_kind=kvx.KV_POOL_DEVICE, staging_slots=2)
    pool = kvx.kv_pool_create(lay.kv, 4, "zero_copy", host_kind=kvx.KV_POOL_DEVICE)
    with pytest.raises(kvx.KvError):
        kvx.kv_pool_set_mode(pool, "staged")
    with pytest.raises(ValueError):
        kvx.pool_view(pool)
    kvx.kv_pool_destroy(pool)


def test_device_pool_128k_per_layer():
    """The benchmark's device-only leg: 131,072 tokens of the 27B-class layout from per-layer caches
    into a 32 GiB device pool in 16-chunk launches, then into a fresh random block set of a second
    replica.  Sampled chunks equal the oracle's bytes; every layer's restored blocks equal the source's;
    blocks outside B's table stay zero."""
    lay, n, NB = B27, 131072, 10240
    nblk, nc = lay.nblk(n), lay.nc(n)
    seed = harness.sub_seed("device-pool-128k", n)
    print(f"[device pool] n={n} NB={NB} nc={nc}", flush=True)
    pool = kvx.kv_pool_create(lay.kv, nc, "zero_copy", host_kind=kvx.KV_POOL_DEVICE)
    info = kvx.kv_pool_get_info(pool)
    assert info["chunks_per_batch"] == 16
    per_layer = NB * 2 * lay.H * lay.BS * lay.D
    A = [torch.empty((NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV) for _ in range(lay.L)]
    B = [torch.zeros_like(t) for t in A]
    for l, t in enumerate(A):
        hg.fill_values(t, l * per_layer, seed, "n01", 2)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    tA, tB = torch.from_numpy(btA).to(DEV), torch.from_numpy(btB).to(DEV)
    ids = harness.chunk_ids(nc, nc)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(A, lay.kv, NB), tA, n, pool, ids, s)
    kvx.kv_load(kvx.Cache(B, lay.kv, NB), tB, n, pool, ids, s)
    s.synchronize()
    assert kvx.kv_pool_async_error(pool) == 0
    bpc = lay.C // lay.BS
    for i in sorted({0, nc // 2, nc - 1}):
        want = _oracle_slot(seed, NB, btA[i * bpc:(i + 1) * bpc], lay.C)
        got = _read(info["device_base"] + i * lay.slot_bytes, lay.slot_bytes, s)
        assert np.array_equal(got, want), f"chunk {i}: device pool differs from the oracle"
    ta = torch.from_numpy(btA.astype(np.int64)).to(DEV)
    tb = torch.from_numpy(btB.astype(np.int64)).to(DEV)
    unused = torch.from_numpy(np.setdiff1d(np.arange(NB), btB)[:256]).to(DEV)
    for l in range(lay.L):
        assert torch.equal(A[l][ta], B[l][tb]), f"layer {l}: restored blocks differ from the source"
        assert not bool(B[l][unused].any()), f"layer {l}: a block outside the table was written"
    kvx.kv_pool_destroy(pool)
    del A, B
    torch.cuda.empty_cache()

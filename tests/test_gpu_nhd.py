"""GPU parity for token-major ("NHD", [2][BS][H][D]) cache blocks, the variant the paper's
patch could not read (Sec. 3.1), and for mixing block orders through one pool.

Expected bytes come from the oracle (block_order NHD/HND) on host-generated inputs.
"""
import numpy as np
import pytest
import torch

import harness
import oracle
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import DEV, Layout, bt_tensor, first_mismatch, layers_of, to_device, to_host

pytestmark = pytest.mark.gpu

POOL_SENT, CACHE_SENT = 0xA5, 0x5A
PAPER = (16, 4, 256, 1, 32, 1568)  # FP8 KV, 16 attention layers, 4 KV heads, D 256, 32-token pages (Table 1)


def _nhd_shape(lay, NB):
    return (lay.L, NB, 2, lay.BS, lay.H, lay.D)


def _oracle(lay, A, order, bt, n, ids, num_slots):
    pool = np.full(num_slots * lay.slot_bytes, POOL_SENT, dtype=np.uint8)
    assert oracle.pack(lay.orc, layers_of(A), lay.block_bytes, A.shape[1], bt, n, pool, ids, 4,
                       block_order=order) == oracle.OK
    return pool


def _oracle_unpack(lay, B0, order, bt, n, pool, ids):
    out = B0.copy()
    assert oracle.unpack(lay.orc, layers_of(out), lay.block_bytes, out.shape[1], bt, n, pool, ids, 4,
                         block_order=order) == oracle.OK
    return out


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("dims,n", [((2, 2, 64, 2, 16, 256), 4096), ((2, 2, 64, 2, 16, 256), 4096 + 192 + 5),
                                    (PAPER, 2 * 1568 + 931), ((3, 3, 16, 4, 4, 12), 53)],
                         ids=["tiny", "tiny-partial", "paper-geometry", "odd"])
def test_nhd_round_trip(mode, dims, n):
    lay = Layout(*dims)
    NB = lay.nblk(n) + 9
    seed = harness.sub_seed("nhd", n, *dims)
    A = harness.gen_cache(seed, "raw", lay.L, NB, lay.H, lay.BS, lay.D, lay.E).reshape(_nhd_shape(lay, NB))
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    nc = lay.nc(n)
    ids = harness.chunk_ids(nc, nc + 1, seed=seed + 3)
    pool = kvx.kv_pool_create(lay.kv, nc + 1, mode, staging_slots=2, chunks_per_batch=2)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(A)
    dB = torch.empty_like(dA)
    dB.view(torch.uint8).fill_(CACHE_SENT)
    cA = kvx.Cache(dA, lay.kv, NB, block_order=kvx.KV_BLOCK_NHD)
    cB = kvx.Cache(dB, lay.kv, NB, block_order=kvx.KV_BLOCK_NHD)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(cA, tA, n, pool, ids, s)
    kvx.kv_load(cB, tB, n, pool, ids, s)
    s.synchronize()
    want_pool = _oracle(lay, A, oracle.BLOCK_NHD, btA, n, ids, nc + 1)
    assert np.array_equal(view, want_pool), first_mismatch(view, want_pool)
    B0 = np.full(A.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[...] = CACHE_SENT
    want_B = _oracle_unpack(lay, B0, oracle.BLOCK_NHD, btB, n, want_pool, ids)
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), first_mismatch(got_B, want_B)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("src_order,dst_order", [(kvx.KV_BLOCK_NHD, kvx.KV_BLOCK_HND),
                                                 (kvx.KV_BLOCK_HND, kvx.KV_BLOCK_NHD)])
def test_mixed_block_orders_share_one_pool(mode, src_order, dst_order):
    """A replica with token-major blocks stores; a replica with head-major blocks restores (and back)."""
    lay = Layout(2, 4, 32, 2, 16, 256)
    n = 3 * 256 + 40
    NB = lay.nblk(n) + 5
    seed = harness.sub_seed("mixed", src_order, dst_order)
    A = harness.gen_cache(seed, "raw", lay.L, NB, lay.H, lay.BS, lay.D, lay.E)
    if src_order == kvx.KV_BLOCK_NHD:
        A = A.reshape(_nhd_shape(lay, NB))
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    nc = lay.nc(n)
    ids = np.arange(nc)
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=2)
    dA = to_device(A)
    B_shape = _nhd_shape(lay, NB) if dst_order == kvx.KV_BLOCK_NHD else (lay.L, NB, 2, lay.H, lay.BS, lay.D)
    dB = torch.zeros(B_shape, dtype=dA.dtype, device=DEV)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB, block_order=src_order), tA, n, pool, ids)
    kvx.kv_load(kvx.Cache(dB, lay.kv, NB, block_order=dst_order), tB, n, pool, ids)
    torch.cuda.synchronize()
    want_pool = _oracle(lay, A, src_order, btA, n, ids, nc)
    want_B = _oracle_unpack(lay, np.zeros(B_shape, dtype=A.dtype), dst_order, btB, n, want_pool, ids)
    got_B = dB.cpu().numpy().view(A.dtype).reshape(B_shape)
    assert np.array_equal(got_B, want_B), first_mismatch(got_B, want_B)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["staged", "zero_copy"])
def test_paper_layout_fullsize_128k(mode):
    """The paper's attention layout at a 131,072-token prefix (84 chunks of 1,568 tokens, the last
    holding 928): 4 GiB per direction, sampled oracle chunks plus whole-prefix round-trip identity."""
    lay = Layout(*PAPER)
    n, NB = 131072, 5120
    nblk, nc = lay.nblk(n), lay.nc(n)
    seed = harness.sub_seed("paper-fullsize")
    shape = _nhd_shape(lay, NB)
    A = torch.empty(shape, dtype=torch.uint8, device=DEV)
    B = torch.zeros_like(A)
    hg.fill_values(A, 0, seed, "raw", 1)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    tA, tB = torch.from_numpy(btA).to(DEV), torch.from_numpy(btB).to(DEV)
    ids = np.arange(nc)
    pool = kvx.kv_pool_create(lay.kv, nc, mode)
    view = kvx.pool_view(pool)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(A, lay.kv, NB, block_order=kvx.KV_BLOCK_NHD), tA, n, pool, ids, s)
    kvx.kv_load(kvx.Cache(B, lay.kv, NB, block_order=kvx.KV_BLOCK_NHD), tB, n, pool, ids, s)
    s.synchronize()
    bpc = lay.C // lay.BS
    for i in (0, nc // 2, nc - 1):
        r = min(lay.C, n - i * lay.C)
        nb = -(-r // lay.BS)
        blocks = btA[i * bpc:i * bpc + nb]
        src = harness.gen_blocks(seed, "raw", lay.L, NB, lay.H, lay.BS, lay.D, lay.E, blocks=blocks)
        src = src.reshape(lay.L, nb, 2, lay.BS, lay.H, lay.D)
        want = np.zeros(lay.slot_bytes, dtype=np.uint8)
        assert oracle.pack(lay.orc, layers_of(np.ascontiguousarray(src)), lay.block_bytes, nb,
                           np.arange(nb, dtype=np.int32), r, want, [0], 8, block_order=oracle.BLOCK_NHD) == 0
        got = view[i * lay.slot_bytes:i * lay.slot_bytes + r * lay.token_bytes]
        assert np.array_equal(got, want[:r * lay.token_bytes]), f"chunk {i} differs from the oracle"
    ta = torch.from_numpy(btA.astype(np.int64)).to(DEV)
    tb = torch.from_numpy(btB.astype(np.int64)).to(DEV)
    for k0 in range(0, nblk, 1024):
        assert torch.equal(A[:, ta[k0:k0 + 1024]], B[:, tb[k0:k0 + 1024]]), "restored prefix differs"
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)

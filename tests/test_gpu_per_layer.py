"""GPU parity with one cache allocation per layer, the way serving engines (and the benchmark)
hold their caches: kv_store / kv_load through the C ABI, byte-compared with the CPU oracle.
"""
import numpy as np
import pytest
import torch

import harness
from paper_2609_15021_amd import kvx
from tests.gpu_support import (DEV, TORCH_INT, Layout, bt_tensor, first_mismatch, host_cache, oracle_pool,
                               oracle_unpack_into, to_device)

pytestmark = pytest.mark.gpu

POOL_SENT = 0xA5
CACHE_SENT = 0x5A


def _explain_slabs(lay, A, bt, n, cid, view, tA, tB, btB):
    """On a wrong pool: for each wrong (chunk, layer, K/V, block) slab, which source block's bytes it
    holds (the block-table entry the store effectively used) and the launch's workgroup id of that
    slab (XCD = id mod 8); and the tables as they read back now."""
    bpc, rows = lay.C // lay.BS, lay.H * lay.D * lay.E
    src = A.view(np.uint8).reshape(lay.L, A.shape[1], 2, lay.H, lay.BS, lay.D * lay.E)
    out = []
    for i in range(lay.nc(n)):
        r = min(lay.C, n - i * lay.C)
        base = int(cid[i]) * lay.slot_bytes
        for l in range(lay.L):
            for kv in range(2):
                plane = base + (l * 2 + kv) * r * rows
                for j in range(-(-r // lay.BS)):
                    bs = min(lay.BS, r - j * lay.BS)
                    got = view[plane + j * lay.BS * rows:plane + (j * lay.BS + bs) * rows]
                    want_b = int(bt[i * bpc + j])
                    as_rows = lambda b: src[l, b, kv, :, :bs, :].transpose(1, 0, 2).reshape(-1)
                    if np.array_equal(got, as_rows(want_b)):
                        continue
                    seen = [b for b in range(A.shape[1]) if np.array_equal(got, as_rows(b))]
                    wg = ((i * lay.L + l) * 2 + kv) * bpc + j
                    out.append(f"(c{i} l{l} kv{kv} j{j} wg{wg} xcd{wg % 8}: want block {want_b}, got {seen[:2]})")
    ta, tb = tA.cpu().numpy(), tB.cpu().numpy()
    return (f"{len(out)} wrong slabs: " + " ".join(out[:24]) +
            f"; table A intact now: {np.array_equal(ta, bt)}; table B intact now: {np.array_equal(tb, btB)}")


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("dims", [(2, 2, 64, 2, 16, 256), (70, 1, 8, 2, 16, 256)], ids=["tiny", "70-layers"])
def test_per_layer_allocations(mode, dims):
    """Caches held as one device allocation per layer (as a serving engine allocates them, and as
    the tier's replicas and the benchmark use them): store from separate per-layer tensors, load
    into separate per-layer tensors of another replica; pool and caches equal the oracle's bytes.
    70 layers also splits the launch's layer pointers across two launches."""
    lay = Layout(*dims)
    NB, n = 96, 5 * lay.C + 33
    seed = harness.sub_seed("parity", "per-layer", mode, lay.L)
    A = host_cache(lay, NB, seed, "raw")
    nblk, nc = lay.nblk(n), lay.nc(n)
    btA, btB = harness.block_table(seed + 1, NB, nblk), harness.block_table(seed + 2, NB, nblk)
    cid = harness.chunk_ids(nc, nc + 1, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, nc + 1, mode, staging_slots=2, chunks_per_batch=2)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    la = [to_device(np.ascontiguousarray(A[l])) for l in range(lay.L)]
    lb = [torch.empty((NB, 2, lay.H, lay.BS, lay.D), dtype=TORCH_INT[lay.E], device=DEV) for _ in range(lay.L)]
    for t in lb:
        t.view(torch.uint8).fill_(CACHE_SENT)
    tA, tB = bt_tensor(btA), bt_tensor(btB)  # valid until the calls complete on s (the ABI's rule)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    assert np.array_equal(tA.cpu().numpy(), btA) and np.array_equal(tB.cpu().numpy(), btB)
    kvx.kv_store(kvx.Cache(la, lay.kv, NB), tA, n, pool, cid, s)
    kvx.kv_load(kvx.Cache(lb, lay.kv, NB), tB, n, pool, cid, s)
    s.synchronize()
    want_pool = oracle_pool(lay, A, btA, n, cid, nc + 1, POOL_SENT)
    assert np.array_equal(view, want_pool), ("pool: " + first_mismatch(view, want_pool) + "; " +
                                             _explain_slabs(lay, A, btA, n, cid, view, tA, tB, btB))
    B0 = np.full(A.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0, btB, n, want_pool, cid)
    got_B = torch.stack(lb).cpu().numpy().view(A.dtype).reshape(A.shape)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    # The library never writes a block table.
    assert np.array_equal(tA.cpu().numpy(), btA) and np.array_equal(tB.cpu().numpy(), btB)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)

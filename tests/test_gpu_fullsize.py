"""Full-size parity on the 27B-class layout (64 layers, 8 KV heads, head_dim 128, bf16,
16-token blocks, 256-token chunks), in the launch configuration the benchmark times.

* Sampled outputs: for the first, a middle and the last chunk, the pool slot equals
  the oracle's store of the host-generated source blocks, byte for byte.
* Property at any size: after the load, every logical block of the prefix in
  replica B equals the same logical block of replica A (round-trip identity,
  compared on the device), blocks outside B's table are untouched, and the
  unwritten tail of a partial chunk's slot keeps its sentinel.
"""
import numpy as np
import pytest
import torch

import harness
import oracle
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import B27, DEV

pytestmark = pytest.mark.gpu

TB = B27.token_bytes
SENT = 0xC3


def _oracle_slot(seed, num_blocks, blocks, r):
    src = harness.gen_blocks(seed, "n01", B27.L, num_blocks, B27.H, B27.BS, B27.D, B27.E, blocks=blocks)
    layers = [np.ascontiguousarray(src[l]).reshape(-1).view(np.uint8) for l in range(B27.L)]
    out = np.zeros(B27.slot_bytes, dtype=np.uint8)
    nb = len(blocks)
    assert oracle.pack(B27.orc, layers, B27.block_bytes, nb, np.arange(nb, dtype=np.int32), r, out, [0], 8) == 0
    return out[:r * TB]


def _blocks_equal(A, btA, B, btB, nblk, step=512):
    ta = torch.from_numpy(btA[:nblk].astype(np.int64)).to(DEV)
    tb = torch.from_numpy(btB[:nblk].astype(np.int64)).to(DEV)
    for k0 in range(0, nblk, step):
        if not torch.equal(A[:, ta[k0:k0 + step]], B[:, tb[k0:k0 + step]]):
            return False
    return True


@pytest.mark.parametrize("mode", ["staged", "zero_copy"])
@pytest.mark.parametrize("n,NB", [(32768, 2560), (131072, 10240), (262336, 20480)],
                         ids=["32k", "128k", "256k+192"])
def test_fullsize_store_load(mode, n, NB):
    lay = B27
    nblk, nc = lay.nblk(n), lay.nc(n)
    seed = harness.sub_seed("fullsize", n)
    print(f"[fullsize] mode={mode} n={n} NB={NB} nc={nc}", flush=True)
    A = torch.empty((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
    B = torch.zeros_like(A)
    hg.fill_values(A, 0, seed, "n01", 2)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    tA, tB = torch.from_numpy(btA).to(DEV), torch.from_numpy(btB).to(DEV)
    ids = harness.chunk_ids(nc, nc)
    try:
        pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=3 if mode == "staged" else 0)
    except kvx.KvError as e:
        # Only the environment's pinned-memory ceiling (about 65.5 GiB per process on these
        # machines, against 64.06 GiB for the 256k pool) is a reason to skip; anything else fails.
        if e.status == kvx.KV_ENOMEM and n > 131072:
            pytest.skip(f"this machine cannot pin the {nc * lay.slot_bytes / 2**30:.2f} GiB pool: {e}")
        raise
    view = kvx.pool_view(pool)
    r_last = n - (nc - 1) * lay.C
    if r_last < lay.C:
        view[(nc - 1) * lay.slot_bytes + r_last * TB:nc * lay.slot_bytes] = SENT
    cA, cB = kvx.Cache(A, lay.kv, NB), kvx.Cache(B, lay.kv, NB)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()  # fills ran on the default stream; s is non-blocking
    kvx.kv_store(cA, tA, n, pool, ids, s)
    kvx.kv_load(cB, tB, n, pool, ids, s)
    s.synchronize()
    assert kvx.kv_pool_async_error(pool) == 0
    bpc = lay.C // lay.BS
    for i in sorted({0, nc // 2, nc - 1}):
        r = min(lay.C, n - i * lay.C)
        want = _oracle_slot(seed, NB, btA[i * bpc:i * bpc + -(-r // lay.BS)], r)
        got = view[i * lay.slot_bytes:i * lay.slot_bytes + r * TB]
        assert np.array_equal(got, want), f"chunk {i}: pool differs from the oracle"
    if r_last < lay.C:
        assert np.all(view[(nc - 1) * lay.slot_bytes + r_last * TB:nc * lay.slot_bytes] == SENT)
    assert _blocks_equal(A, btA, B, btB, nblk), "restored prefix differs from the source"
    unused = np.setdiff1d(np.arange(NB), btB)[:256]
    assert not bool(B[:, torch.from_numpy(unused).to(DEV)].any()), "a block outside the table was written"
    kvx.kv_pool_destroy(pool)
    del A, B
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["staged", "zero_copy"])
def test_fullsize_per_layer_128k(mode):
    """The benchmark's own configuration: each replica holds its cache as one device allocation
    per layer (64 tensors of 10,240 blocks), 128k tokens, the pool's default batch and ring.
    Sampled chunks equal the oracle's bytes; every layer's restored blocks equal the source's;
    blocks outside B's table stay zero."""
    lay, n, NB = B27, 131072, 10240
    nblk, nc = lay.nblk(n), lay.nc(n)
    seed = harness.sub_seed("fullsize-per-layer", n)
    print(f"[fullsize] per-layer mode={mode} n={n} NB={NB} nc={nc}", flush=True)
    per_layer = NB * 2 * lay.H * lay.BS * lay.D  # elements per layer
    A = [torch.empty((NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV) for _ in range(lay.L)]
    B = [torch.zeros_like(t) for t in A]
    for l, t in enumerate(A):  # the same values as layer l of one [L][NB]... tensor
        hg.fill_values(t, l * per_layer, seed, "n01", 2)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    tA, tB = torch.from_numpy(btA).to(DEV), torch.from_numpy(btB).to(DEV)
    ids = harness.chunk_ids(nc, nc)
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=3 if mode == "staged" else 0)
    view = kvx.pool_view(pool)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()  # fills ran on the default stream; s is non-blocking
    kvx.kv_store(kvx.Cache(A, lay.kv, NB), tA, n, pool, ids, s)
    kvx.kv_load(kvx.Cache(B, lay.kv, NB), tB, n, pool, ids, s)
    s.synchronize()
    assert kvx.kv_pool_async_error(pool) == 0
    bpc = lay.C // lay.BS
    for i in sorted({0, nc // 2, nc - 1}):
        want = _oracle_slot(seed, NB, btA[i * bpc:(i + 1) * bpc], lay.C)
        assert np.array_equal(view[i * lay.slot_bytes:(i + 1) * lay.slot_bytes], want), \
            f"chunk {i}: pool differs from the oracle"
    ta = torch.from_numpy(btA.astype(np.int64)).to(DEV)
    tb = torch.from_numpy(btB.astype(np.int64)).to(DEV)
    unused = torch.from_numpy(np.setdiff1d(np.arange(NB), btB)[:256]).to(DEV)
    for l in range(lay.L):
        assert torch.equal(A[l][ta], B[l][tb]), f"layer {l}: restored blocks differ from the source"
        assert not bool(B[l][unused].any()), f"layer {l}: a block outside the table was written"
    kvx.kv_pool_destroy(pool)
    del A, B
    torch.cuda.empty_cache()


def test_six_turn_session_with_producer_delays():
    """Initial 128k context, six turns, 2,048 new tokens per later turn; the producer stores only
    its new chunks after a seeded 5-50 ms spin and its own fill on the same stream; the other
    replica, with freshly fragmented blocks, loads the whole prefix; producers alternate."""
    lay = B27
    NB = 10240
    n0, add, turns = 131072, 2048, 6
    n_final = n0 + add * (turns - 1)
    seed = harness.sub_seed("session")
    delays = harness.spin_delays_ms(seed, turns)
    # Ground truth of the session, logical block k at G[:, k].
    G = torch.empty((lay.L, lay.nblk(n_final), 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV)
    hg.fill_values(G, 0, seed, "n01", 2)
    reps = [torch.zeros((lay.L, NB, 2, lay.H, lay.BS, lay.D), dtype=torch.int16, device=DEV) for _ in range(2)]
    caches = [kvx.Cache(t, lay.kv, NB) for t in reps]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    tables = [None, None]
    pool = kvx.kv_pool_create(lay.kv, lay.nc(n_final), "staged")
    torch.cuda.synchronize()  # G and the replicas were filled on the default stream
    n_prev = 0
    rng = np.random.default_rng(seed)
    for t in range(turns):
        prod, cons = t % 2, 1 - t % 2
        n = n0 + add * t
        nblk = lay.nblk(n)
        if tables[prod] is None:
            tables[prod] = rng.permutation(NB)[:nblk].astype(np.int32)
        else:  # append new blocks to the producer's table from its free blocks
            free = np.setdiff1d(np.arange(NB), tables[prod])
            extra = rng.permutation(free)[:nblk - len(tables[prod])]
            tables[prod] = np.concatenate([tables[prod], extra]).astype(np.int32)
        s = streams[prod]
        k0 = lay.nblk(n_prev)
        with torch.cuda.stream(s):
            hg.spin(float(delays[t]), s)
            idx = torch.from_numpy(tables[prod][k0:nblk].astype(np.int64)).to(DEV)
            reps[prod][:, idx] = G[:, k0:nblk]  # the producer writes its new tokens' KV
        c0 = n_prev // lay.C
        new_ids = np.arange(c0, lay.nc(n))
        # Store only the new chunks: the prefix tail [c0*C, n) seen through the table offset.
        bt_new = torch.from_numpy(tables[prod][c0 * (lay.C // lay.BS):nblk]).to(DEV)
        kvx.kv_store(caches[prod], bt_new, n - c0 * lay.C, pool, new_ids, s)
        s.synchronize()  # host completion before the other replica reads the pool
        # Consumer: drop its blocks, draw a fresh fragmented set, restore the whole prefix.
        with torch.cuda.stream(streams[cons]):
            reps[cons].zero_()
        tables[cons] = rng.permutation(NB)[:nblk].astype(np.int32)
        tc = torch.from_numpy(tables[cons]).to(DEV)
        kvx.kv_load(caches[cons], tc, n, pool, np.arange(lay.nc(n)), streams[cons])
        streams[cons].synchronize()
        ti = torch.from_numpy(tables[cons].astype(np.int64)).to(DEV)
        for b0 in range(0, nblk, 512):
            assert torch.equal(reps[cons][:, ti[b0:b0 + 512]], G[:, b0:min(b0 + 512, nblk)]), f"turn {t}"
        assert kvx.kv_pool_async_error(pool) == 0
        n_prev = n
        print(f"[session] turn {t}: producer {prod} stored {len(new_ids)} chunks after {delays[t]:.1f} ms; "
              f"replica {cons} restored {n} tokens", flush=True)
    kvx.kv_pool_destroy(pool)

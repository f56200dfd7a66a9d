"""GPU parity: kv_store / kv_load through the C ABI, byte-compared with the CPU oracle.

Inputs come from the seeded host generator; expected pool and cache bytes come
from the oracle applied to those host inputs.  The bar is bit-exact: this path
moves integers (opaque bytes), so any difference is a failure.
"""
import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from paper_2609_15021_amd import kvx
from tests.gpu_support import (TINY, Layout, bt_tensor, device_cache, first_mismatch, host_cache,
                               oracle_pool, oracle_unpack_into, to_device, to_host)

pytestmark = pytest.mark.gpu

POOL_SENT = 0xA5
CACHE_SENT = 0x5A


def _round_trip(lay: Layout, NB: int, n: int, mode: str, host_kind=0, shuffled=False, dist="u11", seed_tag="t",
                extra_slots=2, stream=None, block_stride=0, **pool_kw):
    """Store A -> pool -> load into B (second allocation); compare both with the oracle."""
    seed = harness.sub_seed("parity", seed_tag, n, lay.L, lay.H, lay.D, lay.E, lay.BS, lay.C)
    A = host_cache(lay, NB, seed, dist)
    nblk = lay.nblk(n)
    btA = harness.block_table(seed + 1, NB, nblk)
    btB = harness.block_table(seed + 2, NB, nblk)
    nc = lay.nc(n)
    num_slots = nc + extra_slots
    cid = harness.chunk_ids(nc, num_slots, seed + 3 if shuffled else None)
    pool = kvx.kv_pool_create(lay.kv, num_slots, mode, host_kind=host_kind, **pool_kw)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(A)
    dB = device_cache(lay, NB, fill=CACHE_SENT)
    cA, cB = kvx.Cache(dA, lay.kv, NB), kvx.Cache(dB, lay.kv, NB)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    s = stream if stream is not None else torch.cuda.Stream()
    kvx.kv_store(cA, tA, n, pool, cid, s)
    torch.cuda.synchronize()
    want_pool = oracle_pool(lay, A, btA, n, cid, num_slots, POOL_SENT)
    assert np.array_equal(view, want_pool), "pool: " + first_mismatch(view, want_pool)
    kvx.kv_load(cB, tB, n, pool, cid, s)
    torch.cuda.synchronize()
    B0 = np.full_like(A, 0).view(np.uint8)
    B0[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0.view(A.dtype).reshape(A.shape), btB, n, want_pool, cid)
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    np.testing.assert_array_equal(to_host(dA, A), A)  # store never writes the source
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("host_kind", [kvx.KV_HOST_COHERENT, kvx.KV_HOST_NONCOHERENT])
@pytest.mark.parametrize("shuffled", [False, True])
def test_tiny_config_round_trip(mode, host_kind, shuffled):
    """2 layers, 2 KV heads, D 64, BS 16, bf16 U[-1,1]; 4,096 tokens on 256 random blocks of 512;
    16 chunks of 256 tokens; load into a different random 256-block set of a second allocation."""
    _round_trip(TINY, 512, 4096, mode, host_kind, shuffled)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("n", [4096 + 192, 4096 + 128, 4096 + 64, 4096 + 1, 4, 17, 1, 255, 257])
def test_partial_chunks_and_blocks(mode, n):
    """Partial final chunk (compact r*TB bytes, slot tail untouched) and partial final block."""
    _round_trip(TINY, 512, n, mode, shuffled=True)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
@pytest.mark.parametrize("dims", [
    (70, 1, 8, 2, 16, 256),     # more layers than one launch carries; 16-byte rows
    (3, 3, 24, 2, 16, 256),     # 48-byte rows (3 vectors), 3 heads
    (2, 2, 4, 4, 1, 8),         # E = 4, one-token blocks, tiny chunks
    (16, 4, 256, 1, 32, 1568),  # the paper's attention geometry: FP8, 4 KV heads, D 256, 32-token pages,
                                # 1,568-token chunks (Table 1 and Sec. 3.1)
    (1, 8, 128, 2, 16, 16),     # chunk == block
    (2, 1, 2048, 2, 4, 64),     # 4 KiB rows (more vectors per row than work-items)
])
def test_layout_variants(mode, dims):
    lay = Layout(*dims)
    n = (2 if lay.C > 256 else 3) * lay.C + lay.BS + 1
    NB = lay.nblk(n) + 7
    _round_trip(lay, NB, n, mode, shuffled=True, dist="raw", staging_slots=2, chunks_per_batch=2)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_all_16bit_patterns_bit_exact(mode):
    """Raw bit patterns (NaN payloads, +-Inf, -0, subnormals as bf16) survive the GPU path."""
    _round_trip(TINY, 512, 4096, mode, dist="raw", seed_tag="raw")


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_small_staging_ring_many_batches(mode):
    """A 2-slot staging ring with one chunk per batch over 64 chunks: staging reuse stays ordered."""
    _round_trip(TINY, 4096 + 64, 64 * 256, mode, shuffled=True, staging_slots=2, chunks_per_batch=1,
                side_streams=2)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_padded_block_stride(mode):
    """Blocks with padding between them: padding is neither read into chunks nor written."""
    lay = TINY
    NB, pad = 300, 64  # padding in elements of 2 bytes
    n = 1000
    seed = harness.sub_seed("stride")
    raw = np.random.default_rng(seed).integers(0, 1 << 16, size=(lay.L, NB, lay.block_elems + pad),
                                               dtype=np.uint64).astype(np.uint16)
    A = np.ascontiguousarray(raw[:, :, :lay.block_elems]).reshape(lay.L, NB, 2, lay.H, lay.BS, lay.D)
    stride = (lay.block_elems + pad) * 2
    btA = harness.block_table(seed + 1, NB, lay.nblk(n))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n))
    nc = lay.nc(n)
    cid = np.arange(nc)
    pool = kvx.kv_pool_create(lay.kv, nc, mode)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(raw)
    dB = torch.full_like(dA, 0x7777)
    cA = kvx.Cache(dA, lay.kv, NB, stride)
    cB = kvx.Cache(dB, lay.kv, NB, stride)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    kvx.kv_store(cA, tA, n, pool, cid)
    kvx.kv_load(cB, tB, n, pool, cid)
    torch.cuda.synchronize()
    want_pool = oracle_pool(lay, A, btA, n, cid, nc, POOL_SENT)
    assert np.array_equal(view, want_pool), first_mismatch(view, want_pool)
    gotB = dB.cpu().numpy().view(np.uint16).reshape(lay.L, NB, lay.block_elems + pad)
    assert np.all(gotB[:, :, lay.block_elems:] == 0x7777)
    B0 = np.full((lay.L, NB, 2, lay.H, lay.BS, lay.D), 0x7777, dtype=np.uint16)
    want_B = oracle_unpack_into(lay, B0, btB, n, want_pool, cid)
    np.testing.assert_array_equal(np.ascontiguousarray(gotB[:, :, :lay.block_elems]).reshape(want_B.shape), want_B)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_load_into_disjoint_blocks_of_same_allocation(mode):
    """Tiny config: 256 source blocks and 256 disjoint destination blocks in one 512-block
    allocation; the load never touches the source blocks."""
    lay, NB, n = TINY, 512, 4096
    seed = harness.sub_seed("disjoint")
    A = host_cache(lay, NB, seed, "u11")
    btA = harness.block_table(seed + 1, NB, 256)
    btB = harness.block_table(seed + 2, NB, 256, exclude=btA)
    pool = kvx.kv_pool_create(lay.kv, 16, mode)
    dA = to_device(A)
    cA = kvx.Cache(dA, lay.kv, NB)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    cid = np.arange(16)
    kvx.kv_store(cA, tA, n, pool, cid)
    kvx.kv_load(cA, tB, n, pool, cid)
    torch.cuda.synchronize()
    want_pool = oracle_pool(lay, A, btA, n, cid, 16, 0)
    want = oracle_unpack_into(lay, A, btB, n, want_pool, cid)
    got = to_host(dA, A)
    assert np.array_equal(got, want), first_mismatch(got, want)
    np.testing.assert_array_equal(got[:, btA], A[:, btA])
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_load_with_repeated_chunk_ids(mode):
    """A load may name one slot for several chunks (they are reads): here slot 2 for chunks 0 and
    2 of the restored prefix, whose last chunk is partial (100 of 256 tokens, read from a full
    slot).  Cache B equals the oracle's unpack of the same ids, byte for byte."""
    lay, NB = TINY, 512
    seed = harness.sub_seed("parity", "repeated-ids", mode)
    A = host_cache(lay, NB, seed, "raw")
    n_s, ids_s = 3 * lay.C + 40, [0, 1, 2, 3]
    n_l, ids_l = 3 * lay.C + 100, [2, 0, 2, 1]
    btA = harness.block_table(seed + 1, NB, lay.nblk(n_s))
    btB = harness.block_table(seed + 2, NB, lay.nblk(n_l))
    pool = kvx.kv_pool_create(lay.kv, 4, mode, staging_slots=2, chunks_per_batch=2)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA, dB = to_device(A), device_cache(lay, NB, fill=CACHE_SENT)
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), tA, n_s, pool, ids_s, s)
    kvx.kv_load(kvx.Cache(dB, lay.kv, NB), tB, n_l, pool, ids_l, s)
    s.synchronize()
    want_pool = oracle_pool(lay, A, btA, n_s, ids_s, 4, POOL_SENT)
    assert np.array_equal(view, want_pool), "pool: " + first_mismatch(view, want_pool)
    B0 = np.full_like(A, 0).view(np.uint8)
    B0[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0.view(A.dtype).reshape(A.shape), btB, n_l, want_pool, ids_l)
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_zero_tokens_is_noop(mode):
    lay = TINY
    pool = kvx.kv_pool_create(lay.kv, 2, mode)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    d = device_cache(lay, 8, fill=CACHE_SENT)
    c = kvx.Cache(d, lay.kv, 8)
    kvx.kv_store(c, None, 0, pool, [])
    kvx.kv_load(c, None, 0, pool, [])
    torch.cuda.synchronize()
    assert np.all(view == POOL_SENT)
    assert bool((d.view(torch.uint8) == CACHE_SENT).all())
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_out_of_range_block_is_flagged_and_skipped(mode):
    """A block id outside [0, num_blocks) is reported, its cache block is never read, and its
    chunk rows are zeros in both modes (no stale staging bytes reach the shared pool)."""
    lay, NB, n = TINY, 64, 512
    seed = harness.sub_seed("badblock")
    A = host_cache(lay, NB, seed, "u11")
    bt = harness.block_table(seed + 1, NB, 32)
    bad = bt.copy()
    bad[5] = NB          # one past the end
    bad[20] = -3
    pool = kvx.kv_pool_create(lay.kv, 2, mode)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(A)
    c = kvx.Cache(dA, lay.kv, NB)
    t = bt_tensor(bad)
    kvx.kv_store(c, t, n, pool, [0, 1])
    torch.cuda.synchronize()
    assert kvx.kv_pool_async_error(pool) == kvx.KV_ASYNC_BAD_BLOCK
    # Expected: the oracle's store of the same request with the two bad blocks' rows zeroed.
    A0 = A.copy()
    spare = np.concatenate([A0, np.zeros_like(A0[:, :1])], axis=1)  # block NB = all zeros
    bt0 = bt.copy()
    bt0[5] = NB
    bt0[20] = NB
    want = oracle_pool(lay, spare, bt0, n, [0, 1], 2, POOL_SENT)
    assert np.array_equal(view, want), first_mismatch(view, want)
    assert kvx.kv_pool_async_error(pool, clear=True) == kvx.KV_ASYNC_BAD_BLOCK
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_binding_keeps_a_temporary_block_table_until_the_stream_used_it(mode):
    """Python callers may pass a temporary block table: the binding records it as in use on the
    call's stream, so torch's caching allocator does not hand its memory to the next tensor (here
    another table of the same size, uploaded on the default stream) while the call's kernels on
    another stream have yet to read it.  Without that, the store reads the other table's entries.
    The producer stream starts behind a 20 ms spin so the kernels run well after the upload."""
    lay = TINY
    NB, n = 512, 4096 + 192
    seed = harness.sub_seed("parity", "temporary-table", mode)
    A = host_cache(lay, NB, seed, "raw")
    nblk, nc = lay.nblk(n), lay.nc(n)
    btA, btX = harness.block_table(seed + 1, NB, nblk), harness.block_table(seed + 2, NB, nblk)
    cid = harness.chunk_ids(nc, nc, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, nc, mode, staging_slots=2, chunks_per_batch=2)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(A)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    hg.spin(20.0, s)
    kvx.kv_store(kvx.Cache(dA, lay.kv, NB), bt_tensor(btA), n, pool, cid, s)  # the table is dropped here
    other = bt_tensor(btX)  # same size: the allocator's first candidate for the freed block
    s.synchronize()
    del other
    want = oracle_pool(lay, A, btA, n, cid, nc, POOL_SENT)
    assert np.array_equal(view, want), "pool: " + first_mismatch(view, want)
    kvx.kv_pool_destroy(pool)


@pytest.mark.parametrize("store_mode,load_mode", [("staged", "zero_copy"), ("zero_copy", "staged")])
def test_separate_store_and_load_modes(store_mode, load_mode):
    """kv_pool_set_modes gives stores and loads their own mode.  On one stream with no host sync in
    between: store (one mode), load (the other), then a second store of other chunks and a load of
    them; pools and caches equal the oracle's bytes, and the pool reports both modes."""
    lay = TINY
    NB, n = 512, 4096 + 192
    seed = harness.sub_seed("parity", "modes", store_mode)
    A = host_cache(lay, NB, seed, "raw")
    nblk, nc = lay.nblk(n), lay.nc(n)
    btA, btB = harness.block_table(seed + 1, NB, nblk), harness.block_table(seed + 2, NB, nblk)
    num_slots = 2 * nc
    ids = harness.chunk_ids(2 * nc, num_slots, seed + 3)
    pool = kvx.kv_pool_create(lay.kv, num_slots, "staged", staging_slots=2, chunks_per_batch=2)
    kvx.kv_pool_set_modes(pool, store_mode, load_mode)
    info = kvx.kv_pool_get_info(pool)
    assert (info["mode"], info["load_mode"]) == (kvx.MODES[store_mode], kvx.MODES[load_mode])
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA = to_device(A)
    dB1, dB2 = device_cache(lay, NB, fill=CACHE_SENT), device_cache(lay, NB, fill=CACHE_SENT)
    cA, cB1, cB2 = (kvx.Cache(d, lay.kv, NB) for d in (dA, dB1, dB2))
    tA, tB = bt_tensor(btA), bt_tensor(btB)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(cA, tA, n, pool, ids[:nc], s)
    kvx.kv_load(cB1, tB, n, pool, ids[:nc], s)
    kvx.kv_store(cA, tB, n, pool, ids[nc:], s)  # other blocks of A into the other slots
    kvx.kv_load(cB2, tA, n, pool, ids[nc:], s)
    s.synchronize()
    want = oracle_pool(lay, A, btA, n, ids[:nc], num_slots, POOL_SENT)
    other = oracle_pool(lay, A, btB, n, ids[nc:], num_slots, POOL_SENT)
    for i in ids[nc:]:
        want[i * lay.slot_bytes:(i + 1) * lay.slot_bytes] = other[i * lay.slot_bytes:(i + 1) * lay.slot_bytes]
    assert np.array_equal(view, want), "pool: " + first_mismatch(view, want)
    B0 = np.full(A.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[:] = CACHE_SENT
    for got_t, bt, cid in ((dB1, btB, ids[:nc]), (dB2, btA, ids[nc:])):
        want_B = oracle_unpack_into(lay, B0, bt, n, want, cid)
        got = to_host(got_t, A)
        assert np.array_equal(got, want_B), "cache: " + first_mismatch(got, want_B)
    kvx.kv_pool_set_mode(pool, "zero_copy")
    info = kvx.kv_pool_get_info(pool)
    assert info["mode"] == info["load_mode"] == kvx.KV_MODE_ZERO_COPY
    kvx.kv_pool_destroy(pool)
    zc = kvx.kv_pool_create(lay.kv, 2, "zero_copy")  # no staging: staged is refused in either direction
    for modes in (("staged", "zero_copy"), ("zero_copy", "staged")):
        with pytest.raises(kvx.KvError) as e:
            kvx.kv_pool_set_modes(zc, *modes)
        assert e.value.status == kvx.KV_EINVAL
    kvx.kv_pool_destroy(zc)


@pytest.mark.parametrize("mode", ["zero_copy", "staged"])
def test_concurrent_store_and_load_on_two_streams(mode):
    """Two replicas use one pool at once: one stores prefix Q into slots Y on stream s1 while
    another loads prefix P from slots X on stream s2 (the caller orders nothing between them:
    the two calls touch disjoint slots).  With a 2-slot ring of 1-chunk batches, the store's and
    the load's batches take turns in the shared staging ring many times while both are in
    flight; s1 starts behind a 20 ms spin so that the load runs first and the two interleave.
    Pool and caches equal the oracle's bytes."""
    lay = TINY
    NB, n = 512, 5 * lay.C + 77
    nc, nblk = lay.nc(n), lay.nblk(n)
    seed = harness.sub_seed("parity", "two-streams", mode)
    A = host_cache(lay, NB, seed, "raw")
    Q = host_cache(lay, NB, seed + 10, "raw")
    btA, btQ, btB = (harness.block_table(seed + k, NB, nblk) for k in (1, 2, 3))
    num_slots = 2 * nc + 1
    ids = harness.chunk_ids(2 * nc, num_slots, seed + 4)
    idsX, idsY = ids[:nc], ids[nc:]
    pool = kvx.kv_pool_create(lay.kv, num_slots, mode, staging_slots=2, chunks_per_batch=1)
    view = kvx.pool_view(pool)
    view[:] = POOL_SENT
    dA, dQ = to_device(A), to_device(Q)
    dB = device_cache(lay, NB, fill=CACHE_SENT)
    cA, cQ, cB = (kvx.Cache(d, lay.kv, NB) for d in (dA, dQ, dB))
    tA, tQ, tB = bt_tensor(btA), bt_tensor(btQ), bt_tensor(btB)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    kvx.kv_store(cA, tA, n, pool, idsX, s2)     # prefix P in slots X
    s2.synchronize()
    hg.spin(20.0, s1)
    for _ in range(3):                          # the same bytes each time
        kvx.kv_store(cQ, tQ, n, pool, idsY, s1)
        kvx.kv_load(cB, tB, n, pool, idsX, s2)
    s1.synchronize()
    s2.synchronize()
    want_pool = oracle_pool(lay, A, btA, n, idsX, num_slots, POOL_SENT)
    qpool = oracle_pool(lay, Q, btQ, n, idsY, num_slots, POOL_SENT)
    for i in idsY:
        want_pool[i * lay.slot_bytes:(i + 1) * lay.slot_bytes] = qpool[i * lay.slot_bytes:(i + 1) * lay.slot_bytes]
    assert np.array_equal(view, want_pool), "pool: " + first_mismatch(view, want_pool)
    B0 = np.full(A.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0, btB, n, want_pool, idsX)
    got_B = to_host(dB, A)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)
    assert kvx.kv_pool_async_error(pool) == 0
    kvx.kv_pool_destroy(pool)


def test_pool_info_and_errors():
    lay = TINY
    pool = kvx.kv_pool_create(lay.kv, 4, "zero_copy")
    info = kvx.kv_pool_get_info(pool)
    assert info["is_pinned"] == 1 and info["pool_bytes"] == 4 * lay.slot_bytes and info["staging_bytes"] == 0
    assert info["staging_contiguous"] == 0
    staged = kvx.kv_pool_create(lay.kv, 2, "staged", staging_slots=2, chunks_per_batch=1)
    sinfo = kvx.kv_pool_get_info(staged)
    # One ring of 2 slots x 1 chunk per direction (stores and loads each have their own lane).
    assert sinfo["staging_bytes"] == 2 * 2 * lay.slot_bytes and sinfo["staging_contiguous"] == 0
    assert sinfo["side_streams"] == 1 and sinfo["staging_slots"] == 2
    kvx.kv_pool_destroy(staged)
    assert kvx.kv_pool_slot_bytes(pool) == lay.slot_bytes and kvx.kv_pool_num_slots(pool) == 4
    assert kvx.kv_pool_slot(pool, 3) == info["host_base"] + 3 * lay.slot_bytes
    assert kvx.kv_pool_slot(pool, 4) == 0
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_set_mode(pool, "staged")  # no staging was allocated
    assert e.value.status == kvx.KV_EINVAL
    d = device_cache(lay, 8)
    c = kvx.Cache(d, kvx.make_layout(2, 2, 64, 2, 32, 256), 4)
    t = bt_tensor(np.arange(8))
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_store(c, t, 64, pool, [0])     # layout differs from the pool's
    assert e.value.status == kvx.KV_EINVAL and "differs" in str(e.value)
    kvx.kv_pool_destroy(pool)
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(lay.kv, 4, 7)       # no silent mode selection
    assert e.value.status == kvx.KV_EINVAL


def test_oversized_pool_is_enomem_not_pageable():
    """An impossible pinned request fails with KV_ENOMEM; nothing falls back to pageable memory."""
    lay = Layout(64, 8, 128, 2, 16, 256)  # 64 MiB slots
    with pytest.raises(kvx.KvError) as e:
        kvx.kv_pool_create(lay.kv, 1 << 24, "zero_copy")  # 1 PiB
    assert e.value.status == kvx.KV_ENOMEM


def test_readme_usage():
    """The README's Python usage, at a small size: per-layer bf16 tensors, the current stream,
    store then load with no host sync in between; the restored blocks equal the stored ones."""
    L, H, D, BS, C, NB, n = 4, 2, 64, 16, 256, 64, 700
    lay = kvx.make_layout(L, H, D, 2, BS, C)
    nc = -(-n // C)
    pool = kvx.kv_pool_create(lay, nc, "staged", staging_slots=3)
    g = torch.Generator().manual_seed(harness.sub_seed("readme"))
    layers_a = [torch.randn((NB, 2, H, BS, D), generator=g).to(torch.bfloat16).to("cuda:0") for _ in range(L)]
    layers_b = [torch.zeros_like(t) for t in layers_a]
    bt_a = harness.block_table(harness.sub_seed("readme", 1), NB, -(-n // BS))
    bt_b = harness.block_table(harness.sub_seed("readme", 2), NB, -(-n // BS))
    block_table_a, block_table_b = bt_tensor(bt_a), bt_tensor(bt_b)
    chunk_ids = list(range(nc))
    cache_a, cache_b = kvx.Cache(layers_a, lay, NB), kvx.Cache(layers_b, lay, NB)
    s = torch.cuda.current_stream()
    kvx.kv_store(cache_a, block_table_a, n, pool, chunk_ids, s)
    kvx.kv_load(cache_b, block_table_b, n, pool, chunk_ids, s)
    s.synchronize()
    assert kvx.kv_pool_async_error(pool) == 0
    full = n // BS  # whole blocks: every token slot restored
    ia = torch.from_numpy(bt_a[:full].astype(np.int64)).to("cuda:0")
    ib = torch.from_numpy(bt_b[:full].astype(np.int64)).to("cuda:0")
    for a, b in zip(layers_a, layers_b):
        assert torch.equal(a[ia].view(torch.int16), b[ib].view(torch.int16))
    kvx.kv_pool_destroy(pool)

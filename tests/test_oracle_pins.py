"""Pins for the CPU oracle (runs on the CPU; no GPU).

The oracle is only trusted because these tests tie it to things other than
itself: an independent numpy fancy-indexing formulation (a library routine),
closed-form coordinate tags, exhaustive brute force over tiny block tables,
round-trip identity, untouched sentinels, degenerate cases that reduce to a
memcpy or a reshape, raw bit patterns, and the paper's own chunk/page numbers.
Each is chosen so that a plausible slip in the oracle (a dropped K/V or head
term, swapped head and slot, plane stride C instead of r for a partial chunk,
a transposed plane) fails at least one of them.
"""
import itertools
import os

import numpy as np
import pytest

import oracle
from tests.numpy_formulation import expected_chunks, scatter_tokens, token_view

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SENT = 0xA5


def _dt(E):
    return {1: np.uint8, 2: np.uint16, 4: np.uint32}[E]


def _layers(A):
    return [A[l].reshape(-1).view(np.uint8) for l in range(A.shape[0])]


def _run_pack(A, bt, n, C, chunk_ids, num_slots, nthreads=1, E=None):
    L, NB, _, H, BS, D = A.shape
    E = A.dtype.itemsize
    lay = oracle.make_layout(L, H, D, E, BS, C)
    sb = oracle.slot_bytes(lay)
    pool = np.full(num_slots * sb, SENT, dtype=np.uint8)
    rc = oracle.pack(lay, _layers(A), 2 * H * BS * D * E, NB, bt, n, pool, chunk_ids, nthreads)
    return rc, pool, sb


def _check_pool(A, bt, n, C, pool, sb, chunk_ids):
    L, NB, _, H, BS, D = A.shape
    E = A.dtype.itemsize
    written = np.zeros(len(pool), dtype=bool)
    for i, ch in enumerate(expected_chunks(A, bt, n, BS, C)):
        start = int(chunk_ids[i]) * sb
        nbytes = ch.nbytes
        got = pool[start:start + nbytes].view(A.dtype).reshape(ch.shape)
        np.testing.assert_array_equal(got, ch)
        written[start:start + nbytes] = True
    # Bytes not named by the definition (slot tails, unused slots) are untouched.
    assert np.all(pool[~written] == SENT)


# ---------------------------------------------------------------- P1: numpy formulation
@pytest.mark.parametrize("E", [1, 2, 4])
@pytest.mark.parametrize("BS", [1, 2, 16])
def test_pack_matches_numpy_formulation(E, BS):
    rng = np.random.default_rng(1000 + 10 * E + BS)
    for L, H, D in itertools.product((1, 2), (1, 2, 3), (8, 64)):
        for C in sorted({BS, 2 * BS, 256}):
            if C % BS:
                continue
            for n in sorted({0, 1, BS - 1, BS, BS + 1, C - 1, C, C + 1, 3 * C + BS + 1}):
                if n < 0:
                    continue
                nblk = -(-n // BS)
                NB = nblk + 3
                A = rng.integers(0, 1 << (8 * E), size=(L, NB, 2, H, BS, D), dtype=np.uint64).astype(_dt(E))
                # Store may name a block twice (two tokens can never share a slot, but
                # nothing in the definition forbids it): sample with replacement.
                bt = rng.integers(0, NB, size=nblk).astype(np.int32)
                nc = -(-n // C)
                num_slots = nc + 2
                cid = rng.permutation(num_slots)[:nc].astype(np.int64)
                rc, pool, sb = _run_pack(A, bt, n, C, cid, num_slots)
                assert rc == oracle.OK
                _check_pool(A, bt, n, C, pool, sb, cid)


# ---------------------------------------------------------------- P4: closed-form tags
def _tag(l, kv, t, h, d, H, D, T):
    return ((((l * 2 + kv) * T + t) * H + h) * D + d) + 1


@pytest.mark.parametrize("n", [4096, 4096 + 192, 4096 + 128, 4096 + 64, 4096 + 1, 4, 17])
def test_tags_closed_form(n):
    """E = 4, each cache word tags (l, kv, logical token, h, d): every chunk word must equal its tag."""
    L, H, D, BS, C = 2, 2, 64, 16, 256
    NB = 512
    nblk = -(-n // BS)
    bt = np.random.default_rng(7).permutation(NB)[:nblk].astype(np.int32)
    A = np.full((L, NB, 2, H, BS, D), 0xFFFFFFFF, dtype=np.uint32)
    l, kv, t, h, d = np.meshgrid(np.arange(L), np.arange(2), np.arange(n), np.arange(H), np.arange(D),
                                 indexing="ij")
    tags = _tag(l, kv, t, h, d, H, D, n).astype(np.uint32)
    scatter_tokens(A, bt, tags, BS)
    nc = -(-n // C)
    cid = np.arange(nc, dtype=np.int64)[::-1].copy()  # reversed slots
    rc, pool, sb = _run_pack(A, bt, n, C, cid, nc + 1)
    assert rc == oracle.OK
    for i in range(nc):
        r = min(C, n - i * C)
        got = pool[cid[i] * sb: cid[i] * sb + r * 2 * L * H * D * 4].view(np.uint32).reshape(L, 2, r, H, D)
        np.testing.assert_array_equal(got, tags[:, :, i * C:i * C + r])
        # Compact layout: nothing beyond r*TB in the slot.
        assert np.all(pool[cid[i] * sb + r * 2 * L * H * D * 4:(cid[i] + 1) * sb] == SENT)
    # Load into a fresh, differently fragmented cache: tags land at the new token slots only.
    bt2 = np.random.default_rng(8).permutation(NB)[:nblk].astype(np.int32)
    B = np.full_like(A, 0x5A5A5A5A)
    lay = oracle.make_layout(L, H, D, 4, BS, C)
    assert oracle.unpack(lay, _layers(B), 2 * H * BS * D * 4, NB, bt2, n, pool, cid) == oracle.OK
    np.testing.assert_array_equal(token_view(B, bt2, n, BS), tags)
    mask = np.ones(B.shape, dtype=bool)
    tt = np.arange(n)
    mask[:, bt2[tt // BS], :, :, tt % BS, :] = False
    assert np.all(B[mask] == 0x5A5A5A5A)


# ---------------------------------------------------------------- P2 + P3: round trip, untouched bytes
@pytest.mark.parametrize("n,nthreads", [(4096, 1), (4096, 5), (4096 + 192, 3), (4, 1), (0, 1), (300, 2)])
def test_round_trip_identity_and_sentinels(n, nthreads):
    L, H, D, E, BS, C = 2, 2, 64, 2, 16, 256
    NB = 512
    rng = np.random.default_rng(99 + n)
    A = rng.integers(0, 1 << 16, size=(L, NB, 2, H, BS, D), dtype=np.uint64).astype(np.uint16)
    nblk = -(-n // BS)
    perm = rng.permutation(NB)
    btA = perm[:nblk].astype(np.int32)
    btB = rng.permutation(NB)[:nblk].astype(np.int32)
    nc = -(-n // C)
    cid = rng.permutation(nc + 2)[:nc].astype(np.int64)
    rc, pool, sb = _run_pack(A, btA, n, C, cid, nc + 2, nthreads)
    assert rc == oracle.OK
    A_before = A.copy()
    B = np.full_like(A, 0xA5A5)
    lay = oracle.make_layout(L, H, D, E, BS, C)
    pool_before = pool.copy()
    assert oracle.unpack(lay, _layers(B), 2 * H * BS * D * E, NB, btB, n, pool, cid, nthreads) == oracle.OK
    np.testing.assert_array_equal(pool, pool_before)  # load only reads the pool
    np.testing.assert_array_equal(A, A_before)        # store only reads the cache
    np.testing.assert_array_equal(token_view(B, btB, n, BS), token_view(A, btA, n, BS))
    mask = np.ones(B.shape, dtype=bool)
    t = np.arange(n)
    mask[:, btB[t // BS], :, :, t % BS, :] = False
    assert np.all(B[mask] == 0xA5A5)


def test_padded_block_stride_untouched():
    """block_stride larger than one block: padding bytes are neither read into the pool nor written."""
    L, H, D, E, BS, C = 2, 2, 8, 4, 4, 8
    NB, pad = 10, 12  # extra elements per block
    blk = 2 * H * BS * D
    rng = np.random.default_rng(5)
    raw = rng.integers(0, 1 << 32, size=(L, NB, blk + pad), dtype=np.uint64).astype(np.uint32)
    n = 13
    bt = rng.permutation(NB)[:4].astype(np.int32)
    lay = oracle.make_layout(L, H, D, E, BS, C)
    sb = oracle.slot_bytes(lay)
    pool = np.full(2 * sb, SENT, dtype=np.uint8)
    layers = [raw[l].reshape(-1).view(np.uint8) for l in range(L)]
    stride = (blk + pad) * 4
    assert oracle.pack(lay, layers, stride, NB, bt, n, pool, [1, 0]) == oracle.OK
    A = np.ascontiguousarray(raw[:, :, :blk]).reshape(L, NB, 2, H, BS, D)
    _check_pool(A, bt, n, C, pool, sb, np.array([1, 0]))
    out = np.full_like(raw, 0x77777777)
    layers_out = [out[l].reshape(-1).view(np.uint8) for l in range(L)]
    assert oracle.unpack(lay, layers_out, stride, NB, bt, n, pool, [1, 0]) == oracle.OK
    assert np.all(out[:, :, blk:] == 0x77777777)
    B = np.ascontiguousarray(out[:, :, :blk]).reshape(L, NB, 2, H, BS, D)
    np.testing.assert_array_equal(token_view(B, bt, n, BS), token_view(A, bt, n, BS))


# ---------------------------------------------------------------- P5: degenerate cases
def test_single_head_block_equals_chunk_is_memcpy():
    """H = 1 and BS = C: each chunk plane is byte-for-byte the block's (l, kv) slab."""
    L, H, D, E, BS, C = 3, 1, 16, 2, 32, 32
    NB, n = 9, 5 * 32
    rng = np.random.default_rng(3)
    A = rng.integers(0, 1 << 16, size=(L, NB, 2, H, BS, D), dtype=np.uint64).astype(np.uint16)
    bt = rng.permutation(NB)[:5].astype(np.int32)
    rc, pool, sb = _run_pack(A, bt, n, C, np.arange(5), 5)
    assert rc == oracle.OK
    for i in range(5):
        for l in range(L):
            for kv in range(2):
                plane = pool[i * sb + (l * 2 + kv) * BS * D * E:i * sb + (l * 2 + kv + 1) * BS * D * E]
                assert plane.tobytes() == A[l, bt[i], kv].tobytes()


def test_identity_table_unit_blocks_is_reshape():
    """BS = 1 with the identity block table: the packed prefix is a transpose-reshape of the cache."""
    L, H, D, E, BS, C = 2, 3, 8, 4, 1, 4
    NB = n = 12
    rng = np.random.default_rng(4)
    A = rng.integers(0, 1 << 32, size=(L, NB, 2, H, BS, D), dtype=np.uint64).astype(np.uint32)
    rc, pool, sb = _run_pack(A, np.arange(NB, dtype=np.int32), n, C, np.arange(3), 3)
    assert rc == oracle.OK
    want = A[:, :, :, :, 0, :].transpose(0, 2, 1, 3, 4)  # [L][2][T][H][D]
    for i in range(3):
        got = pool[i * sb:(i + 1) * sb].view(np.uint32).reshape(L, 2, C, H, D)
        np.testing.assert_array_equal(got, want[:, :, i * C:(i + 1) * C])


def test_zero_tokens_is_noop():
    L, H, D, E, BS, C = 1, 1, 8, 2, 4, 8
    lay = oracle.make_layout(L, H, D, E, BS, C)
    A = np.zeros((L, 2, 2, H, BS, D), dtype=np.uint16)
    pool = np.full(oracle.slot_bytes(lay), SENT, dtype=np.uint8)
    assert oracle.pack(lay, _layers(A), 2 * H * BS * D * E, 2, np.zeros(0, np.int32), 0, pool, np.zeros(0)) == 0
    assert np.all(pool == SENT)
    assert oracle.unpack(lay, _layers(A), 2 * H * BS * D * E, 2, np.zeros(0, np.int32), 0, pool, np.zeros(0)) == 0
    assert np.all(A == 0)


# ---------------------------------------------------------------- brute force over tiny tables
def test_brute_force_all_tables_tiny():
    """Every block table (ordered choice of 3 of 4 blocks) x every slot assignment, BS = 1, C = 2."""
    L, H, D, E, BS, C = 1, 2, 4, 1, 1, 2
    NB, n = 4, 3
    rng = np.random.default_rng(11)
    A = rng.integers(0, 256, size=(L, NB, 2, H, BS, D), dtype=np.uint64).astype(np.uint8)
    cases = 0
    for bt in itertools.permutations(range(NB), 3):
        for cid in itertools.permutations(range(3), 2):
            bt_a = np.array(bt, dtype=np.int32)
            rc, pool, sb = _run_pack(A, bt_a, n, C, np.array(cid), 3)
            assert rc == oracle.OK
            # Hand enumeration of every output byte from the meaning of the layout.
            for i, r in ((0, 2), (1, 1)):
                for l, kv, u, h, d in itertools.product(range(L), range(2), range(r), range(H), range(D)):
                    t = i * C + u
                    want = A[l, bt[t], kv, h, 0, d]
                    pos = cid[i] * sb + (((l * 2 + kv) * r + u) * H + h) * D + d
                    assert pool[pos] == want
            cases += 1
    assert cases == 24 * 6


# ---------------------------------------------------------------- P7: raw bit patterns
def test_all_uint16_patterns_survive():
    """Every 16-bit pattern (NaN payloads, +-Inf, -0, subnormals as bf16) is moved bit-exactly."""
    L, H, D, E, BS, C = 1, 2, 64, 2, 16, 256
    # 65,536 values = 1 layer x 2 (K/V) x 2 heads x 64 dims x 256 tokens: 16 blocks.
    NB = 20
    A = np.full((L, NB, 2, H, BS, D), 0xDEAD, dtype=np.uint16)
    bt = np.random.default_rng(12).permutation(NB)[:16].astype(np.int32)
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(L, 2, 256, H, D)
    scatter_tokens(A, bt, pats, BS)
    rc, pool, sb = _run_pack(A, bt, 256, C, np.array([0]), 1)
    assert rc == oracle.OK
    np.testing.assert_array_equal(pool.view(np.uint16).reshape(L, 2, 256, H, D), pats)
    assert len(np.unique(pool.view(np.uint16))) == 65536


# ---------------------------------------------------------------- validation
def test_validation_rejects():
    lay = oracle.make_layout(2, 2, 64, 2, 16, 256)
    bs = 2 * 2 * 16 * 64 * 2
    bt = np.arange(16, dtype=np.int32)
    cid = np.arange(1, dtype=np.int64)
    ok = oracle.validate(lay, 16, bs, bt, 256, 1, cid, True)
    assert ok == oracle.OK
    assert oracle.validate(lay, 16, bs, bt, -1, 1, cid, True) == oracle.EINVAL
    assert oracle.validate(lay, 16, bs - 16, bt, 256, 1, cid, True) == oracle.EINVAL
    assert oracle.validate(lay, 15, bs, bt, 256, 1, cid, True) == oracle.EINVAL      # bt entry 15 out of range
    assert oracle.validate(lay, 0, bs, None, 0, 1, None, True) == oracle.EINVAL     # a cache without blocks
    assert oracle.validate(lay, 16, bs, bt, 256, 1, np.array([1]), True) == oracle.EINVAL  # slot out of range
    # Two chunks stored into one slot would leave the slot order dependent (last writer wins), so a
    # store naming a slot twice is refused; a load may read one slot into two places.  Every other
    # argument is valid here, so the duplicate is the only reason for the refusal.
    bt2 = np.arange(32, dtype=np.int32)
    assert oracle.validate(lay, 32, bs, bt2, 512, 2, np.array([0, 1]), True) == oracle.OK
    assert oracle.validate(lay, 32, bs, bt2, 512, 2, np.array([1, 1]), True) == oracle.EINVAL   # duplicate store slot
    assert oracle.validate(lay, 32, bs, bt2, 512, 2, np.array([1, 1]), False) == oracle.OK  # duplicate load slot
    A = np.zeros((2, 32, 2, 2, 16, 64), dtype=np.uint16)
    pool = np.full(2 * oracle.slot_bytes(lay), SENT, dtype=np.uint8)
    assert oracle.pack(lay, [A[l].reshape(-1).view(np.uint8) for l in range(2)], bs, 32, bt2, 512, pool,
                       [1, 1]) == oracle.EINVAL
    assert np.all(pool == SENT)  # refused before any byte moves
    assert oracle.validate(oracle.make_layout(2, 2, 64, 3, 16, 256), 16, 3 * bs, bt, 256, 1, cid, True) == oracle.EINVAL
    # Sec. 3.1: a chunk must be a whole number of pages; 1,568 tokens over 48-token pages is not.
    assert oracle.validate(oracle.make_layout(1, 1, 8, 1, 48, 1568), 64, 2 * 48 * 8, bt, 0, 0, None, True) == oracle.EINVAL
    assert oracle.validate(oracle.make_layout(1, 1, 8, 1, 32, 1568), 64, 2 * 32 * 8, bt, 0, 0, None, True) == oracle.OK


# ---------------------------------------------------------------- P8: the paper's chunk/page numbers
def _golden(name):
    rows = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = line.split("=", 1)
                rows[k.strip()] = int(v.strip().replace(",", ""))
    return rows


def test_paper_chunk_page_arithmetic():
    """Sec. 3.1/3.2: a 1,568-token chunk is 49 pages of 32 tokens; hits of 25,088 and 127,008 tokens
    are 16 and 81 whole chunks.  Run the oracle at those sizes (tiny per-token rows) and count."""
    g = _golden("paper_chunk_arithmetic.txt")
    C, page = g["chunk_tokens"], g["page_tokens"]
    assert g["pages_per_chunk"] * page == C
    L, H, D, E = 1, 1, 1, 4
    lay = oracle.make_layout(L, H, D, E, page, C)
    sb = oracle.slot_bytes(lay)
    for key in ("hit_tokens_small", "hit_tokens_large"):
        n = g[key]
        nblk = -(-n // page)
        NB = nblk + 5
        rng = np.random.default_rng(n)
        bt = rng.permutation(NB)[:nblk].astype(np.int32)
        # Each cache word holds its own physical block id, so a chunk's words name its pages.
        A = np.broadcast_to(np.arange(NB, dtype=np.uint32)[None, :, None, None, None, None],
                            (L, NB, 2, H, page, D)).copy()
        nc_slots = g[key.replace("hit_tokens", "chunks")] + 1
        pool = np.full(nc_slots * sb, SENT, dtype=np.uint8)
        nc = -(-n // C)
        assert nc == g[key.replace("hit_tokens", "chunks")]
        assert oracle.pack(lay, _layers(A), 2 * page * 4, NB, bt, n, pool, np.arange(nc)) == oracle.OK
        for i in range(nc):
            words = pool[i * sb:(i + 1) * sb].view(np.uint32)
            assert len(np.unique(words)) == g["pages_per_chunk"]  # whole chunk: every word written
        assert np.all(pool[nc * sb:] == SENT)


def test_paper_probe_signature():
    """Sec. 3.2: an unordered 1 MiB probe mismatches every byte (1,048,576).  With the tiny layout
    (1 KiB of KV per token) 1 MiB is 1,024 tokens: the oracle's store of a cache filled with the
    producer's byte 37 differs from a stale all-zero pool in exactly that many bytes."""
    g = _golden("paper_probes.txt")
    L, H, D, E, BS, C = 2, 2, 64, 2, 16, 256
    n = g["probe_bytes_1mib"] // (2 * L * H * D * E)
    assert n == 1024
    NB = 80
    A = np.full((L, NB, 2, H, BS, D), g["d2h_new_value"] * 0x0101, dtype=np.uint16)
    bt = np.random.default_rng(1).permutation(NB)[:n // BS].astype(np.int32)
    lay = oracle.make_layout(L, H, D, E, BS, C)
    pool = np.full(4 * oracle.slot_bytes(lay), g["old_value"], dtype=np.uint8)
    stale = pool.copy()
    assert oracle.pack(lay, _layers(A), 2 * H * BS * D * E, NB, bt, n, pool, np.arange(4)) == oracle.OK
    assert int(np.count_nonzero(pool != stale)) == g["mismatching_bytes_1mib"]
    assert np.all(pool == g["d2h_new_value"])
    # The control matrix's size: 3 sizes x 2 directions x 2 delays x 10 trials x 2 processes per control.
    cells = g["sizes"] * g["directions"] * g["delays"] * g["trials"] * g["processes"]
    assert cells // g["delays"] == g["raw_delayed_failures"] == g["raw_undelayed_passes"]
    assert cells * g["ordered_controls"] == g["ordered_passes"]

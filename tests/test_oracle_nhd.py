"""Pins for the oracle's token-major ("NHD") cache blocks [2][BS][H][D] (CPU only).

NHD is the cache layout the paper's packed-page patch rejected (Sec. 3.1); the
packed chunk format does not depend on the cache's block order, so the same
tokens must pack to the same bytes from either layout.
"""
import itertools

import numpy as np
import pytest

import oracle
from tests.numpy_formulation import expected_chunks, token_view, token_view_nhd

SENT = 0x3C


def _layers(A):
    return [A[l].reshape(-1).view(np.uint8) for l in range(A.shape[0])]


def _dt(E):
    return {1: np.uint8, 2: np.uint16, 4: np.uint32}[E]


def _pack(A, order, bt, n, L, H, D, E, BS, C, ids, slots):
    lay = oracle.make_layout(L, H, D, E, BS, C)
    pool = np.full(slots * oracle.slot_bytes(lay), SENT, dtype=np.uint8)
    rc = oracle.pack(lay, _layers(A), 2 * H * BS * D * E, A.shape[1], bt, n, pool, ids, 2, block_order=order)
    assert rc == oracle.OK
    return pool


@pytest.mark.parametrize("E,BS,C", [(1, 32, 1568), (2, 16, 256), (4, 1, 8), (2, 4, 4)])
def test_nhd_matches_numpy_formulation(E, BS, C):
    rng = np.random.default_rng(E * 100 + BS)
    for L, H, D in itertools.product((1, 2), (1, 3, 4), (16, 32)):
        for n in sorted({1, BS, C - 1, C, C + BS + 1, 2 * C + 3}):
            nblk = -(-n // BS)
            NB = nblk + 2
            A = rng.integers(0, 1 << (8 * E), size=(L, NB, 2, BS, H, D), dtype=np.uint64).astype(_dt(E))
            bt = rng.permutation(NB)[:nblk].astype(np.int32)
            nc = -(-n // C)
            ids = rng.permutation(nc + 1)[:nc]
            pool = _pack(A, oracle.BLOCK_NHD, bt, n, L, H, D, E, BS, C, ids, nc + 1)
            tv = token_view_nhd(A, bt, n, BS)
            sb = len(pool) // (nc + 1)
            written = np.zeros(len(pool), dtype=bool)
            for i in range(nc):
                ch = np.ascontiguousarray(tv[:, :, i * C:i * C + C])
                got = pool[ids[i] * sb:ids[i] * sb + ch.nbytes].view(A.dtype).reshape(ch.shape)
                np.testing.assert_array_equal(got, ch)
                written[ids[i] * sb:ids[i] * sb + ch.nbytes] = True
            assert np.all(pool[~written] == SENT)


def test_nhd_and_hnd_pack_the_same_tokens_identically():
    """Invariant: one set of tokens stored in an NHD cache and in an HND cache gives one pool."""
    L, H, D, E, BS, C = 2, 3, 8, 4, 4, 8
    NB, n = 11, 29
    rng = np.random.default_rng(9)
    A_nhd = rng.integers(0, 1 << 32, size=(L, NB, 2, BS, H, D), dtype=np.uint64).astype(np.uint32)
    A_hnd = np.ascontiguousarray(A_nhd.transpose(0, 1, 2, 4, 3, 5))  # [L][NB][2][H][BS][D]
    bt = rng.permutation(NB)[:8].astype(np.int32)
    ids = np.array([3, 0, 2, 1])
    p_nhd = _pack(A_nhd, oracle.BLOCK_NHD, bt, n, L, H, D, E, BS, C, ids, 4)
    p_hnd = _pack(A_hnd, oracle.BLOCK_HND, bt, n, L, H, D, E, BS, C, ids, 4)
    np.testing.assert_array_equal(p_nhd, p_hnd)
    np.testing.assert_array_equal(token_view_nhd(A_nhd, bt, n, BS), token_view(A_hnd, bt, n, BS))
    # Unpack into an NHD cache restores the NHD token view; untouched slots keep their fill.
    lay = oracle.make_layout(L, H, D, E, BS, C)
    B = np.full_like(A_nhd, 0x11111111)
    bt2 = rng.permutation(NB)[:8].astype(np.int32)
    assert oracle.unpack(lay, _layers(B), 2 * H * BS * D * E, NB, bt2, n, p_nhd, ids,
                         block_order=oracle.BLOCK_NHD) == oracle.OK
    np.testing.assert_array_equal(token_view_nhd(B, bt2, n, BS), token_view_nhd(A_nhd, bt, n, BS))
    mask = np.ones(B.shape, dtype=bool)
    t = np.arange(n)
    mask[:, bt2[t // BS], :, t % BS, :, :] = False
    assert np.all(B[mask] == 0x11111111)


def test_nhd_padded_block_stride():
    """Token-major blocks with a block stride larger than one block: the pool holds each block's
    unpadded token rows, and unpack writes no padding byte."""
    L, H, D, E, BS, C = 2, 3, 4, 4, 4, 8
    NB, pad = 9, 20  # extra 4-byte words after each block
    blk = 2 * BS * H * D
    rng = np.random.default_rng(17)
    raw = rng.integers(0, 1 << 32, size=(L, NB, blk + pad), dtype=np.uint64).astype(np.uint32)
    n = 21
    nblk = -(-n // BS)
    bt = rng.permutation(NB)[:nblk].astype(np.int32)
    lay = oracle.make_layout(L, H, D, E, BS, C)
    sb = oracle.slot_bytes(lay)
    stride = (blk + pad) * E
    pool = np.full(3 * sb, SENT, dtype=np.uint8)
    ids = np.array([2, 0, 1])
    layers = [raw[l].reshape(-1).view(np.uint8) for l in range(L)]
    assert oracle.pack(lay, layers, stride, NB, bt, n, pool, ids, block_order=oracle.BLOCK_NHD) == oracle.OK
    A = np.ascontiguousarray(raw[:, :, :blk]).reshape(L, NB, 2, BS, H, D)
    tv = token_view_nhd(A, bt, n, BS)
    for i in range(3):
        ch = np.ascontiguousarray(tv[:, :, i * C:i * C + C])
        got = pool[ids[i] * sb:ids[i] * sb + ch.nbytes].view(np.uint32).reshape(ch.shape)
        np.testing.assert_array_equal(got, ch)
    out = np.full_like(raw, 0x5A5A5A5A)
    layers_out = [out[l].reshape(-1).view(np.uint8) for l in range(L)]
    assert oracle.unpack(lay, layers_out, stride, NB, bt, n, pool, ids, block_order=oracle.BLOCK_NHD) == oracle.OK
    assert np.all(out[:, :, blk:] == 0x5A5A5A5A)
    B = np.ascontiguousarray(out[:, :, :blk]).reshape(L, NB, 2, BS, H, D)
    np.testing.assert_array_equal(token_view_nhd(B, bt, n, BS), tv)


def test_nhd_tags_paper_geometry():
    """The paper's attention geometry (FP8-sized 1-byte elements, 32-token pages, 1,568-token chunks,
    Sec. 3.1 / Table 1) in an NHD cache; E = 4 tags keep every word unique."""
    L, H, D, E, BS, C = 2, 4, 4, 4, 32, 1568
    n = 1568 + 931
    nblk = -(-n // BS)
    NB = nblk + 3
    bt = np.random.default_rng(4).permutation(NB)[:nblk].astype(np.int32)
    A = np.full((L, NB, 2, BS, H, D), 0xFFFFFFFF, dtype=np.uint32)
    l, kv, t, h, d = np.meshgrid(np.arange(L), np.arange(2), np.arange(n), np.arange(H), np.arange(D),
                                 indexing="ij")
    tags = (((((l * 2 + kv) * n + t) * H + h) * D + d) + 1).astype(np.uint32)
    tt = np.arange(n)
    A[:, bt[tt // BS], :, tt % BS, :, :] = tags.transpose(2, 0, 1, 3, 4)
    pool = _pack(A, oracle.BLOCK_NHD, bt, n, L, H, D, E, BS, C, np.array([1, 0]), 2)
    sb = len(pool) // 2
    for i, slot in ((0, 1), (1, 0)):
        r = min(C, n - i * C)
        got = pool[slot * sb:slot * sb + r * 2 * L * H * D * E].view(np.uint32).reshape(L, 2, r, H, D)
        np.testing.assert_array_equal(got, tags[:, :, i * C:i * C + r])


def test_unknown_block_order_rejected():
    lay = oracle.make_layout(1, 1, 16, 1, 4, 8)
    A = np.zeros((1, 2, 2, 4, 1, 16), dtype=np.uint8)
    pool = np.zeros(oracle.slot_bytes(lay), dtype=np.uint8)
    assert oracle.pack(lay, _layers(A), 128, 2, np.array([0], np.int32), 4, pool, [0], block_order=2) == oracle.EINVAL

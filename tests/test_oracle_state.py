"""Pins for the oracle's recurrent-state snapshot pages (Sec. 2.2), CPU only.

The expected values never come from byte offsets: an independent numpy formulation indexes a
stacked page array A[G][num_pages][page_stride] by page ids and lets advanced indexing build the
packed slots; closed-form word tags, round trips, untouched sentinels and validation rules pin
the rest.
"""
import numpy as np
import pytest

import oracle

SENT = 0xC3


def _layers(A):
    return [np.ascontiguousarray(A[g]).reshape(-1) for g in range(A.shape[0])]


def _formulation(A, page_bytes, pages, num_slots, slot_ids):
    """pool[slot_ids[k]] = concatenation over g of A[g, pages[k], :page_bytes]."""
    G = A.shape[0]
    pool = np.full((num_slots, G, page_bytes), SENT, dtype=np.uint8)
    pool[np.asarray(slot_ids, dtype=np.int64)] = A[:, np.asarray(pages, dtype=np.int64), :page_bytes].transpose(1, 0, 2)
    return pool.reshape(-1)


CASES = [  # G, page_bytes, page_stride, num_pages, n, num_slots
    (1, 1, 1, 1, 1, 1),
    (1, 16, 48, 5, 3, 4),
    (3, 64, 80, 7, 4, 6),
    (4, 48, 48, 9, 9, 9),
    (5, 13, 29, 11, 6, 8),
    (2, 4096, 4352, 4, 2, 3),
]


@pytest.mark.parametrize("G,pb,stride,npages,n,nslots", CASES)
def test_pack_matches_numpy_formulation(G, pb, stride, npages, n, nslots):
    rng = np.random.default_rng(hash((G, pb, stride, npages, n, nslots)) & 0xFFFF)
    A = rng.integers(0, 256, size=(G, npages, stride), dtype=np.uint8)
    pages = rng.choice(npages, size=n, replace=n > npages)
    slots = rng.permutation(nslots)[:n]
    pool = np.full(nslots * G * pb, SENT, dtype=np.uint8)
    assert oracle.state_pack(_layers(A), pb, stride, pages, pool, slots) == oracle.OK
    assert np.array_equal(pool, _formulation(A, pb, pages, nslots, slots))


def test_word_tags_closed_form():
    """With 4-byte words tagged (g, page, word), every word of slot s equals the tag of the page
    snapshot k = slot_ids.index(s) in layer g."""
    G, npages, words, stride_words = 3, 6, 24, 28
    g, p, w = np.meshgrid(np.arange(G), np.arange(npages), np.arange(stride_words), indexing="ij")
    A = ((g << 20) | (p << 10) | w).astype(np.uint32)
    pages, slots = np.array([4, 0, 5, 2]), np.array([1, 3, 0, 2])
    pool = np.zeros(4 * G * words, dtype=np.uint32)
    assert oracle.state_pack([np.ascontiguousarray(A[i]).view(np.uint8).reshape(-1) for i in range(G)], words * 4,
                             stride_words * 4, pages, pool.view(np.uint8), slots) == oracle.OK
    got = pool.reshape(4, G, words)
    for k in range(4):
        for gg in range(G):
            for ww in range(words):
                assert got[slots[k], gg, ww] == (gg << 20) | (pages[k] << 10) | ww


def test_round_trip_restores_pages_and_leaves_the_rest():
    G, pb, stride, npages = 3, 40, 56, 8
    rng = np.random.default_rng(7)
    A = rng.integers(0, 256, size=(G, npages, stride), dtype=np.uint8)
    pagesA, pagesB, slots = np.array([6, 1, 3]), np.array([0, 7, 2]), np.array([2, 0, 4])
    pool = np.full(5 * G * pb, SENT, dtype=np.uint8)
    assert oracle.state_pack(_layers(A), pb, stride, pagesA, pool, slots) == oracle.OK
    untouched = np.setdiff1d(np.arange(5), slots)
    assert (pool.reshape(5, -1)[untouched] == SENT).all()
    B = np.full_like(A, 0x5A)
    layersB = _layers(B)
    assert oracle.state_unpack(layersB, pb, stride, pagesB, pool, slots) == oracle.OK
    Bg = np.stack([x.reshape(npages, stride) for x in layersB])
    assert np.array_equal(Bg[:, pagesB, :pb], A[:, pagesA, :pb])
    assert (Bg[:, pagesB, pb:] == 0x5A).all(), "padding between pages was written"
    others = np.setdiff1d(np.arange(npages), pagesB)
    assert (Bg[:, others] == 0x5A).all(), "a page outside the request was written"


def test_last_page_needs_only_page_bytes():
    """A layer buffer may end right after its last page (no trailing stride padding)."""
    G, pb, stride, npages = 2, 32, 64, 3
    rng = np.random.default_rng(11)
    full = rng.integers(0, 256, size=(G, npages, stride), dtype=np.uint8)
    layers = [np.ascontiguousarray(full[g].reshape(-1)[:(npages - 1) * stride + pb]) for g in range(G)]
    pool = np.zeros(G * pb, dtype=np.uint8)
    assert oracle.state_pack(layers, pb, stride, [npages - 1], pool, [0]) == oracle.OK
    assert np.array_equal(pool.reshape(G, pb), full[:, npages - 1, :pb])


def test_validation_rules():
    v = oracle.state_validate
    assert v(2, 16, 32, 4, [0, 3], 2, 2, [1, 0], True) == oracle.OK
    assert v(2, 16, 32, 4, None, 0, 0, None, True) == oracle.OK                 # n = 0
    assert v(0, 16, 32, 4, [0], 1, 2, [0], True) == oracle.EINVAL               # no layers
    assert v(2, 0, 32, 4, [0], 1, 2, [0], True) == oracle.EINVAL                # empty page
    assert v(2, 16, 8, 4, [0], 1, 2, [0], True) == oracle.EINVAL                # stride < page
    assert v(2, 16, 32, 4, [4], 1, 2, [0], True) == oracle.EINVAL               # page out of range
    assert v(2, 16, 32, 4, [-1], 1, 2, [0], True) == oracle.EINVAL
    assert v(2, 16, 32, 4, [0], 1, 2, [2], True) == oracle.EINVAL               # slot out of range
    assert v(2, 16, 32, 4, [0], 1, 2, [2], False) == oracle.EINVAL              # ... for a load as well
    assert v(2, 16, 32, 4, [0, 1], 2, 2, [1, 1], True) == oracle.EINVAL         # store writes one slot twice
    assert v(2, 16, 32, 4, [0, 1], 2, 2, [1, 1], False) == oracle.OK            # a load may read it twice
    assert v(2, 16, 32, 4, [2, 2], 2, 2, [0, 1], False) == oracle.EINVAL        # load writes one page twice
    assert v(2, 16, 32, 4, [2, 2], 2, 2, [0, 1], True) == oracle.OK             # a store may read it twice
    assert v(2, 16, 32, 4, None, 1, 2, [0], True) == oracle.EINVAL              # missing ids
    assert v(2, 16, 32, 4, [0], -1, 2, [0], True) == oracle.EINVAL


def test_rejected_request_writes_nothing():
    A = np.arange(2 * 3 * 16, dtype=np.uint8).reshape(2, 3, 16)
    pool = np.full(2 * 2 * 16, SENT, dtype=np.uint8)
    assert oracle.state_pack(_layers(A), 16, 16, [0, 1], pool, [1, 1]) == oracle.EINVAL
    assert (pool == SENT).all()


def test_null_layer_pointer_rejected():
    """A snapshot request whose layer list holds a NULL pointer is refused before any byte moves."""
    import ctypes
    A = np.arange(2 * 3 * 16, dtype=np.uint8).reshape(2, 3, 16)
    pool = np.full(2 * 2 * 16, SENT, dtype=np.uint8)
    layers = (ctypes.c_void_p * 2)(np.ascontiguousarray(A[0]).ctypes.data, None)
    pages = np.array([0, 1], dtype=np.int64)
    slots = np.array([0, 1], dtype=np.int64)
    rc = oracle._load().oracle_state_pack(2, 16, 16, 3, layers, pages.ctypes.data, 2, pool.ctypes.data, 2,
                                          slots.ctypes.data)
    assert rc == oracle.EINVAL and (pool == SENT).all()

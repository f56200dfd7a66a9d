"""The seeded input generators (CPU): known answers and distribution properties."""
import numpy as np

import harness


def test_splitmix64_published_vectors():
    # First five outputs of SplitMix64 seeded with 1234567, as published with the
    # reference implementation (Vigna, splitmix64.c).
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423,
            4593380528125082431, 16408922859458223821]
    assert [int(x) for x in harness.splitmix_at(1234567, np.arange(5))] == want


def test_bf16_round_to_nearest_even():
    f = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0, -0.0, 1.0 + 2 ** -9], dtype=np.float32)
    assert [int(x) for x in harness.f32_to_bf16_rne(f)] == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x0000, 0x8000, 0x3F80]


def _bf16_to_f32(b):
    return (b.astype(np.uint32) << 16).view(np.float32)


def test_uniform_and_normal_shapes():
    z = harness.splitmix_at(42, np.arange(1 << 20))
    u = _bf16_to_f32(harness.values_from_z(z, "u11", 2))
    assert u.min() >= -1.0 and u.max() <= 1.0
    assert abs(u.mean()) < 5e-3 and abs(u.var() - 1 / 3) < 5e-3
    g = _bf16_to_f32(harness.values_from_z(z, "n01", 2))
    assert abs(g.mean()) < 5e-3 and abs(g.std() - 1.0) < 1e-2
    assert np.abs(g).max() <= 3.47
    r = harness.values_from_z(z, "raw", 2)
    assert r.dtype == np.uint16 and len(np.unique(r)) > 60000


def test_block_subset_regenerates_same_values():
    full = harness.gen_cache(7, "u11", 2, 10, 2, 4, 8, 2)
    part = harness.gen_blocks(7, "u11", 2, 10, 2, 4, 8, 2, layers=[1], blocks=[9, 3])
    np.testing.assert_array_equal(part[0, 0], full[1, 9])
    np.testing.assert_array_equal(part[0, 1], full[1, 3])


def test_block_tables():
    bt = harness.block_table(5, 512, 256)
    assert len(set(bt.tolist())) == 256 and bt.min() >= 0 and bt.max() < 512
    bt2 = harness.block_table(6, 512, 256, exclude=bt)
    assert not set(bt.tolist()) & set(bt2.tolist())
    assert sorted(bt.tolist() + bt2.tolist()) == list(range(512))
    d = harness.spin_delays_ms(1, 100)
    assert d.min() >= 5.0 and d.max() <= 50.0

"""The device twin of the seeded generator matches the host generator bit for bit."""
import numpy as np
import pytest
import torch

import harness
from harness import gpu as hg
from tests.gpu_support import TORCH_INT

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dist,E", [("u11", 2), ("n01", 2), ("raw", 2), ("raw", 1), ("raw", 4)])
@pytest.mark.parametrize("k", range(4))
def test_device_fill_matches_host(dist, E, k):
    L, NB, H, BS, D = 2, 37, 2, 16, 64
    seed = harness.sub_seed("twin", dist, E, k)
    want = harness.gen_cache(seed, dist, L, NB, H, BS, D, E)
    t = torch.empty(want.shape, dtype=TORCH_INT[E], device="cuda:0")
    hg.fill_values(t, 0, seed, dist, E)
    torch.cuda.synchronize()
    got = t.cpu().numpy().view(want.dtype)
    np.testing.assert_array_equal(got, want)
    # A sub-range at a counter offset: the block (1, 5) regenerated alone.
    part = torch.empty((2, H, BS, D), dtype=TORCH_INT[E], device="cuda:0")
    hg.fill_values(part, (1 * NB + 5) * 2 * H * BS * D, seed, dist, E)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(part.cpu().numpy().view(want.dtype), want[1, 5])

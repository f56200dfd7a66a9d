"""A native C program calls the C ABI directly (tests/native/kvx_native_caller.c: plain C against
include/kvx.h and the HIP C API; no Python binding, no torch in that process).  Inputs come from
the seeded generator and are handed over as files; the pool and the restored cache it writes back
are compared with the CPU oracle byte for byte, in both transfer modes."""
import os
import subprocess

import numpy as np
import pytest

import harness
from paper_2609_15021_amd import build
from tests.gpu_support import TINY, Layout, first_mismatch, host_cache, oracle_pool, oracle_unpack_into

pytestmark = pytest.mark.gpu

POOL_SENT, CACHE_SENT = 0xA5, 0x5A


@pytest.mark.parametrize("mode", ["staged", "zero_copy"])
@pytest.mark.parametrize("dims,NB,n", [((2, 2, 64, 2, 16, 256), 512, 4096 + 192),
                                       ((16, 4, 256, 1, 32, 1568), 160, 3 * 1568 + 100)],
                         ids=["tiny", "paper-geometry"])
def test_native_caller_round_trip(mode, dims, NB, n, tmp_path):
    assert os.path.exists(build.NATIVE_BIN), "native caller not built; run __graft_entry__.build()"
    lay = Layout(*dims)
    seed = harness.sub_seed("native", mode, lay.L)
    A = host_cache(lay, NB, seed, "raw")
    nblk, nc = lay.nblk(n), lay.nc(n)
    btA, btB = harness.block_table(seed + 1, NB, nblk), harness.block_table(seed + 2, NB, nblk)
    nslots = nc + 2
    ids = harness.chunk_ids(nc, nslots, seed + 3)
    A.tofile(tmp_path / "a.bin")
    np.asarray(btA, dtype=np.int32).tofile(tmp_path / "bta.bin")
    np.asarray(btB, dtype=np.int32).tofile(tmp_path / "btb.bin")
    np.asarray(ids, dtype=np.int64).tofile(tmp_path / "ids.bin")
    print(f"[native] mode={mode} dims={dims} NB={NB} n={n}", flush=True)
    r = subprocess.run([build.NATIVE_BIN, mode, *map(str, dims), str(NB), str(n), str(nslots), str(tmp_path)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "NATIVE OK" in r.stdout, (r.stdout + r.stderr)[-2000:]
    pool = np.fromfile(tmp_path / "pool.bin", dtype=np.uint8)
    want_pool = oracle_pool(lay, A, btA, n, ids, nslots, POOL_SENT)
    assert np.array_equal(pool, want_pool), "pool: " + first_mismatch(pool, want_pool)
    B0 = np.full(A.shape, 0, dtype=A.dtype)
    B0.view(np.uint8)[:] = CACHE_SENT
    want_B = oracle_unpack_into(lay, B0, btB, n, want_pool, ids)
    got_B = np.fromfile(tmp_path / "b.bin", dtype=A.dtype).reshape(A.shape)
    assert np.array_equal(got_B, want_B), "cache B: " + first_mismatch(got_B, want_B)

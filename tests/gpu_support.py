"""Helpers for the GPU tests: seeded inputs on host and device, oracle expectations.

Expected values always come from the oracle applied to host-generated inputs
(``harness`` generator); nothing expected is ever read back from the HIP path.
"""
from __future__ import annotations

import numpy as np
import torch

import harness
import oracle
from paper_2609_15021_amd import kvx

DEV = torch.device("cuda:0")
TORCH_INT = {1: torch.uint8, 2: torch.int16, 4: torch.int32}
NP_SIGNED = {1: np.uint8, 2: np.int16, 4: np.int32}


class Layout:
    def __init__(self, L, H, D, E, BS, C):
        self.L, self.H, self.D, self.E, self.BS, self.C = L, H, D, E, BS, C
        self.kv = kvx.make_layout(L, H, D, E, BS, C)
        self.orc = oracle.make_layout(L, H, D, E, BS, C)
        self.block_elems = 2 * H * BS * D
        self.block_bytes = self.block_elems * E
        self.token_bytes = 2 * L * H * D * E
        self.slot_bytes = C * self.token_bytes

    def nc(self, n):
        return -(-n // self.C)

    def nblk(self, n):
        return -(-n // self.BS)


TINY = Layout(2, 2, 64, 2, 16, 256)
B27 = Layout(64, 8, 128, 2, 16, 256)


def host_cache(lay: Layout, NB: int, seed: int, dist: str) -> np.ndarray:
    """Host cache [L][NB][2][H][BS][D] from the seeded generator."""
    return harness.gen_cache(seed, dist, lay.L, NB, lay.H, lay.BS, lay.D, lay.E)


def to_device(a: np.ndarray) -> torch.Tensor:
    E = a.dtype.itemsize
    return torch.from_numpy(np.ascontiguousarray(a).view(NP_SIGNED[E])).to(DEV)


def to_host(t: torch.Tensor, like: np.ndarray) -> np.ndarray:
    return t.cpu().numpy().view(like.dtype).reshape(like.shape)


def device_cache(lay: Layout, NB: int, fill=None) -> torch.Tensor:
    shape = (lay.L, NB, 2, lay.H, lay.BS, lay.D)
    t = torch.empty(shape, dtype=TORCH_INT[lay.E], device=DEV)
    if fill is not None:
        t.view(torch.uint8).fill_(fill)
    return t


def layers_of(a: np.ndarray):
    return [a[l].reshape(-1).view(np.uint8) for l in range(a.shape[0])]


def oracle_pool(lay: Layout, A: np.ndarray, bt, n, chunk_ids, num_slots, sentinel) -> np.ndarray:
    pool = np.full(num_slots * lay.slot_bytes, sentinel, dtype=np.uint8)
    rc = oracle.pack(lay.orc, layers_of(A), lay.block_bytes, A.shape[1], bt, n, pool, chunk_ids, nthreads=4)
    assert rc == oracle.OK
    return pool


def oracle_unpack_into(lay: Layout, B: np.ndarray, bt, n, pool: np.ndarray, chunk_ids) -> np.ndarray:
    out = B.copy()
    rc = oracle.unpack(lay.orc, layers_of(out), lay.block_bytes, out.shape[1], bt, n, pool, chunk_ids, nthreads=4)
    assert rc == oracle.OK
    return out


def bt_tensor(bt: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)


def first_mismatch(got: np.ndarray, want: np.ndarray) -> str:
    g, w = got.reshape(-1).view(np.uint8), want.reshape(-1).view(np.uint8)
    bad = np.flatnonzero(g != w)
    if bad.size == 0:
        return "equal"
    return f"{bad.size} bytes differ; first at byte {bad[0]}: got {g[bad[0]]} want {w[bad[0]]}"

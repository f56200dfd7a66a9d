"""Seeded synthetic inputs for the KV store/load tests and benchmark.

This module holds none of the store/load arithmetic: it only makes inputs
(cache values, block tables, chunk ids, producer delays).  Both the oracle side
and the HIP side of a test draw their inputs from here, so it must stay free of
any gather/scatter logic.

Value generator (host twin of ``harness.hip``'s ``kvh_fill_cache`` kernel; the
two must agree bit for bit, which ``tests/test_gpu_inputs.py`` checks):

* counter-based SplitMix64 (Steele, Lea and Flood, "Fast splittable
  pseudorandom number generators", OOPSLA 2014): output k of stream ``seed`` is
  ``mix64(seed + (k + 1) * 0x9E3779B97F4A7C15)`` with the published finaliser
  ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27; z *= 0x94D049BB133111EB;
  z ^= z >> 31`` (all mod 2**64);
* the counter k of a cache element is its linear element index in the
  layer-stacked, packed cache ``[L][NB][2][H][BS][D]`` (so any block can be
  regenerated on its own);
* distributions: ``"u11"`` bf16 ~U[-1, 1): ((z >> 40) - 2**23) * 2**-23, exact in
  fp32, then bf16 by integer round-to-nearest-even; ``"n01"`` bf16 ~N(0, 1)
  (Irwin-Hall): the four 16-bit fields of z summed, minus 131070, times fp32
  sqrt(3)/65536 (one IEEE rounding), then bf16 RNE; ``"raw"``: the low 8*E bits
  of z (every bit pattern, NaN payloads included, for E = 1, 2 or 4).
"""
from __future__ import annotations

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
M1 = np.uint64(0xBF58476D1CE4E5B9)
M2 = np.uint64(0x94D049BB133111EB)
N01_SCALE = np.float32(np.sqrt(np.float64(3.0)) / 65536.0)

# Base seed: the request seed the paper's workloads use (Sec. 4.2).
BASE_SEED = 314159

DISTS = ("u11", "n01", "raw")


def sub_seed(*parts) -> int:
    """Derive a 64-bit sub-seed from the base seed and a purpose path, e.g. ("values", "A", 2)."""
    h = np.uint64(BASE_SEED)
    with np.errstate(over="ignore"):
        for p in parts:
            if isinstance(p, str):
                v = np.uint64(int.from_bytes(p.encode()[:8].ljust(8, b"\0"), "little"))
            else:
                v = np.uint64(int(p) & 0xFFFFFFFFFFFFFFFF)
            h = mix64(np.array([h ^ v], dtype=np.uint64) + GAMMA)[0]
    return int(h)


def mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser, elementwise on a uint64 array."""
    z = np.asarray(z, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= M1
        z ^= z >> np.uint64(27)
        z *= M2
        z ^= z >> np.uint64(31)
    return z


def splitmix_at(seed: int, counters: np.ndarray) -> np.ndarray:
    """Output of stream ``seed`` at 64-bit counters ``counters``."""
    c = np.asarray(counters, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return mix64(np.uint64(seed) + (c + np.uint64(1)) * GAMMA)


def f32_to_bf16_rne(f: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 bits, round-to-nearest-even, by integer arithmetic (no NaN input)."""
    u = np.asarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    return ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)


def values_from_z(z: np.ndarray, dist: str, elem_bytes: int) -> np.ndarray:
    """Map SplitMix64 outputs to element values (as unsigned integers of elem_bytes)."""
    if dist == "raw":
        dt = {1: np.uint8, 2: np.uint16, 4: np.uint32}[elem_bytes]
        return (z & np.uint64((1 << (8 * elem_bytes)) - 1)).astype(dt)
    if elem_bytes != 2:
        raise ValueError(f"dist {dist!r} is bf16 and needs elem_bytes == 2")
    if dist == "u11":
        k = (z >> np.uint64(40)).astype(np.int64) - (1 << 23)
        f = k.astype(np.float32) * np.float32(2.0 ** -23)
        return f32_to_bf16_rne(f)
    if dist == "n01":
        m = np.uint64(0xFFFF)
        s = ((z & m) + ((z >> np.uint64(16)) & m) + ((z >> np.uint64(32)) & m)
             + ((z >> np.uint64(48)) & m)).astype(np.int64) - 131070
        f = s.astype(np.float32) * N01_SCALE
        return f32_to_bf16_rne(f)
    raise ValueError(f"unknown dist {dist!r}")


def element_dtype(elem_bytes: int):
    return {1: np.uint8, 2: np.uint16, 4: np.uint32}[elem_bytes]


def gen_blocks(seed: int, dist: str, L: int, NB: int, H: int, BS: int, D: int, E: int,
               layers=None, blocks=None) -> np.ndarray:
    """Values of selected (layer, block) pieces of the packed cache [L][NB][2][H][BS][D].

    Returns an array [len(layers)][len(blocks)][2][H][BS][D] of unsigned ints of E
    bytes, generated from the element counters of those blocks only.
    """
    layers = np.arange(L) if layers is None else np.asarray(layers, dtype=np.int64)
    blocks = np.arange(NB) if blocks is None else np.asarray(blocks, dtype=np.int64)
    be = 2 * H * BS * D
    e = np.arange(be, dtype=np.uint64)
    base = (layers[:, None].astype(np.uint64) * np.uint64(NB) + blocks[None, :].astype(np.uint64)) * np.uint64(be)
    ctr = base[:, :, None] + e[None, None, :]
    z = splitmix_at(seed, ctr.reshape(-1))
    v = values_from_z(z, dist, E)
    return v.reshape(len(layers), len(blocks), 2, H, BS, D)


def gen_cache(seed: int, dist: str, L: int, NB: int, H: int, BS: int, D: int, E: int) -> np.ndarray:
    """The whole packed cache [L][NB][2][H][BS][D]."""
    return gen_blocks(seed, dist, L, NB, H, BS, D, E)


def block_table(seed: int, num_blocks: int, n_used: int, exclude=None) -> np.ndarray:
    """A seeded random selection of n_used distinct blocks, in random order.

    Fisher-Yates over 0..num_blocks-1 (numpy's permutation), dropping ``exclude``,
    then the first n_used.  Accidental adjacent pairs are allowed; nothing may
    rely on contiguity.
    """
    perm = np.random.default_rng(seed).permutation(num_blocks)
    if exclude is not None:
        ex = np.zeros(num_blocks, dtype=bool)
        ex[np.asarray(exclude, dtype=np.int64)] = True
        perm = perm[~ex[perm]]
    if n_used > len(perm):
        raise ValueError(f"need {n_used} blocks, only {len(perm)} available")
    return perm[:n_used].astype(np.int32)


def chunk_ids(n_chunks: int, num_slots: int, seed=None, first: int = 0) -> np.ndarray:
    """Slot ids for n_chunks chunks: sequential from ``first`` or, with a seed, a random distinct draw."""
    if seed is None:
        return np.arange(first, first + n_chunks, dtype=np.int64)
    return np.random.default_rng(seed).permutation(num_slots)[:n_chunks].astype(np.int64)


def spin_delays_ms(seed: int, count: int, lo: float = 5.0, hi: float = 50.0) -> np.ndarray:
    """Seeded producer delays in [lo, hi] milliseconds."""
    return np.random.default_rng(seed).uniform(lo, hi, size=count)


def prompt_tokens(seed: int, n: int, vocab: int = 151000) -> np.ndarray:
    """A seeded synthetic prompt of n token ids (int32); prompts sharing a prefix come from
    slicing or concatenating these."""
    return np.random.default_rng(seed).integers(0, vocab, size=n).astype(np.int32)

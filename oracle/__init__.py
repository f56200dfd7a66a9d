"""CPU oracle for the shared-KV store/load path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package.  The product path (``paper_2609_15021_amd``) never
imports, links or runs it, and the two share no code: this package wraps the
plain C library ``libkvx_oracle.so`` built from ``kvx_oracle.c`` with gcc.

What the oracle computes is the plain definition of the paper's state transfer
(Sec. 2.2: KV state as opaque bytes; Sec. 3.1: a logical chunk spans a whole
number of paged blocks, and the layout is validated rather than inferred), and
the hybrid model's recurrent-state snapshot pages moved as opaque bytes (Sec.
2.2).  See ``kvx_oracle.h`` for the exact byte-level definitions, and
``recovery.py`` for the aligned-recovery rule.

Every function here is pinned by ``tests/test_oracle_*.py`` against values and
properties the paper and the mathematics fix (numpy fancy-indexing
formulation, closed-form coordinate tags, round-trip identity, untouched
sentinels, degenerate cases, the paper's chunk/page arithmetic).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvx_oracle.c")
LIB_PATH = os.path.join(_HERE, "libkvx_oracle.so")
# Test hook: the mutation test points this at a deliberately broken copy of the
# oracle to prove the pins catch it.  Never set outside tests/.
_LIB_OVERRIDE = os.environ.get("KVX_ORACLE_LIB")

OK = 0
EINVAL = -1
BLOCK_HND = 0  # cache block [2][H][BS][D]
BLOCK_NHD = 1  # cache block [2][BS][H][D]


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (plain C11, pthreads) into ``libkvx_oracle.so``."""
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror",
           "-o", LIB_PATH + ".tmp", _SRC, "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


class OracleLayout(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("chunk_tokens", ctypes.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = _LIB_OVERRIDE or LIB_PATH
    if not _LIB_OVERRIDE and not os.path.exists(LIB_PATH):
        build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_slot_bytes.argtypes = [ctypes.POINTER(OracleLayout)]
    lib.oracle_slot_bytes.restype = i64
    lib.oracle_validate.argtypes = [ctypes.POINTER(OracleLayout), i64, i64, P, i64, i64, P, ctypes.c_int]
    lib.oracle_validate.restype = ctypes.c_int
    for fn in (lib.oracle_pack, lib.oracle_unpack):
        fn.argtypes = [ctypes.POINTER(OracleLayout), ctypes.c_int, P, i64, i64, P, i64, P, i64, P, ctypes.c_int]
        fn.restype = ctypes.c_int
    lib.oracle_state_validate.argtypes = [i64, i64, i64, i64, P, i64, i64, P, ctypes.c_int]
    lib.oracle_state_validate.restype = ctypes.c_int
    for fn in (lib.oracle_state_pack, lib.oracle_state_unpack):
        fn.argtypes = [i64, i64, i64, i64, P, P, i64, P, i64, P]
        fn.restype = ctypes.c_int
    _lib = lib
    return lib


def make_layout(L, H, D, E, BS, C) -> OracleLayout:
    return OracleLayout(L, H, D, E, BS, C)


def slot_bytes(lay: OracleLayout) -> int:
    return int(_load().oracle_slot_bytes(ctypes.byref(lay)))


def _ptr(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _layer_ptr_array(layers):
    arr = (ctypes.c_void_p * len(layers))()
    for i, a in enumerate(layers):
        arr[i] = a.ctypes.data
    return arr


def _check_bytes(a, name, writable=False):
    if not isinstance(a, np.ndarray) or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous numpy array")
    if writable and not a.flags.writeable:
        raise TypeError(f"{name} must be writable")


def validate(lay, num_blocks, block_stride, block_table, n_tokens, num_slots, chunk_ids, for_pack):
    bt = None if block_table is None else np.ascontiguousarray(block_table, dtype=np.int32)
    ci = None if chunk_ids is None else np.ascontiguousarray(chunk_ids, dtype=np.int64)
    return int(_load().oracle_validate(ctypes.byref(lay), int(num_blocks), int(block_stride), _ptr(bt),
                                       int(n_tokens), int(num_slots), _ptr(ci), int(bool(for_pack))))


def pack(lay, layers, block_stride, num_blocks, block_table, n_tokens, pool, chunk_ids, nthreads=1,
         block_order=BLOCK_HND):
    """Store: cache layers (list of L host byte arrays) -> pool (uint8, num_slots*slot_bytes)."""
    for k, a in enumerate(layers):
        _check_bytes(a, f"layers[{k}]")
    _check_bytes(pool, "pool", writable=True)
    sb = slot_bytes(lay)
    num_slots = pool.nbytes // sb
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    ci = np.ascontiguousarray(chunk_ids, dtype=np.int64)
    return int(_load().oracle_pack(ctypes.byref(lay), int(block_order), _layer_ptr_array(layers), int(num_blocks),
                                   int(block_stride), _ptr(bt), int(n_tokens), _ptr(pool),
                                   int(num_slots), _ptr(ci), int(nthreads)))


def unpack(lay, layers, block_stride, num_blocks, block_table, n_tokens, pool, chunk_ids, nthreads=1,
           block_order=BLOCK_HND):
    """Load: pool -> cache layers (list of L writable host byte arrays)."""
    for k, a in enumerate(layers):
        _check_bytes(a, f"layers[{k}]", writable=True)
    _check_bytes(pool, "pool")
    sb = slot_bytes(lay)
    num_slots = pool.nbytes // sb
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    ci = np.ascontiguousarray(chunk_ids, dtype=np.int64)
    return int(_load().oracle_unpack(ctypes.byref(lay), int(block_order), _layer_ptr_array(layers), int(num_blocks),
                                     int(block_stride), _ptr(bt), int(n_tokens), _ptr(pool),
                                     int(num_slots), _ptr(ci), int(nthreads)))


# ---- Recurrent-state snapshot pages (Sec. 2.2); definition in kvx_oracle.h ----

def state_validate(num_layers, page_bytes, page_stride, num_pages, pages, n, num_state_slots, slot_ids, for_pack):
    pg = None if pages is None else np.ascontiguousarray(pages, dtype=np.int64)
    si = None if slot_ids is None else np.ascontiguousarray(slot_ids, dtype=np.int64)
    return int(_load().oracle_state_validate(int(num_layers), int(page_bytes), int(page_stride), int(num_pages),
                                             _ptr(pg), int(n), int(num_state_slots), _ptr(si),
                                             int(bool(for_pack))))


def _state_call(fn, layers, page_bytes, page_stride, pages, state_pool, slot_ids, writable_layers):
    for k, a in enumerate(layers):
        _check_bytes(a, f"layers[{k}]", writable=writable_layers)
    _check_bytes(state_pool, "state_pool", writable=not writable_layers)
    G = len(layers)
    num_pages = min(a.nbytes for a in layers) // page_stride if G else 0
    # A last page needs only page_bytes, not a whole stride.
    if G and min(a.nbytes for a in layers) - num_pages * page_stride >= page_bytes:
        num_pages += 1
    num_state_slots = state_pool.nbytes // (G * page_bytes) if G and page_bytes > 0 else 0
    pg = np.ascontiguousarray(pages, dtype=np.int64)
    si = np.ascontiguousarray(slot_ids, dtype=np.int64)
    return int(fn(int(G), int(page_bytes), int(page_stride), int(num_pages), _layer_ptr_array(layers), _ptr(pg),
                  int(pg.size), _ptr(state_pool), int(num_state_slots), _ptr(si)))


def state_pack(layers, page_bytes, page_stride, pages, state_pool, slot_ids):
    """Store snapshots: pages[k] of every layer (list of G host byte arrays) -> state slot slot_ids[k]."""
    return _state_call(_load().oracle_state_pack, layers, page_bytes, page_stride, pages, state_pool, slot_ids,
                       False)


def state_unpack(layers, page_bytes, page_stride, pages, state_pool, slot_ids):
    """Load snapshots: state slot slot_ids[k] -> pages[k] of every layer."""
    return _state_call(_load().oracle_state_unpack, layers, page_bytes, page_stride, pages, state_pool, slot_ids,
                       True)

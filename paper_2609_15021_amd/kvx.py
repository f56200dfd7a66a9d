"""Python binding of the kvx C ABI (``include/kvx.h``): argument marshalling only.

Every step of store and load runs in the HIP library ``libkvx.so``; this module
only converts torch tensors, numpy arrays and streams into the plain pointers
and sizes the C ABI takes.  The names are the C ABI's.

The library must bind to the HIP runtime that torch loaded, so torch is
imported before the library is opened.  If ``libkvx.so`` is missing the import
fails loudly: there is no CPU or Python fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # noqa: F401  (must precede the library: it provides the process's HIP runtime)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvx.so")

KV_OK = 0
KV_EINVAL = -1
KV_ENOMEM = -2
KV_EHIP = -3
KV_EUNSUPPORTED = -4
KV_EASYNC = -5
KV_EBUSY = -6

KV_MODE_ZERO_COPY = 1
KV_MODE_STAGED = 2
KV_HOST_COHERENT = 0
KV_HOST_NONCOHERENT = 1
KV_POOL_DEVICE = 2
KV_ASYNC_BAD_BLOCK = 1
KV_BLOCK_HND = 0
KV_BLOCK_NHD = 1
KV_LOOKUP_REQUIRE_STATE = 1
KV_LOOKUP_PIN = 2

MODES = {"zero_copy": KV_MODE_ZERO_COPY, "staged": KV_MODE_STAGED}


class KvLayout(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("chunk_tokens", ctypes.c_int32)]


class KvCache(ctypes.Structure):
    _fields_ = [("layout", KvLayout), ("num_blocks", ctypes.c_int32), ("device", ctypes.c_int32),
                ("block_order", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("layer_ptrs", ctypes.POINTER(ctypes.c_void_p)), ("block_stride_bytes", ctypes.c_int64)]


class KvPoolOptions(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_uint32), ("host_kind", ctypes.c_uint32),
                ("staging_slots", ctypes.c_int32), ("chunks_per_batch", ctypes.c_int32),
                ("side_streams", ctypes.c_int32), ("profile", ctypes.c_int32),
                ("num_state_slots", ctypes.c_int64), ("state_slot_bytes", ctypes.c_int64)]


class KvPoolInfo(ctypes.Structure):
    _fields_ = [("num_slots", ctypes.c_int64), ("slot_bytes", ctypes.c_int64),
                ("pool_bytes", ctypes.c_int64), ("staging_bytes", ctypes.c_int64),
                ("alloc_seconds", ctypes.c_double), ("device", ctypes.c_int32),
                ("mode", ctypes.c_uint32), ("host_kind", ctypes.c_uint32),
                ("is_pinned", ctypes.c_int32), ("staging_slots", ctypes.c_int32),
                ("chunks_per_batch", ctypes.c_int32), ("side_streams", ctypes.c_int32),
                ("staging_contiguous", ctypes.c_int32), ("host_base", ctypes.c_void_p),
                ("device_base", ctypes.c_void_p), ("num_state_slots", ctypes.c_int64),
                ("state_slot_bytes", ctypes.c_int64), ("state_host_base", ctypes.c_void_p),
                ("load_mode", ctypes.c_uint32), ("pad", ctypes.c_uint32)]


class KvState(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("device", ctypes.c_int32), ("page_bytes", ctypes.c_int64),
                ("page_stride", ctypes.c_int64), ("num_pages", ctypes.c_int64),
                ("layer_ptrs", ctypes.POINTER(ctypes.c_void_p))]


class KvLookup(ctypes.Structure):
    _fields_ = [("kv_chunks", ctypes.c_int64), ("hit_chunks", ctypes.c_int64), ("hit_tokens", ctypes.c_int64),
                ("state_slot", ctypes.c_int64)]


class KvIndexStats(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int64) for name in ("entries", "pending", "free_slots", "state_entries",
                                                      "free_state_slots", "evictions", "state_evictions")]


class KvIpcBuffer(ctypes.Structure):
    _fields_ = [("handle", ctypes.c_uint8 * 64), ("offset", ctypes.c_int64), ("allocation_bytes", ctypes.c_int64)]


class KvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


def _open():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"kvx HIP library not built ({LIB_PATH} missing); run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    sig = {
        "kv_pool_create": ([ctypes.POINTER(KvLayout), i64, ctypes.POINTER(KvPoolOptions), ctypes.POINTER(P)], i32),
        "kv_pool_destroy": ([P], i32),
        "kv_pool_get_info": ([P, ctypes.POINTER(KvPoolInfo)], i32),
        "kv_pool_slot": ([P, i64], P),
        "kv_pool_slot_bytes": ([P], i64),
        "kv_pool_num_slots": ([P], i64),
        "kv_pool_set_mode": ([P, u32], i32),
        "kv_pool_set_modes": ([P, u32, u32], i32),
        "kv_pool_async_error": ([P, ctypes.c_int], i32),
        "kv_pool_kernel_stats": ([P, ctypes.c_int, ctypes.c_int, ctypes.POINTER(i64),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)], i32),
        "kv_check": ([ctypes.POINTER(KvCache), ctypes.POINTER(KvLayout), i64, i64, P, ctypes.c_int], i32),
        "kv_store": ([ctypes.POINTER(KvCache), P, i64, P, P, P], i32),
        "kv_load": ([ctypes.POINTER(KvCache), P, i64, P, P, P], i32),
        "kv_load_noalloc": ([ctypes.POINTER(KvCache), P, i64, P, P, P], i32),
        "kv_pool_state_slot": ([P, i64], P),
        "kv_check_state": ([ctypes.POINTER(KvState), i64, i64, i64, P, P, ctypes.c_int], i32),
        "kv_store_state": ([ctypes.POINTER(KvState), P, i64, P, P, P], i32),
        "kv_load_state": ([ctypes.POINTER(KvState), P, i64, P, P, P], i32),
        "kv_index_create": ([i32, i64, i64, ctypes.POINTER(P)], i32),
        "kv_index_destroy": ([P], i32),
        "kv_index_keys": ([P, ctypes.c_uint64, P, i64, P], i32),
        "kv_index_lookup": ([P, ctypes.c_uint64, P, i64, u32, P, ctypes.POINTER(KvLookup)], i32),
        "kv_index_unpin": ([P, P, i64], i32),
        "kv_index_reserve": ([P, ctypes.c_uint64, P, i64, P, P, ctypes.POINTER(i64)], i32),
        "kv_index_commit": ([P, P, P, i64, ctypes.c_int], i32),
        "kv_index_reserve_state": ([P, i64, ctypes.POINTER(i64), ctypes.POINTER(i32)], i32),
        "kv_index_commit_state": ([P, i64, ctypes.c_int], i32),
        "kv_index_get_stats": ([P, ctypes.POINTER(KvIndexStats)], i32),
        "kv_ipc_export": ([P, ctypes.POINTER(KvIpcBuffer)], i32),
        "kv_ipc_check": ([ctypes.POINTER(KvIpcBuffer), i64], i32),
        "kv_tier_serve": ([P, P, ctypes.c_int], i32),
        "kv_tier_listen": ([ctypes.c_char_p, ctypes.POINTER(ctypes.c_int)], i32),
        "kv_tier_run": ([P, P, ctypes.c_int, i32], i32),
        "kv_tier_store_prefix": ([ctypes.c_int, ctypes.POINTER(KvCache), P, ctypes.POINTER(KvState), i64,
                                  ctypes.c_uint64, P, i64, ctypes.POINTER(i64), ctypes.POINTER(i32), P], i32),
        "kv_tier_load_prefix": ([ctypes.c_int, ctypes.POINTER(KvCache), P, ctypes.POINTER(KvState), i64,
                                 ctypes.c_uint64, P, i64, ctypes.POINTER(i64), P], i32),
        "kv_tier_store": ([ctypes.c_int, ctypes.POINTER(KvCache), P, i64, P, P], i32),
        "kv_tier_load": ([ctypes.c_int, ctypes.POINTER(KvCache), P, i64, P, P], i32),
        "kv_last_error": ([], ctypes.c_char_p),
        "kv_status_name": ([i32], ctypes.c_char_p),
        "kv_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _open()

EXPORTS = ("kv_pool_create", "kv_pool_destroy", "kv_pool_get_info", "kv_pool_slot", "kv_pool_slot_bytes",
           "kv_pool_num_slots", "kv_pool_set_mode", "kv_pool_set_modes", "kv_pool_async_error",
           "kv_pool_kernel_stats", "kv_check",
           "kv_store", "kv_load", "kv_load_noalloc", "kv_last_error", "kv_status_name", "kv_version",
           "kv_pool_state_slot",
           "kv_check_state", "kv_store_state", "kv_load_state", "kv_index_create", "kv_index_destroy",
           "kv_index_keys", "kv_index_lookup", "kv_index_unpin", "kv_index_reserve", "kv_index_commit",
           "kv_index_reserve_state", "kv_index_commit_state", "kv_index_get_stats", "kv_ipc_export", "kv_ipc_check",
           "kv_tier_serve", "kv_tier_store", "kv_tier_load", "kv_tier_listen", "kv_tier_run",
           "kv_tier_store_prefix", "kv_tier_load_prefix")


def kv_last_error() -> str:
    return _lib.kv_last_error().decode()


def kv_status_name(status: int) -> str:
    return _lib.kv_status_name(int(status)).decode()


def kv_version() -> str:
    return _lib.kv_version().decode()


def _raise(status: int):
    if status != KV_OK:
        raise KvError(status, kv_last_error() or kv_status_name(status))


def make_layout(L, H, D, E, BS, C) -> KvLayout:
    return KvLayout(int(L), int(H), int(D), int(E), int(BS), int(C))


class Cache:
    """A replica's paged cache as the C ABI sees it (keeps the tensors and pointer array alive).

    ``layers``: one tensor [L][NB][2][H][BS][D] ([L][NB][2][BS][H][D] with block_order
    KV_BLOCK_NHD; any dtype of elem_bytes), or a list of L per-layer tensors [NB][...];
    ``block_stride_bytes`` 0 means packed blocks.
    """

    def __init__(self, layers, layout: KvLayout, num_blocks: int, block_stride_bytes: int = 0,
                 block_order: int = KV_BLOCK_HND):
        if isinstance(layers, torch.Tensor):
            tensors = [layers[l] for l in range(layers.shape[0])]
            self._keep = [layers]
        else:
            tensors = list(layers)
            self._keep = tensors
        if len(tensors) != layout.num_layers:
            raise ValueError(f"{len(tensors)} layer buffers for a {layout.num_layers}-layer layout")
        dev = tensors[0].device
        if dev.type != "cuda":
            raise ValueError("cache layers must be device tensors")
        block_bytes = 2 * layout.num_kv_heads * layout.block_size * layout.head_dim * layout.elem_bytes
        need = int(num_blocks) * int(block_stride_bytes or block_bytes)
        for k, t in enumerate(tensors):
            if t.device != dev or not t.is_contiguous() or t.numel() * t.element_size() < need:
                raise ValueError(f"layer {k}: need a contiguous device buffer of >= {need} bytes on {dev}")
        self._ptrs = (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
        self.struct = KvCache(layout, int(num_blocks), int(dev.index if dev.index is not None else 0),
                              int(block_order), 0, ctypes.cast(self._ptrs, ctypes.POINTER(ctypes.c_void_p)),
                              int(block_stride_bytes))
        self.layout = layout


class Pool:
    """Owning handle of a kv_pool (destroyed by ``kv_pool_destroy`` or garbage collection)."""

    def __init__(self, handle: ctypes.c_void_p, layout: KvLayout):
        self.handle = handle
        self.layout = layout

    def __del__(self):
        if getattr(self, "handle", None):
            try:
                _lib.kv_pool_destroy(self.handle)
            except Exception:
                pass
            self.handle = None


def _stream_handle(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, (torch.cuda.Stream, torch.cuda.ExternalStream)):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def kv_pool_create(layout: KvLayout, num_slots: int, mode="staged", host_kind=KV_HOST_COHERENT,
                   staging_slots=0, chunks_per_batch=0, side_streams=0, profile=False, num_state_slots=0,
                   state_slot_bytes=0) -> Pool:
    m = MODES[mode] if isinstance(mode, str) else int(mode)
    opts = KvPoolOptions(m, int(host_kind), int(staging_slots), int(chunks_per_batch), int(side_streams),
                         1 if profile else 0, int(num_state_slots), int(state_slot_bytes))
    out = ctypes.c_void_p()
    _raise(_lib.kv_pool_create(ctypes.byref(layout), int(num_slots), ctypes.byref(opts), ctypes.byref(out)))
    return Pool(out, layout)


def kv_pool_destroy(pool: Pool) -> None:
    h, pool.handle = pool.handle, None
    _raise(_lib.kv_pool_destroy(h))


def kv_pool_get_info(pool: Pool) -> dict:
    info = KvPoolInfo()
    _raise(_lib.kv_pool_get_info(pool.handle, ctypes.byref(info)))
    return {name: getattr(info, name) for name, _ in KvPoolInfo._fields_}


def kv_pool_slot(pool: Pool, slot: int) -> int:
    return _lib.kv_pool_slot(pool.handle, int(slot)) or 0


def kv_pool_slot_bytes(pool: Pool) -> int:
    return int(_lib.kv_pool_slot_bytes(pool.handle))


def kv_pool_num_slots(pool: Pool) -> int:
    return int(_lib.kv_pool_num_slots(pool.handle))


def kv_pool_set_mode(pool: Pool, mode) -> None:
    _raise(_lib.kv_pool_set_mode(pool.handle, MODES[mode] if isinstance(mode, str) else int(mode)))


def kv_pool_set_modes(pool: Pool, store_mode, load_mode) -> None:
    def code(m):
        return MODES[m] if isinstance(m, str) else int(m)
    _raise(_lib.kv_pool_set_modes(pool.handle, code(store_mode), code(load_mode)))


def kv_pool_async_error(pool: Pool, clear: bool = False) -> int:
    return int(_lib.kv_pool_async_error(pool.handle, 1 if clear else 0))


def kv_pool_kernel_stats(pool: Pool, which: str, reset: bool = False):
    """(launches, total_ms, algorithmic_bytes) of the pack, unpack, state_pack or state_unpack
    kernels since the last reset."""
    n, ms, b = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double()
    kinds = {"pack": 0, "unpack": 1, "state_pack": 2, "state_unpack": 3}
    _raise(_lib.kv_pool_kernel_stats(pool.handle, kinds[which], 1 if reset else 0,
                                     ctypes.byref(n), ctypes.byref(ms), ctypes.byref(b)))
    return int(n.value), float(ms.value), float(b.value)


def pool_view(pool: Pool) -> np.ndarray:
    """The whole pinned pool as a host uint8 numpy array (touch only when no call is in flight)."""
    info = kv_pool_get_info(pool)
    if not info["host_base"]:
        raise ValueError("a device pool (KV_POOL_DEVICE) has no host address")
    buf = (ctypes.c_uint8 * info["pool_bytes"]).from_address(info["host_base"])
    return np.ctypeslib.as_array(buf)


def state_view(pool: Pool) -> np.ndarray:
    """The pool's state area as a host uint8 numpy array (empty without one)."""
    info = kv_pool_get_info(pool)
    nbytes = info["num_state_slots"] * info["state_slot_bytes"]
    if not nbytes:
        return np.zeros(0, dtype=np.uint8)
    buf = (ctypes.c_uint8 * nbytes).from_address(info["state_host_base"])
    return np.ctypeslib.as_array(buf)


def kv_pool_state_slot(pool: Pool, slot: int) -> int:
    return _lib.kv_pool_state_slot(pool.handle, int(slot)) or 0


class State:
    """A replica's recurrent-state page buffers as the C ABI sees them.

    ``layers``: one tensor [G][num_pages][...] or a list of G per-layer tensors whose bytes
    hold num_pages pages ``page_stride_bytes`` apart (0 = page_bytes).
    """

    def __init__(self, layers, page_bytes: int, num_pages: int, page_stride_bytes: int = 0):
        if isinstance(layers, torch.Tensor):
            tensors = [layers[g] for g in range(layers.shape[0])]
            self._keep = [layers]
        else:
            tensors = list(layers)
            self._keep = tensors
        if not tensors:
            raise ValueError("at least one recurrent layer buffer is needed")
        dev = tensors[0].device
        if dev.type != "cuda":
            raise ValueError("state layers must be device tensors")
        stride = int(page_stride_bytes or page_bytes)
        need = (int(num_pages) - 1) * stride + int(page_bytes)
        for g, t in enumerate(tensors):
            if t.device != dev or not t.is_contiguous() or t.numel() * t.element_size() < need:
                raise ValueError(f"state layer {g}: need a contiguous device buffer of >= {need} bytes on {dev}")
        self._ptrs = (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])
        self.struct = KvState(len(tensors), int(dev.index if dev.index is not None else 0), int(page_bytes),
                              int(page_stride_bytes), int(num_pages),
                              ctypes.cast(self._ptrs, ctypes.POINTER(ctypes.c_void_p)))


def kv_check_state(state, pool_state_slot_bytes: int, pool_state_slots: int, n: int, pages, slot_ids,
                   for_store: bool) -> int:
    """``state``: a State or a KvState structure."""
    struct = state.struct if isinstance(state, State) else state
    pg, pp = _chunk_ids(pages) if pages is not None else (None, None)
    si, sp = _chunk_ids(slot_ids) if slot_ids is not None else (None, None)
    return int(_lib.kv_check_state(ctypes.byref(struct), int(pool_state_slot_bytes), int(pool_state_slots), int(n),
                                   pp, sp, 1 if for_store else 0))


def _state_args(pages, slot_ids):
    pg, pp = _chunk_ids(pages)
    si, sp = _chunk_ids(slot_ids)
    if pg.size != si.size:
        raise ValueError(f"{pg.size} pages but {si.size} slot ids")
    return pg, pp, si, sp


def kv_store_state(state: State, pages, pool: Pool, slot_ids, stream=None) -> None:
    pg, pp, si, sp = _state_args(pages, slot_ids)
    _raise(_lib.kv_store_state(ctypes.byref(state.struct), pp, int(pg.size), pool.handle, sp,
                               _stream_handle(stream)))


def kv_load_state(state: State, pages, pool: Pool, slot_ids, stream=None) -> None:
    pg, pp, si, sp = _state_args(pages, slot_ids)
    _raise(_lib.kv_load_state(ctypes.byref(state.struct), pp, int(pg.size), pool.handle, sp,
                              _stream_handle(stream)))


def _chunk_ids(chunk_ids):
    a = np.ascontiguousarray(np.asarray(chunk_ids, dtype=np.int64))
    return a, (ctypes.c_void_p(a.ctypes.data) if a.size else None)


def _block_table_ptr(block_table, cache: Cache):
    if block_table is None:
        return None
    if not isinstance(block_table, torch.Tensor) or block_table.dtype != torch.int32 or \
            block_table.device.type != "cuda" or not block_table.is_contiguous():
        raise TypeError("block_table must be a contiguous int32 device tensor")
    return ctypes.c_void_p(block_table.data_ptr())


def _check_lengths(layout: KvLayout, n_tokens: int, n_ids: int, table_len: int) -> None:
    """The C ABI reads ceil(n/C) chunk ids and ceil(n/BS) block-table entries; shorter arrays would
    be read past their end (on the host, or by the kernels on the device).  Refused here, before
    any library call."""
    n = int(n_tokens)
    if n <= 0:
        return
    nc = -(-n // int(layout.chunk_tokens)) if layout.chunk_tokens > 0 else 0
    nblk = -(-n // int(layout.block_size)) if layout.block_size > 0 else 0
    if n_ids < nc:
        raise ValueError(f"{n_ids} chunk ids for {n} tokens: {nc} chunks of {layout.chunk_tokens} tokens need {nc}")
    if table_len < nblk:
        raise ValueError(f"block table of {table_len} entries for {n} tokens: {nblk} blocks of "
                         f"{layout.block_size} tokens need {nblk}")


def _table_len(block_table) -> int:
    if block_table is None:
        return 0
    if isinstance(block_table, torch.Tensor):
        return int(block_table.numel())
    return int(np.asarray(block_table).size)


def _in_use_on(t: torch.Tensor, stream) -> None:
    """The C ABI reads the block table from `stream` until the call's work completes there.  For a
    stream torch owns (the current stream or a torch.cuda.Stream it created), tell torch's caching
    allocator, so that a temporary table's memory is not handed out again (and overwritten from
    another stream) before that.  The allocator records an event on that stream when it frees the
    table, so a caller's own stream (a raw handle or an ExternalStream), which the caller may
    destroy first, is left out: there the caller keeps the table alive, as the C ABI requires."""
    if stream is None:
        s = torch.cuda.current_stream()
    elif isinstance(stream, torch.cuda.Stream) and not isinstance(stream, torch.cuda.ExternalStream):
        s = stream
    else:
        return
    t.record_stream(s)


def kv_check(cache: Cache, pool_layout: KvLayout, pool_slots: int, n_tokens: int, chunk_ids, for_store: bool) -> int:
    ids, ptr = _chunk_ids(chunk_ids) if chunk_ids is not None else (None, None)
    return int(_lib.kv_check(ctypes.byref(cache.struct), ctypes.byref(pool_layout), int(pool_slots), int(n_tokens),
                             ptr, 1 if for_store else 0))


def kv_store(cache: Cache, block_table, n_tokens: int, pool: Pool, chunk_ids, stream=None) -> None:
    ids, ptr = _chunk_ids(chunk_ids)
    _check_lengths(cache.layout, n_tokens, ids.size, _table_len(block_table))
    _raise(_lib.kv_store(ctypes.byref(cache.struct), _block_table_ptr(block_table, cache), int(n_tokens),
                         pool.handle, ptr, _stream_handle(stream)))
    if block_table is not None and int(n_tokens) > 0:
        _in_use_on(block_table, stream)


def kv_load(cache: Cache, block_table, n_tokens: int, pool: Pool, chunk_ids, stream=None) -> None:
    ids, ptr = _chunk_ids(chunk_ids)
    _check_lengths(cache.layout, n_tokens, ids.size, _table_len(block_table))
    _raise(_lib.kv_load(ctypes.byref(cache.struct), _block_table_ptr(block_table, cache), int(n_tokens),
                        pool.handle, ptr, _stream_handle(stream)))
    if block_table is not None and int(n_tokens) > 0:
        _in_use_on(block_table, stream)


def kv_load_noalloc(cache: Cache, block_table, n_tokens: int, pool: Pool, chunk_ids, stream=None) -> None:
    """kv_load through the library's static device scratch: allocates nothing (see kvx.h)."""
    ids, ptr = _chunk_ids(chunk_ids)
    _check_lengths(cache.layout, n_tokens, ids.size, _table_len(block_table))
    _raise(_lib.kv_load_noalloc(ctypes.byref(cache.struct), _block_table_ptr(block_table, cache), int(n_tokens),
                                pool.handle, ptr, _stream_handle(stream)))
    if block_table is not None and int(n_tokens) > 0:
        _in_use_on(block_table, stream)


# ---- Pool index (host only) --------------------------------------------------------------

class Index:
    """Owning handle of a kv_index."""

    def __init__(self, handle: ctypes.c_void_p, chunk_tokens: int):
        self.handle = handle
        self.chunk_tokens = chunk_tokens

    def __del__(self):
        if getattr(self, "handle", None):
            try:
                _lib.kv_index_destroy(self.handle)
            except Exception:
                pass
            self.handle = None


def _tokens(tokens):
    t = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    return t, (ctypes.c_void_p(t.ctypes.data) if t.size else None)


def _i64_array(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int64))
    return a, (ctypes.c_void_p(a.ctypes.data) if a.size else None)


def kv_index_create(chunk_tokens: int, num_slots: int, num_state_slots: int = 0) -> Index:
    out = ctypes.c_void_p()
    _raise(_lib.kv_index_create(int(chunk_tokens), int(num_slots), int(num_state_slots), ctypes.byref(out)))
    return Index(out, int(chunk_tokens))


def kv_index_destroy(index: Index) -> None:
    h, index.handle = index.handle, None
    _raise(_lib.kv_index_destroy(h))


def kv_index_keys(index: Index, salt: int, tokens) -> np.ndarray:
    t, tp = _tokens(tokens)
    keys = np.zeros((t.size // index.chunk_tokens, 2), dtype=np.uint64)
    _raise(_lib.kv_index_keys(index.handle, int(salt) & 0xFFFFFFFFFFFFFFFF, tp, int(t.size),
                              ctypes.c_void_p(keys.ctypes.data) if keys.size else None))
    return keys


def kv_index_lookup(index: Index, salt: int, tokens, require_state=False, pin=False) -> dict:
    t, tp = _tokens(tokens)
    slots = np.zeros(t.size // index.chunk_tokens, dtype=np.int64)
    out = KvLookup()
    flags = (KV_LOOKUP_REQUIRE_STATE if require_state else 0) | (KV_LOOKUP_PIN if pin else 0)
    _raise(_lib.kv_index_lookup(index.handle, int(salt) & 0xFFFFFFFFFFFFFFFF, tp, int(t.size), flags,
                                ctypes.c_void_p(slots.ctypes.data) if slots.size else None, ctypes.byref(out)))
    r = {name: int(getattr(out, name)) for name, _ in KvLookup._fields_}
    r["slots"] = slots[:r["hit_chunks"]].copy()
    return r


def kv_index_unpin(index: Index, slots) -> None:
    a, p = _i64_array(slots)
    _raise(_lib.kv_index_unpin(index.handle, p, int(a.size)))


def kv_index_reserve(index: Index, salt: int, tokens):
    """(slots int64[nc], is_new uint8[nc]) for the whole chunks of the prompt; KvError(KV_EBUSY) if full."""
    t, tp = _tokens(tokens)
    nc = t.size // index.chunk_tokens
    slots = np.zeros(nc, dtype=np.int64)
    is_new = np.zeros(nc, dtype=np.uint8)
    n = ctypes.c_int64()
    _raise(_lib.kv_index_reserve(index.handle, int(salt) & 0xFFFFFFFFFFFFFFFF, tp, int(t.size),
                                 ctypes.c_void_p(slots.ctypes.data) if nc else None,
                                 ctypes.c_void_p(is_new.ctypes.data) if nc else None, ctypes.byref(n)))
    return slots, is_new


def kv_index_commit(index: Index, slots, is_new, ok: bool = True) -> None:
    a, p = _i64_array(slots)
    b = np.ascontiguousarray(np.asarray(is_new, dtype=np.uint8))
    if a.size != b.size:
        raise ValueError("slots and is_new differ in length")
    _raise(_lib.kv_index_commit(index.handle, p, ctypes.c_void_p(b.ctypes.data) if b.size else None, int(a.size),
                                1 if ok else 0))


def kv_index_reserve_state(index: Index, slot: int):
    """(state_slot, is_new) of the snapshot after the chunk in ``slot``."""
    ss, new = ctypes.c_int64(), ctypes.c_int32()
    _raise(_lib.kv_index_reserve_state(index.handle, int(slot), ctypes.byref(ss), ctypes.byref(new)))
    return int(ss.value), int(new.value)


def kv_index_commit_state(index: Index, slot: int, ok: bool = True) -> None:
    _raise(_lib.kv_index_commit_state(index.handle, int(slot), 1 if ok else 0))


def kv_index_get_stats(index: Index) -> dict:
    st = KvIndexStats()
    _raise(_lib.kv_index_get_stats(index.handle, ctypes.byref(st)))
    return {name: int(getattr(st, name)) for name, _ in KvIndexStats._fields_}


# ---- Tier: a pool shared by replicas in other processes ----------------------------------

KV_IPC_MAX_ALLOCATION_BYTES = 2 << 30


def kv_ipc_export(ptr) -> KvIpcBuffer:
    """IPC buffer of a device pointer (int or tensor) of this process."""
    out = KvIpcBuffer()
    p = ptr.data_ptr() if isinstance(ptr, torch.Tensor) else int(ptr)
    _raise(_lib.kv_ipc_export(ctypes.c_void_p(p), ctypes.byref(out)))
    return out


def kv_ipc_check(buf: KvIpcBuffer, need: int) -> int:
    """Host-only check of a received IPC buffer (status code; no HIP call)."""
    return int(_lib.kv_ipc_check(ctypes.byref(buf), int(need)))


def kv_tier_serve(pool: Pool, fd: int, index: Index = None) -> None:
    """Serve one replica connection on the connected stream socket ``fd`` until it closes (blocks;
    the GIL is released while it runs); ``index`` enables prefix requests."""
    _raise(_lib.kv_tier_serve(pool.handle, index.handle if index is not None else None, int(fd)))


def kv_tier_listen(path: str) -> int:
    """A listening stream socket at ``path`` (which must not exist); returns its fd."""
    fd = ctypes.c_int(-1)
    _raise(_lib.kv_tier_listen(os.fsencode(path), ctypes.byref(fd)))
    return fd.value


def kv_tier_run(pool: Pool, listen_fd: int, connections: int, index: Index = None) -> None:
    """Accept and serve ``connections`` replica connections (0 = until the socket fails), each on
    its own native thread; returns when all have ended."""
    _raise(_lib.kv_tier_run(pool.handle, index.handle if index is not None else None, int(listen_fd),
                            int(connections)))


def _host_table(block_table):
    t = np.ascontiguousarray(np.asarray(block_table, dtype=np.int32))
    return t, (ctypes.c_void_p(t.ctypes.data) if t.size else None)


def kv_tier_store(fd: int, cache: Cache, block_table, n_tokens: int, chunk_ids, stream=None) -> None:
    """Store through the tier on ``fd``: ``block_table`` is a HOST int32 array; ``stream`` is
    synchronised first; returns once the tier has committed the chunks."""
    t, tp = _host_table(block_table)
    ids, ip = _chunk_ids(chunk_ids)
    _check_lengths(cache.layout, n_tokens, ids.size, t.size)
    _raise(_lib.kv_tier_store(int(fd), ctypes.byref(cache.struct), tp, int(n_tokens), ip, _stream_handle(stream)))


def kv_tier_load(fd: int, cache: Cache, block_table, n_tokens: int, chunk_ids, stream=None) -> None:
    """Load through the tier on ``fd`` into ``cache``; returns once the cache is complete."""
    t, tp = _host_table(block_table)
    ids, ip = _chunk_ids(chunk_ids)
    _check_lengths(cache.layout, n_tokens, ids.size, t.size)
    _raise(_lib.kv_tier_load(int(fd), ctypes.byref(cache.struct), tp, int(n_tokens), ip, _stream_handle(stream)))


def kv_tier_store_prefix(fd: int, cache: Cache, block_table, salt: int, tokens, stream=None, state: State = None,
                         state_page: int = 0):
    """Store the prompt's whole chunks that the tier does not hold yet (and, with ``state``, the
    snapshot in page ``state_page`` at the prompt's last whole-chunk boundary); returns
    (chunks stored, snapshots stored)."""
    t, tp = _host_table(block_table)
    tok, kp = _tokens(tokens)
    _check_lengths(cache.layout, tok.size, tok.size, t.size)  # the table covers the whole prompt
    out, out_state = ctypes.c_int64(), ctypes.c_int32()
    _raise(_lib.kv_tier_store_prefix(int(fd), ctypes.byref(cache.struct), tp,
                                     ctypes.byref(state.struct) if state is not None else None, int(state_page),
                                     int(salt) & 0xFFFFFFFFFFFFFFFF, kp, int(tok.size), ctypes.byref(out),
                                     ctypes.byref(out_state), _stream_handle(stream)))
    return int(out.value), int(out_state.value)


def kv_tier_load_prefix(fd: int, cache: Cache, block_table, salt: int, tokens, stream=None, state: State = None,
                        state_page: int = 0) -> int:
    """Load the prompt's longest whole-chunk hit into the cache (with ``state``: the longest hit
    under aligned recovery, and its boundary snapshot into page ``state_page``); returns the hit
    tokens."""
    t, tp = _host_table(block_table)
    tok, kp = _tokens(tokens)
    _check_lengths(cache.layout, tok.size, tok.size, t.size)  # the table covers the whole prompt
    out = ctypes.c_int64()
    _raise(_lib.kv_tier_load_prefix(int(fd), ctypes.byref(cache.struct), tp,
                                    ctypes.byref(state.struct) if state is not None else None, int(state_page),
                                    int(salt) & 0xFFFFFFFFFFFFFFFF, kp, int(tok.size), ctypes.byref(out),
                                    _stream_handle(stream)))
    return int(out.value)

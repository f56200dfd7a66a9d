"""ctypes binding of the harness HIP library (``libkvx_harness.so``): seeded device fills,
wall-clock producer delays, byte probes and the paper's copy-ordering variants.

Test and benchmark infrastructure only; not part of kvx.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (the HIP runtime must be torch's)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvx_harness.so")
DIST_CODE = {"u11": 0, "n01": 1, "raw": 2}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"harness library not built ({LIB_PATH} missing); run __graft_entry__.build()")
_lib = ctypes.CDLL(LIB_PATH)
_P, _i64, _u64, _i = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int
for _name, _args in {
    "kvh_fill_values": [_P, _u64, _i64, _i, _u64, _i, _P],
    "kvh_spin": [_P, ctypes.c_double],
    "kvh_wall_clock_khz": [],
    "kvh_fill_u8": [_P, _i64, _i, _P],
    "kvh_copy_u8": [_P, _P, _i64, _P],
    "kvh_copy_raw": [_P, _P, _i64],
    "kvh_copy_sync_then_raw": [_P, _P, _i64, _P],
    "kvh_copy_async": [_P, _P, _i64, _P],
    "kvh_stream_create": [_i, ctypes.POINTER(_P)],
    "kvh_stream_destroy": [_P],
    "kvh_stream_sync": [_P],
    "kvh_host_alloc": [_i64, ctypes.POINTER(_P)],
    "kvh_host_free": [_P],
    "kvh_host_device_ptr": [_P, ctypes.POINTER(_P)],
}.items():
    getattr(_lib, _name).argtypes = _args
    getattr(_lib, _name).restype = ctypes.c_int
_lib.kvh_last_error.restype = ctypes.c_char_p


def _ok(rc):
    if rc < 0:
        raise RuntimeError(_lib.kvh_last_error().decode())
    return rc


def _s(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, (torch.cuda.Stream, torch.cuda.ExternalStream)):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _p(x):
    if isinstance(x, torch.Tensor):
        return ctypes.c_void_p(x.data_ptr())
    return ctypes.c_void_p(int(x))


def fill_values(t: torch.Tensor, counter0: int, seed: int, dist: str, elem_bytes: int, stream=None):
    """Fill device tensor t (contiguous) with generator values for counters counter0 .. ."""
    n_elems = t.numel() * t.element_size() // elem_bytes
    _ok(_lib.kvh_fill_values(_p(t), counter0, n_elems, elem_bytes, seed & 0xFFFFFFFFFFFFFFFF, DIST_CODE[dist],
                             _s(stream)))


def spin(ms: float, stream=None):
    _ok(_lib.kvh_spin(_s(stream), float(ms)))


def wall_clock_khz() -> int:
    return _ok(_lib.kvh_wall_clock_khz())


def fill_u8(dst, n, value, stream=None):
    _ok(_lib.kvh_fill_u8(_p(dst), int(n), int(value), _s(stream)))


def copy_u8(dst, src, n, stream=None):
    _ok(_lib.kvh_copy_u8(_p(dst), _p(src), int(n), _s(stream)))


def copy_raw(dst, src, n):
    _ok(_lib.kvh_copy_raw(_p(dst), _p(src), int(n)))


def copy_sync_then_raw(dst, src, n, stream):
    _ok(_lib.kvh_copy_sync_then_raw(_p(dst), _p(src), int(n), _s(stream)))


def copy_async(dst, src, n, stream):
    _ok(_lib.kvh_copy_async(_p(dst), _p(src), int(n), _s(stream)))


class RawStream:
    """A HIP stream with explicit flags (default priority), usable where a stream handle is taken."""

    def __init__(self, non_blocking: bool):
        h = ctypes.c_void_p()
        _ok(_lib.kvh_stream_create(1 if non_blocking else 0, ctypes.byref(h)))
        self.handle = h.value

    def __int__(self):
        return int(self.handle)

    def synchronize(self):
        _ok(_lib.kvh_stream_sync(ctypes.c_void_p(self.handle)))

    def close(self):
        if self.handle:
            _ok(_lib.kvh_stream_destroy(ctypes.c_void_p(self.handle)))
            self.handle = None


class PinnedBuffer:
    """Pinned, mapped host bytes (hipHostMalloc), viewable as a numpy array."""

    def __init__(self, nbytes: int):
        import numpy as np
        h = ctypes.c_void_p()
        _ok(_lib.kvh_host_alloc(int(nbytes), ctypes.byref(h)))
        self.ptr = h.value
        self.nbytes = int(nbytes)
        self.array = np.ctypeslib.as_array((ctypes.c_uint8 * self.nbytes).from_address(self.ptr))
        d = ctypes.c_void_p()
        _ok(_lib.kvh_host_device_ptr(ctypes.c_void_p(self.ptr), ctypes.byref(d)))
        self.device_ptr = d.value

    def __int__(self):
        return int(self.ptr)

    def free(self):
        if self.ptr:
            self.array = None
            _ok(_lib.kvh_host_free(ctypes.c_void_p(self.ptr)))
            self.ptr = None

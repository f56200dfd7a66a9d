"""The paper's copy-ordering control matrix on HIP (Sec. 3.2; Table 2, "Copy-ordering controls").

Pinned host and device buffers stay fixed while only the ordering mechanism
varies.  Device-to-host: a delayed producer writes byte 37 on a non-blocking
stream, then the copy runs; the host must read 37 (the fault delivers the old
0).  Host-to-device: a delayed consumer reads the old device value 0, then the
copy overwrites the buffer with 53; the consumer must see 0 (the fault shows
53).  Variants: the raw synchronous copy that names no stream (the faulty
branch), waiting for the stream before that copy, an asynchronous copy on the
stream, and a same-stream kernel copy.  This exercises HIP itself, not kvx.
"""
from __future__ import annotations

import json
import sys

import numpy as np
import torch

import harness
from harness import gpu as hg

VARIANTS = ("raw", "sync_then_raw", "async_on_stream", "same_stream_kernel")
SIZES = (4096, 1 << 20, 16 << 20)
OLD, D2H_NEW, H2D_NEW = 0, 37, 53


def _copy(variant, dst, src, n, stream):
    if variant == "raw":
        hg.copy_raw(dst, src, n)
    elif variant == "sync_then_raw":
        hg.copy_sync_then_raw(dst, src, n, stream)
    elif variant == "async_on_stream":
        hg.copy_async(dst, src, n, stream)
    else:
        hg.copy_u8(dst, src, n, stream)


def run_matrix(trials: int = 10, seed: int = 0):
    """Returns {(variant, direction, delayed): [mismatching bytes of each trial]}."""
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()  # non-blocking, default priority
    delays = harness.spin_delays_ms(harness.sub_seed("controls", seed), 10 ** 4)
    k = 0
    out = {}
    big = max(SIZES)
    host = hg.PinnedBuffer(big)
    d_buf = torch.zeros(big, dtype=torch.uint8, device=dev)
    d_probe = torch.zeros(big, dtype=torch.uint8, device=dev)
    try:
        for variant in VARIANTS:
            for direction in ("d2h", "h2d"):
                for delayed in (False, True):
                    res = []
                    for size in SIZES:
                        for _ in range(trials):
                            d_buf.zero_()
                            d_probe.fill_(0xEE)
                            torch.cuda.synchronize()
                            ms = float(delays[k]) if delayed else 0.0
                            k += 1
                            if direction == "d2h":
                                host.array[:size] = OLD
                                if ms:
                                    hg.spin(ms, stream)
                                hg.fill_u8(d_buf, size, D2H_NEW, stream)
                                dst = host.device_ptr if variant == "same_stream_kernel" else host.ptr
                                _copy(variant, dst, d_buf.data_ptr(), size, stream)
                                stream.synchronize()
                                res.append(int(np.count_nonzero(host.array[:size] != D2H_NEW)))
                            else:
                                host.array[:size] = H2D_NEW
                                if ms:
                                    hg.spin(ms, stream)
                                hg.copy_u8(d_probe, d_buf, size, stream)  # delayed consumer of the old value
                                src = host.device_ptr if variant == "same_stream_kernel" else host.ptr
                                _copy(variant, d_buf.data_ptr(), src, size, stream)
                                stream.synchronize()
                                seen = d_probe[:size].cpu().numpy()
                                res.append(int(np.count_nonzero(seen != OLD)))
                    out[(variant, direction, delayed)] = res
    finally:
        torch.cuda.synchronize()
        host.free()
    return out


def summarise(results):
    """Pass/fail counts per (variant, delayed), pooled over directions, sizes and trials."""
    s = {}
    for (variant, direction, delayed), res in results.items():
        key = f"{variant}:{'delayed' if delayed else 'undelayed'}"
        p, f = s.get(key, (0, 0))
        s[key] = (p + sum(1 for r in res if r == 0), f + sum(1 for r in res if r != 0))
    return s


if __name__ == "__main__":
    r = run_matrix(trials=int(sys.argv[1]) if len(sys.argv) > 1 else 10,
                   seed=int(sys.argv[2]) if len(sys.argv) > 2 else 0)
    full = {f"{v}:{d}:{int(dl)}": x for (v, d, dl), x in r.items()}
    print("RESULT " + json.dumps(full), flush=True)

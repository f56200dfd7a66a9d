"""Aligned-recovery rule for hybrid state -- TEST INFRASTRUCTURE ONLY (oracle).

Sec. 2.2 of the paper: the KV cache of a hybrid model includes decoding state
recoverable at a common prefix boundary.  Full-attention layers contribute the K/V
pages that precede the boundary; the recurrent (Gated DeltaNet) layers contribute a
snapshot of their convolution and recurrent state at that boundary.  Under aligned
recovery a prefix can be restored only if both are present; a hit on the attention
pages alone does not establish recovery of the whole hybrid state.

Plain definition used here, over the chunks of one prefix in order (chunk i covers
tokens [i*C, (i+1)*C); its snapshot is the state at the boundary after it):
    restorable = the largest k such that chunks 0..k-1 all hold their K/V pages and,
    when recurrent state is required, the snapshot at the boundary after chunk k-1
    is present (k = 0 if none).
"""
from __future__ import annotations

KV = 1     # the chunk's K/V pages are stored
STATE = 2  # the snapshot at the boundary after the chunk is stored


def restorable_chunks(flags, require_state: bool) -> int:
    """flags[i]: bitmask of KV / STATE for chunk i of the prefix, in prefix order."""
    best = 0
    for k in range(1, len(flags) + 1):
        if not all(f & KV for f in flags[:k]):
            break
        if require_state and not (flags[k - 1] & STATE):
            continue
        best = k
    return best

"""An independent formulation of the packed-chunk gather with numpy fancy indexing.

Used only to pin the oracle.  It never computes a byte offset: it indexes a
stacked cache array A[L][NB][2][H][BS][D] by (block, slot) index arrays and lets
numpy's advanced indexing and transpose produce the token-major planes.
"""
import numpy as np


def token_view(A: np.ndarray, bt: np.ndarray, n: int, BS: int) -> np.ndarray:
    """[L][2][n][H][D]: the KV rows of tokens 0..n-1 as seen through the block table."""
    t = np.arange(n)
    blocks = np.asarray(bt, dtype=np.int64)[t // BS]
    slots = t % BS
    # Advanced indices separated by slices move to the front: result [n][L][2][H][D].
    g = A[:, blocks, :, :, slots, :]
    return np.ascontiguousarray(g.transpose(1, 2, 0, 3, 4))


def expected_chunks(A: np.ndarray, bt: np.ndarray, n: int, BS: int, C: int):
    """List of per-chunk arrays [L][2][r_i][H][D] for the prefix of n tokens."""
    tv = token_view(A, bt, n, BS)
    return [np.ascontiguousarray(tv[:, :, i:i + C]) for i in range(0, n, C)]


def scatter_tokens(B: np.ndarray, bt: np.ndarray, tv: np.ndarray, BS: int) -> None:
    """Write token view tv [L][2][n][H][D] into B through block table bt (in place)."""
    n = tv.shape[2]
    t = np.arange(n)
    blocks = np.asarray(bt, dtype=np.int64)[t // BS]
    slots = t % BS
    B[:, blocks, :, :, slots, :] = tv.transpose(2, 0, 1, 3, 4)


def token_view_nhd(A: np.ndarray, bt: np.ndarray, n: int, BS: int) -> np.ndarray:
    """[L][2][n][H][D] for a token-major ("NHD") cache A[L][NB][2][BS][H][D]."""
    t = np.arange(n)
    blocks = np.asarray(bt, dtype=np.int64)[t // BS]
    slots = t % BS
    # Index dims 1 and 3 with arrays (separated by a slice): result [n][L][2][H][D].
    g = A[:, blocks, :, slots, :, :]
    return np.ascontiguousarray(g.transpose(1, 2, 0, 3, 4))

"""Test-side statement of the cache layout documented in include/mlkv.h.

Written from the header's index formulas, independently of the binding's
packer, so that bit-exact cache comparisons do not trust product code."""
import numpy as np


def k_index(kv, b, t, d, B, S, D):
    return ((kv * B + b) * S + t) * D + d


def v_index(kv, b, t, d, B, S, D):
    return ((kv * B + b) * S + (t & ~31)) * D + d * 32 + (t & 31)


def unpack_v(v_plane_flat: np.ndarray, n_kv: int, B: int, S: int, D: int) -> np.ndarray:
    """Physical value plane (flat, any shape) -> logical [n_kv][B][S][D]: element
    (kv, b, t, d) sits in 32-token block t//32 at channel row d, column t%32."""
    blocks = np.ascontiguousarray(v_plane_flat).reshape(n_kv, B, S // 32, D, 32)
    return np.ascontiguousarray(blocks.transpose(0, 1, 2, 4, 3)).reshape(n_kv, B, S, D)


def unpack_k(k_plane_flat: np.ndarray, n_kv: int, B: int, S: int, D: int) -> np.ndarray:
    return np.ascontiguousarray(k_plane_flat).reshape(n_kv, B, S, D)


def pack_v(v_rows: np.ndarray) -> np.ndarray:
    """Logical value rows [..., S, D] -> the plane's blocked order [..., S/32, D, 32]."""
    *lead, S, D = v_rows.shape
    blk = v_rows.reshape(*lead, S // 32, 32, D)
    return np.ascontiguousarray(np.swapaxes(blk, -1, -2))

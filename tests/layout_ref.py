"""Test-side statement of the cache layout documented in include/mlkv.h.

Written from the header's index formulas, independently of the binding and
the kernels, so that bit-exact cache comparisons do not trust product code."""
import numpy as np


def k_chunk(u: int, c: int, D: int) -> int:
    """16-byte chunk (of the 4*D in a 32-token tile) holding channels 8c..8c+7
    of the tile's token u: ((((u >> 2) & 1) * D/32 + (c >> 2)) * 64
    + (c & 3) * 16 + ((u >> 3) << 2) + (u & 3)."""
    return ((((u >> 2) & 1) * (D // 32) + (c >> 2)) * 64 + (c & 3) * 16 + ((u >> 3) << 2)
            + (u & 3))


def k_index(kv, b, t, d, B, S, D):
    return ((kv * B + b) * S + (t & ~31)) * D + 8 * k_chunk(t & 31, d >> 3, D) + (d & 7)


def v_index(kv, b, t, d, B, S, D):
    return ((kv * B + b) * S + (t & ~31)) * D + d * 32 + (t & 31)


def _k_perm(D: int) -> np.ndarray:
    """perm[u * D/8 + c] = the plane chunk of row chunk (u, c) within a tile."""
    return np.array([k_chunk(u, c, D) for u in range(32) for c in range(D // 8)], dtype=np.int64)


def unpack_k(k_plane_flat: np.ndarray, n_kv: int, B: int, S: int, D: int) -> np.ndarray:
    """Physical key plane (flat, any shape) -> logical [n_kv][B][S][D]: the
    chunks of each 32-token tile are put back in token-row order."""
    tiles = np.ascontiguousarray(k_plane_flat).reshape(n_kv, B, S // 32, 4 * D, 8)
    rows = tiles[:, :, :, _k_perm(D), :]
    return np.ascontiguousarray(rows).reshape(n_kv, B, S, D)


def pack_k(k_rows: np.ndarray) -> np.ndarray:
    """Logical key rows [..., S, D] -> the plane's order (same shape)."""
    *lead, S, D = k_rows.shape
    rows = np.ascontiguousarray(k_rows).reshape(*lead, S // 32, 4 * D, 8)
    out = np.empty_like(rows)
    out[..., _k_perm(D), :] = rows
    return out.reshape(*lead, S, D)


def unpack_v(v_plane_flat: np.ndarray, n_kv: int, B: int, S: int, D: int) -> np.ndarray:
    """Physical value plane (flat, any shape) -> logical [n_kv][B][S][D]: element
    (kv, b, t, d) sits in 32-token block t//32 at channel row d, column t%32."""
    blocks = np.ascontiguousarray(v_plane_flat).reshape(n_kv, B, S // 32, D, 32)
    return np.ascontiguousarray(blocks.transpose(0, 1, 2, 4, 3)).reshape(n_kv, B, S, D)


def pack_v(v_rows: np.ndarray) -> np.ndarray:
    """Logical value rows [..., S, D] -> the plane's blocked order [..., S/32, D, 32]."""
    *lead, S, D = v_rows.shape
    blk = v_rows.reshape(*lead, S // 32, 32, D)
    return np.ascontiguousarray(np.swapaxes(blk, -1, -2))

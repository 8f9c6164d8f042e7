"""MLKV decode-attention ORACLE — test infrastructure only.

A plain fp64 CPU reference (``oracle.c``) of what the decode hot path computes,
with numpy wrappers.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product package never
does, and the two share no code (only the seeded input generator in
``synth/`` serves both).

Tensors are in logical order:
  q [B][h][D], caches [n_kv][B][S][D], new rows [B][n_kv][D]; bf16 as uint16 bits.

Paper references (arXiv 2406.09297): attention Section 2.1 Eqs. (1)-(3); GQA
grouping Section 2.3 Eq. (12); KV caching Section 2.4; cache sizes Section 2.5
and Section 3, Table 1; MLKV Section 3 Eqs. (13)-(17), bottom-layer ownership
Figure 2.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c (gcc -O2, OpenMP over (b, head) pairs only)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P, I, L = ctypes.c_void_p, ctypes.c_int, ctypes.c_long
        lib.oracle_map_uniform.argtypes = [I, I, I, I, P, P]
        lib.oracle_map_uniform.restype = I
        lib.oracle_attend_one.argtypes = [P, P, P, L, L, I, P, P]
        lib.oracle_attend_one.restype = None
        lib.oracle_decode_attention.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P]
        lib.oracle_decode_attention.restype = None
        lib.oracle_append.argtypes = [I, I, I, I, I, P, P, P, P, P, P]
        lib.oracle_append.restype = I
        lib.oracle_decode_step.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, P]
        lib.oracle_decode_step.restype = None
        D_ = ctypes.c_double
        lib.oracle_bf16_from_double.argtypes = [D_]
        lib.oracle_bf16_from_double.restype = ctypes.c_uint16
        lib.oracle_rope.argtypes = [P, I, I, D_, L, P]
        lib.oracle_rope.restype = None
        lib.oracle_rope_f64.argtypes = [P, I, I, D_, D_, P]
        lib.oracle_rope_f64.restype = None
        lib.oracle_decode_step_rope.argtypes = [I, I, I, I, I, I, I, D_, P, P, P, P, P, P, P, P,
                                                P, P, P, P]
        lib.oracle_decode_step_rope.restype = None
        lib.oracle_prefill_attention.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P]
        lib.oracle_prefill_attention.restype = None
        lib.oracle_append_rows.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P]
        lib.oracle_append_rows.restype = I
        lib.oracle_prefill_step.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P]
        lib.oracle_prefill_step.restype = None
        lib.oracle_threads.argtypes = [I]
        lib.oracle_threads.restype = I
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _bf16(a, shape=None):
    a = np.ascontiguousarray(a)
    assert a.dtype == np.uint16, "bf16 tensors are passed as uint16 bit patterns"
    if shape is not None:
        assert a.shape == tuple(shape), (a.shape, shape)
    return a


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


# ---------------------------------------------------------------- map ----------

def map_uniform(l: int, h: int, m: int, g: int):
    """kv_of [l][h] and owner_of [m*g] from Eqs. (12), (15), (17), 0-indexed.

    Raises ValueError when m does not divide l or g does not divide h."""
    kv_of = np.empty((l, h), dtype=np.int32)
    owner_of = np.empty(max(m * g, 1), dtype=np.int32)
    if _load().oracle_map_uniform(l, h, m, g, _p(kv_of), _p(owner_of)) != 0:
        raise ValueError(f"uniform MLKV map needs m | l and g | h (l={l} h={h} m={m} g={g})")
    return kv_of, owner_of


def cache_elements(method: str, b: int, s: int, l: int, h: int, d_k: int,
                   m: int | None = None, g: int | None = None) -> int:
    """KV-cache element counts: MHA 2bslhd_k, GQA 2bslgd_k, MQA 2bsld_k (Section 2.5),
    MLKV 2bsmgd_k (Section 3, Table 1)."""
    if method == "mha":
        return 2 * b * s * l * h * d_k
    if method == "gqa":
        return 2 * b * s * l * g * d_k
    if method == "mqa":
        return 2 * b * s * l * d_k
    if method == "mlkv":
        return 2 * b * s * m * g * d_k
    raise ValueError(method)


# ---------------------------------------------------------- attention ----------

def attend_one(q, K, V):
    """One head: returns (o [D] float64, alpha [L] float64) for q [D], K/V [L][D]."""
    q = _bf16(q)
    K = _bf16(K)
    V = _bf16(V)
    D = q.shape[0]
    L = K.shape[0]
    assert K.shape == (L, D) and V.shape == (L, D)
    o = np.empty(D, dtype=np.float64)
    alpha = np.empty(max(L, 1), dtype=np.float64)
    _load().oracle_attend_one(_p(q), _p(K), _p(V), L, D, D, _p(o), _p(alpha))
    return o, alpha[:L]


def decode_attention(layer: int, q, k_cache, v_cache, kv_of, seq_lens):
    """out [B][h][D] float64 of one layer over caches [n_kv][B][S][D]."""
    B, h, D = q.shape
    n_kv, B2, S, D2 = k_cache.shape
    assert B2 == B and D2 == D and v_cache.shape == k_cache.shape
    kv_of = _i32(kv_of)
    seq_lens = _i32(seq_lens)
    assert seq_lens.shape == (B,)
    out = np.empty((B, h, D), dtype=np.float64)
    _load().oracle_decode_attention(layer, B, h, n_kv, S, D, _p(kv_of), _p(_bf16(q)),
                                    _p(_bf16(k_cache)), _p(_bf16(v_cache)), _p(seq_lens),
                                    _p(out))
    return out


def append(layer: int, k_cache, v_cache, k_new, v_new, owner_of, positions) -> int:
    """In-place append of the newest token into the heads `layer` owns."""
    n_kv, B, S, D = k_cache.shape
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    assert k_cache.dtype == np.uint16 and v_cache.dtype == np.uint16
    k_new = _bf16(k_new, (B, n_kv, D))
    v_new = _bf16(v_new, (B, n_kv, D))
    return _load().oracle_append(layer, B, n_kv, S, D, _p(_i32(owner_of)), _p(k_cache),
                                 _p(v_cache), _p(k_new), _p(v_new), _p(_i32(positions)))


def decode_step(q_all, k_cache, v_cache, k_new, v_new, kv_of, owner_of, ctx):
    """Whole step (Eq. 17 order): per layer append then attend over ctx+1 positions.
    Updates the caches in place; returns out_all [l][B][h][D] float64."""
    l, B, h, D = q_all.shape
    n_kv, B2, S, D2 = k_cache.shape
    assert (B2, D2) == (B, D)
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    out = np.empty((l, B, h, D), dtype=np.float64)
    scratch = np.empty(B, dtype=np.int32)
    _load().oracle_decode_step(l, B, h, n_kv, S, D, _p(_i32(kv_of)), _p(_i32(owner_of)),
                               _p(_bf16(q_all)), _p(k_cache), _p(v_cache),
                               _p(_bf16(k_new, (B, n_kv, D))), _p(_bf16(v_new, (B, n_kv, D))),
                               _p(_i32(ctx)), _p(scratch), _p(out))
    return out


def prefill_attention(layer, q, k_cache, v_cache, kv_of, ctx):
    """One layer of causal prefill attention: q [B][T][h][D]; token t of
    sequence b attends positions 0 .. ctx[b] + t.  Returns [B][T][h][D] float64."""
    B, T, h, D = q.shape
    n_kv, B2, S, D2 = k_cache.shape
    assert (B2, D2) == (B, D)
    out = np.empty((B, T, h, D), dtype=np.float64)
    _load().oracle_prefill_attention(layer, B, T, h, n_kv, S, D, _p(_i32(kv_of)), _p(_bf16(q)),
                                     _p(_bf16(k_cache)), _p(_bf16(v_cache)), _p(_i32(ctx)),
                                     _p(out))
    return out


def append_rows(layer, k_cache, v_cache, k_new, v_new, owner_of, ctx) -> int:
    """Owners of `layer` store T new rows [B][T][n_kv][D] at slots ctx[b] + t
    (in place); returns the number of KV heads appended."""
    n_kv, B, S, D = k_cache.shape
    T = k_new.shape[1]
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    return _load().oracle_append_rows(layer, B, T, n_kv, S, D, _p(_i32(owner_of)), _p(k_cache),
                                      _p(v_cache), _p(_bf16(k_new, (B, T, n_kv, D))),
                                      _p(_bf16(v_new, (B, T, n_kv, D))), _p(_i32(ctx)))


def prefill_step(q_all, k_cache, v_cache, k_new, v_new, kv_of, owner_of, ctx):
    """Whole prefill (Eq. 17 order): per layer the owners append the T new
    rows, then every head attends causally.  q_all [l][B][T][h][D], k/v_new
    [B][T][n_kv][D].  Updates the caches in place; returns [l][B][T][h][D]."""
    l, B, T, h, D = q_all.shape
    n_kv, B2, S, D2 = k_cache.shape
    assert (B2, D2) == (B, D)
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    out = np.empty((l, B, T, h, D), dtype=np.float64)
    _load().oracle_prefill_step(l, B, T, h, n_kv, S, D, _p(_i32(kv_of)), _p(_i32(owner_of)),
                                _p(_bf16(q_all)), _p(k_cache), _p(v_cache),
                                _p(_bf16(k_new, (B, T, n_kv, D))),
                                _p(_bf16(v_new, (B, T, n_kv, D))), _p(_i32(ctx)), _p(out))
    return out


def bf16_from_double(x: float) -> int:
    """Nearest bf16 (ties to even) of a double, as its 16-bit pattern."""
    return int(_load().oracle_bf16_from_double(float(x)))


def rope(x, pos: int, rd: int, base: float = 10000.0) -> np.ndarray:
    """GPT-NeoX rotary embedding of one head vector (bf16 bits in and out):
    the first rd channels in rotate-half pairs (j, j + rd/2), angle
    pos * base^(-2j/rd); computed in double, rounded to bf16 (the models of
    Section 4.2 use the GPT-NeoX architecture)."""
    x = _bf16(x)
    D = x.shape[-1]
    assert x.ndim == 1 and rd % 2 == 0 and 0 <= rd <= D
    y = np.empty(D, dtype=np.uint16)
    _load().oracle_rope(_p(x), D, rd, float(base), int(pos), _p(y))
    return y


def rope_f64(x, pos: float, rd: int, base: float = 10000.0) -> np.ndarray:
    """The same rotation on a float64 vector, unrounded."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    _load().oracle_rope_f64(_p(x), x.shape[-1], rd, float(base), float(pos), _p(y))
    return y


def decode_step_rope(q_all, k_cache, v_cache, k_new, v_new, kv_of, owner_of, ctx, rd: int,
                     base: float = 10000.0, return_rotated: bool = False):
    """decode_step with the newest token's queries and keys rotated at
    position ctx[b] (rotary embedding, rd channels).  return_rotated: also
    return the rotated queries [l][B][h][D] and keys [B][n_kv][D] (bf16 bits)."""
    l, B, h, D = q_all.shape
    n_kv, B2, S, D2 = k_cache.shape
    assert (B2, D2) == (B, D) and rd % 2 == 0 and 0 <= rd <= D
    assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous
    out = np.empty((l, B, h, D), dtype=np.float64)
    q_rot = np.empty((l, B, h, D), dtype=np.uint16)
    k_rot = np.empty((B, n_kv, D), dtype=np.uint16)
    scratch = np.empty(B, dtype=np.int32)
    _load().oracle_decode_step_rope(l, B, h, n_kv, S, D, rd, float(base), _p(_i32(kv_of)),
                                    _p(_i32(owner_of)), _p(_bf16(q_all)), _p(k_cache),
                                    _p(v_cache), _p(_bf16(k_new, (B, n_kv, D))),
                                    _p(_bf16(v_new, (B, n_kv, D))), _p(_i32(ctx)), _p(q_rot),
                                    _p(k_rot), _p(scratch), _p(out))
    if return_rotated:
        return out, q_rot, k_rot
    return out


def to_f32_rne(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 rounding of oracle outputs (numpy rounds to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def threads(n: int = 0) -> int:
    """Host threads of the oracle's OpenMP loops: n > 0 sets them; returns
    the count in effect (timing only; results do not depend on it)."""
    return int(_load().oracle_threads(n))

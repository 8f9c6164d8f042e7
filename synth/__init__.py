"""Seeded synthetic inputs (shared by the oracle side and the GPU side).

Holds no attention arithmetic: only the counter-based generator in
``gen.c`` (SplitMix64 + Box-Muller, bf16 round-to-nearest-even) and the
workload shapes of the decode benchmarks.  Every tensor is produced in
*logical* order (``[n_kv][B][S][D]`` rows for the caches); turning rows into
the library's physical cache layout is the caller's business.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .workloads import (WORKLOADS, Workload, capacity_batch, get_workload,  # noqa: F401
                        step_bytes_per_sequence)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libsynth.so")

# Stream ids: one independent sequence per input tensor.
STREAM_Q = 0
STREAM_K_CACHE = 1
STREAM_V_CACHE = 2
STREAM_K_NEW = 3
STREAM_V_NEW = 4
STREAM_LENGTHS = 5

BF16_NAN = 0x7FC0  # quiet NaN, used to poison cache slots that must never be read

_lib = None


def build(force: bool = True) -> str:
    """Compile gen.c into libsynth.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        u64, i64 = ctypes.c_uint64, ctypes.c_int64
        lib.synth_uniform.argtypes = [u64, u64, u64, i64, ctypes.c_void_p]
        lib.synth_uniform_int.argtypes = [u64, u64, u64, i64, i64, i64, ctypes.c_void_p]
        lib.synth_normal_bf16.argtypes = [u64, u64, u64, i64, ctypes.c_double, ctypes.c_void_p]
        lib.synth_rows_bf16.argtypes = [u64, u64, i64, i64, i64, i64, ctypes.c_void_p,
                                        ctypes.c_double, ctypes.c_uint16, ctypes.c_void_p]
        for f in (lib.synth_uniform, lib.synth_uniform_int, lib.synth_normal_bf16,
                  lib.synth_rows_bf16):
            f.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def uniform(seed: int, stream: int, count: int, first: int = 0) -> np.ndarray:
    out = np.empty(count, dtype=np.float64)
    _load().synth_uniform(seed, stream, first, count, _ptr(out))
    return out


def uniform_int(seed: int, stream: int, count: int, lo: int, hi: int, first: int = 0) -> np.ndarray:
    out = np.empty(count, dtype=np.int32)
    _load().synth_uniform_int(seed, stream, first, count, lo, hi, _ptr(out))
    return out


def normal_bf16(seed: int, stream: int, shape, scale: float = 1.0, first: int = 0) -> np.ndarray:
    """bf16 bit patterns (uint16) of scale * N(0,1), element i = deviate first+i."""
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_normal_bf16(seed, stream, first, out.size, scale, _ptr(out))
    return out


def rows_bf16(seed: int, stream: int, n_rows: int, S: int, D: int, lens=None,
              scale: float = 1.0, fill: int = 0, row0: int = 0,
              out: np.ndarray | None = None) -> np.ndarray:
    """[n_rows][S][D] bf16 rows; token t of row r is a pure function of
    (row0 + r, t, d), and tokens t >= lens[r] hold `fill`."""
    if out is None:
        out = np.empty((n_rows, S, D), dtype=np.uint16)
    assert out.shape == (n_rows, S, D) and out.dtype == np.uint16 and out.flags.c_contiguous
    lp = None
    if lens is not None:
        lens = np.ascontiguousarray(lens, dtype=np.int32)
        assert lens.shape == (n_rows,)
        lp = _ptr(lens)
    _load().synth_rows_bf16(seed, stream, row0, n_rows, S, D, lp, scale, fill, _ptr(out))
    return out


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def context_lengths(w: Workload) -> np.ndarray:
    """ctx_b (tokens cached before the step) for every sequence b."""
    if w.ctx is not None:
        return np.full(w.B, w.ctx, dtype=np.int32)
    lo, hi = w.ctx_range
    return uniform_int(w.seed, STREAM_LENGTHS, w.B, lo, hi)


def step_inputs(w: Workload, fill: int = 0, with_cache: bool = True) -> dict:
    """Host inputs of one decode step in logical order.

    q        [l][B][h][D]   bf16 bits (uint16)
    k_new    [B][n_kv][D]   new token's keys (scaled by k_scale), v_new likewise
    k_cache  [n_kv][B][S][D] tokens [0, ctx_b) valid, the rest = fill
    v_cache  [n_kv][B][S][D]
    ctx      [B] int32
    """
    ctx = context_lengths(w)
    S = w.capacity
    out = {
        "ctx": ctx,
        "q": normal_bf16(w.seed, STREAM_Q, (w.l, w.B, w.h, w.D)),
        "k_new": normal_bf16(w.seed, STREAM_K_NEW, (w.B, w.n_kv, w.D), scale=w.k_scale),
        "v_new": normal_bf16(w.seed, STREAM_V_NEW, (w.B, w.n_kv, w.D)),
        "capacity": S,
    }
    if with_cache:
        lens = np.tile(ctx, w.n_kv)
        out["k_cache"] = rows_bf16(w.seed, STREAM_K_CACHE, w.n_kv * w.B, S, w.D, lens,
                                   scale=w.k_scale, fill=fill).reshape(w.n_kv, w.B, S, w.D)
        out["v_cache"] = rows_bf16(w.seed, STREAM_V_CACHE, w.n_kv * w.B, S, w.D, lens,
                                   fill=fill).reshape(w.n_kv, w.B, S, w.D)
    return out


def prefill_inputs(w: Workload, fill: int = 0, with_cache: bool = True) -> dict:
    """Host inputs of one prefill of w.T new tokens per sequence, logical order.

    q        [l][B][T][h][D]   bf16 bits (uint16)
    k_new    [B][T][n_kv][D]   the new tokens' keys (scaled by k_scale), v_new likewise
    k_cache  [n_kv][B][S][D]   tokens [0, ctx_b) valid, the rest = fill
    v_cache  [n_kv][B][S][D]
    ctx      [B] int32         tokens cached before the prefill
    """
    ctx = context_lengths(w)
    S = w.capacity
    out = {
        "ctx": ctx,
        "q": normal_bf16(w.seed, STREAM_Q, (w.l, w.B, w.T, w.h, w.D)),
        "k_new": normal_bf16(w.seed, STREAM_K_NEW, (w.B, w.T, w.n_kv, w.D), scale=w.k_scale),
        "v_new": normal_bf16(w.seed, STREAM_V_NEW, (w.B, w.T, w.n_kv, w.D)),
        "capacity": S,
    }
    if with_cache:
        lens = np.tile(ctx, w.n_kv)
        out["k_cache"] = rows_bf16(w.seed, STREAM_K_CACHE, w.n_kv * w.B, S, w.D, lens,
                                   scale=w.k_scale, fill=fill).reshape(w.n_kv, w.B, S, w.D)
        out["v_cache"] = rows_bf16(w.seed, STREAM_V_CACHE, w.n_kv * w.B, S, w.D, lens,
                                   fill=fill).reshape(w.n_kv, w.B, S, w.D)
    return out


STREAM_WEIGHTS = 16  # first stream of the model weights (one stream per tensor)


def model_weights(seed: int, l: int, h: int, D: int, d_ff: int, owned_per_layer,
                  std: float = 0.02) -> list:
    """Synthetic GPT-NeoX layer weights (bf16 bits, uint16), row-major [in][out]:
    layer-norm scales 1 + 0.1 N(0,1), every other tensor std * N(0,1); a layer
    with owned_per_layer[n] == 0 gets no key/value weights (None)."""
    d = h * D
    names = [("ln1_w", (d,)), ("ln1_b", (d,)), ("ln2_w", (d,)), ("ln2_b", (d,)),
             ("w_q", (d, h * D)), ("b_q", (h * D,)), ("w_k", None), ("b_k", None),
             ("w_v", None), ("b_v", None), ("w_o", (h * D, d)), ("b_o", (d,)),
             ("w_fc1", (d, d_ff)), ("b_fc1", (d_ff,)), ("w_fc2", (d_ff, d)), ("b_fc2", (d,))]
    layers = []
    for n in range(l):
        owned = int(owned_per_layer[n])
        lw = {}
        for t, (name, shape) in enumerate(names):
            if name in ("w_k", "w_v"):
                shape = (d, owned * D) if owned else None
            if name in ("b_k", "b_v"):
                shape = (owned * D,) if owned else None
            if shape is None:
                lw[name] = None
                continue
            stream = STREAM_WEIGHTS + n * len(names) + t
            if name in ("ln1_w", "ln2_w"):
                z = bf16_to_f32(normal_bf16(seed, stream, shape))
                lw[name] = f32_to_bf16(1.0 + 0.1 * z)
            else:
                lw[name] = normal_bf16(seed, stream, shape, scale=std)
        layers.append(lw)
    return layers

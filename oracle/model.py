"""ORACLE of the model-level decode step (test infrastructure only; only
tests/, the smoke check and the benchmark's CPU-baseline leg use it).

One decode step of a GPT-NeoX model (the architecture of the paper's Pythia
models, Section 4.2) whose attention uses an MLKV map (Section 3, Eqs.
13-17): plain numpy in float64, the layer written out in the order the
architecture defines it:

    h1 = LayerNorm1(x),  h2 = LayerNorm2(x)
    q  = h1 W_q + b_q                       (every query head)
    k, v = h1 W_k + b_k, h1 W_v + b_v       (only in a layer that owns KV heads)
    q, k rotated at position ctx_b (rotary embedding of the first rd channels)
    the owner's k, v stored at slot ctx_b; every head attends over ctx_b + 1
    positions of its (possibly shared) KV head          (Section 2.1 Eqs. 1-3)
    a  = o W_o + b_o
    m  = GELU(h2 W_1 + b_1) W_2 + b_2       (exact, erf form)
    x  = x + a + m                          (parallel residual)

With round_bf16=True the values that the GPU path stores in bf16 are rounded
to bf16 at the same points (the layer norms' outputs, the rotated q and k,
v, the attention output and the GELU output; nearest, ties to even), so that
the comparison measures arithmetic, not storage.  With round_bf16=False every
value stays in float64 (the form compared with an independent
implementation of the architecture in the tests).

Weights are passed per layer as a dict of bf16 bit arrays (uint16), matrices
row-major [in][out]:
    ln1_w, ln1_b, ln2_w, ln2_b    [d]
    w_q [d][h*D], b_q [h*D]
    w_k, w_v [d][owned*D], b_k, b_v [owned*D]   (None in a layer owning no KV head)
    w_o [h*D][d], b_o [d]
    w_fc1 [d][d_ff], b_fc1 [d_ff], w_fc2 [d_ff][d], b_fc2 [d]
"""
from __future__ import annotations

import math

import numpy as np

from . import rope_f64


def _f64(bits):
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (ties to even) of every element, as float64: the
    significand rounded to 8 bits (below 2^-126, to multiples of 2^-133)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    y = np.ldexp(np.rint(m * 256.0), e - 8)
    tiny = np.abs(x) < 2.0 ** -126
    y[tiny] = np.rint(x[tiny] * 2.0 ** 133) * 2.0 ** -133
    return y


def layer_norm(x: np.ndarray, w: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """(x - mean) / sqrt(var + eps) * w + b over the last axis (biased variance)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * w + b


def gelu(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2))."""
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """softmax(q . K_t / sqrt(D)) weighted sum of V_t (Section 2.1)."""
    s = K @ q / math.sqrt(q.shape[-1])
    w = np.exp(s - s.max())
    return (w / w.sum()) @ V


def decode_step_model(x, layers, kv_of, owner_of, k_cache, v_cache, ctx, h: int, D: int,
                      rd: int, base: float = 10000.0, eps: float = 1e-5,
                      round_bf16: bool = True, updates: list | None = None) -> np.ndarray:
    """One decode step through every layer.

    x        [B][d] float64, the newest token's residual stream
    k_cache, v_cache  [n_kv][B][S][D] float64 (updated: the owners' rows at
             slot ctx[b]); positions 0 .. ctx[b]-1 hold the cached tokens
    ctx      [B] tokens cached before the step
    Returns the residual stream after the last layer, [B][d] float64.
    updates: if a list, each layer appends its two residual updates (a, m),
    each [B][d] (for error estimates in the tests; nothing else changes).
    """
    rb = to_bf16 if round_bf16 else (lambda a: a)
    x = np.array(x, dtype=np.float64)
    B, d = x.shape
    kv_of = np.asarray(kv_of)
    owner_of = np.asarray(owner_of)
    for n, w in enumerate(layers):
        g = {k: (_f64(v) if v is not None else None) for k, v in w.items()}
        h1 = rb(layer_norm(x, g["ln1_w"], g["ln1_b"], eps))
        h2 = rb(layer_norm(x, g["ln2_w"], g["ln2_b"], eps))
        q = (h1 @ g["w_q"] + g["b_q"]).reshape(B, h, D)
        q = rb(np.stack([np.stack([rope_f64(q[b, i], int(ctx[b]), rd, base) for i in range(h)])
                         for b in range(B)]))
        owned = [kv for kv in range(len(owner_of)) if owner_of[kv] == n]
        if owned:
            k = (h1 @ g["w_k"] + g["b_k"]).reshape(B, len(owned), D)
            v = rb((h1 @ g["w_v"] + g["b_v"]).reshape(B, len(owned), D))
            k = rb(np.stack([np.stack([rope_f64(k[b, c], int(ctx[b]), rd, base)
                                       for c in range(len(owned))]) for b in range(B)]))
            for c, kv in enumerate(owned):
                for b in range(B):
                    k_cache[kv, b, ctx[b]] = k[b, c]
                    v_cache[kv, b, ctx[b]] = v[b, c]
        o = np.empty((B, h, D))
        for b in range(B):
            L = int(ctx[b]) + 1
            for i in range(h):
                kv = kv_of[n, i]
                o[b, i] = attend(q[b, i], k_cache[kv, b, :L], v_cache[kv, b, :L])
        o = rb(o)
        a = o.reshape(B, h * D) @ g["w_o"] + g["b_o"]
        f = rb(gelu(h2 @ g["w_fc1"] + g["b_fc1"]))
        m = f @ g["w_fc2"] + g["b_fc2"]
        if updates is not None:
            updates.append((a, m))
        x = x + a + m
    return x

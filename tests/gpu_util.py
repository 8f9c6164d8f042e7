"""Helpers shared by the GPU parity tests: seeded inputs uploaded to the device
through the binding, read-back in logical order (via tests/layout_ref.py), and
the tolerance checks.

Tolerances for fp32 outputs (bf16 inputs, fp32 accumulation): max |diff|
<= 1e-2 and mean |diff| <= 1e-3 against the fp64 oracle, everywhere.  Inside
that, each element is held to the bound its arithmetic allows where the test
can compute it (softmax_rounding_bound: the kernels round every softmax
weight to bf16 before the P.V product and sum the same rounded weights into
the denominator), else to max |diff| <= 2e-3 * max(1, max |ref|), a bar that
flags regressions long before the outer one.
"""
import sys

import numpy as np
import torch

import oracle
import synth
import paper_2406_09297_amd as mlkv
from layout_ref import unpack_k, unpack_v

MAX_ABS = 1e-2
MEAN_ABS = 1e-3
INTERNAL_REL = 2e-3


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def f64(bits: np.ndarray) -> np.ndarray:
    return synth.bf16_to_f32(bits).astype(np.float64)


def check_close(out: np.ndarray, ref: np.ndarray, tag: str, bound: np.ndarray = None):
    """Outer bars always; then every element within `bound` (same shape as
    ref) when given, else the internal bar relative to max |ref|."""
    out = np.asarray(out, dtype=np.float64)
    assert out.shape == ref.shape, (out.shape, ref.shape)
    assert np.all(np.isfinite(out)), f"{tag}: non-finite output"
    d = np.abs(out - ref)
    mx, mean = float(d.max(initial=0.0)), float(d.mean()) if d.size else 0.0
    scale = max(1.0, float(np.abs(ref).max(initial=0.0)))
    extra = ""
    if bound is not None:
        assert bound.shape == ref.shape, (bound.shape, ref.shape)
        ratio = float((d / np.maximum(bound, 1e-300)).max(initial=0.0))
        extra = f" max|d|/bound={ratio:.3f}"
    say(f"  {tag}: max|d|={mx:.3e} mean|d|={mean:.3e} max|ref|={np.abs(ref).max(initial=0):.3f}"
        + extra)
    assert mx <= MAX_ABS, f"{tag}: max abs error {mx}"
    assert mean <= MEAN_ABS, f"{tag}: mean abs error {mean}"
    if bound is not None:
        worst = np.unravel_index(int(np.argmax(d - bound)), d.shape)
        assert np.all(d <= bound), \
            f"{tag}: error {d[worst]} above its rounding bound {bound[worst]} at {worst}"
    else:
        assert mx <= INTERNAL_REL * scale, f"{tag}: max abs error {mx} above internal bar"
    return mx, mean


U = 2.0 ** -24  # unit roundoff of fp32


def softmax_rounding_bound(q: np.ndarray, K: np.ndarray, V: np.ndarray, ref: np.ndarray,
                           lens: np.ndarray) -> np.ndarray:
    """Bound on |device - ref| for rows of one head that share a key/value set.

    q [r][D], K/V [L][D] (float64 values of the bf16 inputs), ref [r][D] the
    oracle's outputs, lens [r] the number of leading positions each row
    attends (0: an empty row, whose output is exactly 0).

    With w_i the exact softmax weights and e_i the relative error of the
    weight the device uses, numerator and denominator built from the same
    weights give out - ref = sum_i w_i e_i (v_i - ref) / (1 + sum_i w_i e_i).
    e_i is the bf16 rounding of the weight (at most 2^-8 relative: 8
    significant bits, ties to even), plus the fp32 error of its exponent (a
    D-term dot product, the scale and the reference subtracted: at most about
    (D + 2) u |q||k_i| scale + 2 u (|y_i| + |y_max| + 8) in log2 units, times
    ln 2), plus the exponential's own error; the fp32 accumulations over L
    terms (products, denominator, split merges and the rescales) add at most
    about 2 (L + 32) u of sum_i w_i |v_i| + |ref|.  The reference a kernel
    divides by need not be the row's maximum (it is moved only when a score
    exceeds it by 2^8), so the dominant weight carries a rounding error too
    and no term is dropped.
    """
    r, D = q.shape
    L = K.shape[0]
    bound = np.zeros((r, D))
    live = lens > 0
    if L == 0 or not live.any():
        return bound
    scale_log2 = np.log2(np.e) / np.sqrt(D)
    y = (q @ K.T) * scale_log2
    cols = np.arange(L)[None, :]
    mask = cols < lens[:, None]
    y = np.where(mask, y, -np.inf)
    ymax = np.where(live, y.max(axis=1), 0.0)
    w = np.where(mask, np.exp2(y - ymax[:, None]), 0.0)
    w /= np.maximum(w.sum(axis=1, keepdims=True), 1e-300)
    dy = U * ((D + 2) * scale_log2 * (np.abs(q) @ np.abs(K).T)
              + 2 * (np.abs(np.where(mask, y, 0.0)) + np.abs(ymax)[:, None] + 8))
    eta = 2.0 ** -8 + np.log(2.0) * dy + 4 * U
    a = w * eta
    first = np.empty((r, D))
    for i0 in range(0, r, 32):  # sum_i a_ri |v_ic - ref_rc| in row chunks
        sl = slice(i0, min(r, i0 + 32))
        first[sl] = np.einsum("rl,rld->rd", a[sl], np.abs(V[None, :, :] - ref[sl, None, :]))
    first /= 1.0 - eta.max()
    accum = 2 * (L + 32) * U * (w @ np.abs(V) + np.abs(ref))
    bound = np.where(live[:, None], first + accum, 0.0)
    return bound


# Beyond a few thousand positions the worst-case fp32 accumulation term of
# softmax_rounding_bound outgrows the rounding term, and the bound is no
# tighter than the relative bar; longer rows keep that bar.
BOUND_MAX_POSITIONS = 4096


def layer_rounding_bound(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                         kv_row: np.ndarray, lens: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """softmax_rounding_bound for every output of one layer's decode
    attention: q [B][h][D] bf16 bits, caches [n_kv][B][S][D] bf16 bits, head i
    attends positions 0 .. lens[b] - 1 of KV head kv_row[i]; ref [B][h][D]."""
    B, h, D = q.shape
    bound = np.zeros_like(ref)
    for b in range(B):
        L = int(lens[b])
        if L <= 0:
            continue
        for kv in np.unique(kv_row):
            heads = np.nonzero(kv_row == kv)[0]
            K, V = f64(k_cache[kv, b, :L]), f64(v_cache[kv, b, :L])
            bound[b, heads] = softmax_rounding_bound(f64(q[b, heads]), K, V, ref[b, heads],
                                                     np.full(heads.size, L))
    return bound


def step_rounding_bound(q_all: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                        kv_of: np.ndarray, ctx: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """The same for a decode step: q_all [l][B][h][D], caches after the
    step's appends, ref [l][B][h][D]; every layer attends ctx[b] + 1
    positions."""
    lens = np.asarray(ctx, dtype=np.int64) + 1
    return np.stack([layer_rounding_bound(q_all[n], k_cache, v_cache, kv_of[n], lens, ref[n])
                     for n in range(q_all.shape[0])])


def prefill_rounding_bound(q_all: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                           kv_of: np.ndarray, ctx: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """The same for a prefill: q_all [l][B][T][h][D], ref [l][B][T][h][D];
    token t of sequence b attends positions 0 .. ctx[b] + t."""
    l, B, T, h, D = q_all.shape
    bound = np.zeros_like(ref)
    for b in range(B):
        L = int(ctx[b]) + T
        lens = np.arange(T) + int(ctx[b]) + 1
        for kv in np.unique(kv_of):
            K, V = f64(k_cache[kv, b, :L]), f64(v_cache[kv, b, :L])
            for n in range(l):
                heads = np.nonzero(kv_of[n] == kv)[0]
                if not heads.size:
                    continue
                q = f64(q_all[n, b][:, heads]).reshape(T * heads.size, D)
                rr = ref[n, b][:, heads].reshape(T * heads.size, D)
                bb = softmax_rounding_bound(q, K, V, rr, np.repeat(lens, heads.size))
                bound[n, b][:, heads] = bb.reshape(T, heads.size, D)
    return bound


class DeviceWorkload:
    """One workload's seeded inputs on host (logical) and device (binding layout)."""

    def __init__(self, w: synth.Workload, fill: int = synth.BF16_NAN, device="cuda"):
        self.w = w
        inp = synth.step_inputs(w, fill=fill)
        self.host = inp
        self.S = inp["capacity"]
        self.map = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
        self.kv_of, self.owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
        self.cache = mlkv.Cache.empty(w.n_kv, w.B, self.S, w.D, device)
        self.cache.load_rows(inp["k_cache"], inp["v_cache"])
        self.q = mlkv.bf16_tensor(inp["q"], device)
        self.k_new = mlkv.bf16_tensor(inp["k_new"], device)
        self.v_new = mlkv.bf16_tensor(inp["v_new"], device)
        self.ctx = torch.from_numpy(inp["ctx"]).to(device)
        self.ws = mlkv.workspace(self.map, w.B, self.S, w.D, device)

    def read_cache(self):
        """Device cache -> logical host arrays (K, V), [n_kv][B][S][D] uint16."""
        torch.cuda.synchronize()
        w = self.w
        k = unpack_k(mlkv.bf16_bits(self.cache.k), w.n_kv, w.B, self.S, w.D)
        v = unpack_v(mlkv.bf16_bits(self.cache.v), w.n_kv, w.B, self.S, w.D)
        return k, v

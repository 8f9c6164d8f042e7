"""The per-element tolerance of the GPU parity tests (gpu_util's
softmax_rounding_bound), checked on the CPU against an emulation of the
arithmetic it bounds: every softmax weight (Section 2.1 Eq. 3) taken
relative to a reference that may sit up to 2^8 below the row's maximum,
rounded to bf16 (ties to even), and used for both the P.V numerator and the
denominator.  The emulated outputs must lie inside the bound for every
element, and the bound must not be vacuous (some element comes close to it).
"""
import numpy as np
import pytest

pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from gpu_util import f64, softmax_rounding_bound  # noqa: E402


def _bf16_round(x: np.ndarray) -> np.ndarray:
    return f64(synth.f32_to_bf16(x.astype(np.float32)))


def _emulate(q, K, V, lens, offsets):
    """Rows of one head: weights 2^(y - ref) with ref = max - offset, rounded
    to bf16, numerator and denominator from the rounded weights (fp64 sums)."""
    D = q.shape[1]
    y = (q @ K.T) * (np.log2(np.e) / np.sqrt(D))
    out = np.zeros((q.shape[0], D))
    for r in range(q.shape[0]):
        L = lens[r]
        if L == 0:
            continue
        yr = y[r, :L]
        p = _bf16_round(np.exp2(yr - (yr.max() - offsets[r])))
        out[r] = (p @ V[:L]) / p.sum()
    return out


@pytest.mark.parametrize("D,L,k_scale,seed", [(64, 1, 1.0, 1), (64, 33, 1.0, 2), (128, 300, 1.0, 3),
                                              (64, 700, 4.0, 4), (128, 96, 8.0, 5)])
def test_emulated_bf16_weights_stay_inside_the_bound(D, L, k_scale, seed):
    rng = np.random.default_rng(seed)
    r = 48
    q = f64(synth.f32_to_bf16(rng.standard_normal((r, D)).astype(np.float32)))
    K = f64(synth.f32_to_bf16((k_scale * rng.standard_normal((L, D))).astype(np.float32)))
    V = f64(synth.f32_to_bf16(rng.standard_normal((L, D)).astype(np.float32)))
    lens = rng.integers(0, L + 1, r)
    lens[:3] = [0, 1, L]
    ref = np.zeros((r, D))
    for i in range(r):
        if lens[i]:
            ref[i] = oracle.attend_one(synth.f32_to_bf16(q[i].astype(np.float32)),
                                       synth.f32_to_bf16(K[:lens[i]].astype(np.float32)),
                                       synth.f32_to_bf16(V[:lens[i]].astype(np.float32)))[0]
    bound = softmax_rounding_bound(q, K, V, ref, lens)
    assert np.all(bound[lens == 0] == 0)
    worst = 0.0
    for offsets in (np.zeros(r), rng.uniform(0, 8, r), np.full(r, 8.0)):
        d = np.abs(_emulate(q, K, V, lens, offsets) - ref)
        assert np.all(d <= bound), float((d / np.maximum(bound, 1e-300)).max())
        live = lens > 1
        if live.any():
            worst = max(worst, float((d[live] / bound[live]).max()))
    if L > 1:
        assert worst > 0.3, worst  # the bound is within a small factor of what rounding does


def test_bound_catches_a_dropped_token():
    """An output that leaves out one attended position (the kind of mistake
    the parity tests are for) falls outside the bound."""
    rng = np.random.default_rng(9)
    D, L, r = 64, 40, 12
    q = f64(synth.f32_to_bf16(rng.standard_normal((r, D)).astype(np.float32)))
    K = f64(synth.f32_to_bf16(rng.standard_normal((L, D)).astype(np.float32)))
    V = f64(synth.f32_to_bf16(rng.standard_normal((L, D)).astype(np.float32)))
    lens = np.full(r, L)
    y = q @ K.T / np.sqrt(D)
    w = np.exp(y - y.max(axis=1, keepdims=True))
    ref = (w / w.sum(axis=1, keepdims=True)) @ V
    bound = softmax_rounding_bound(q, K, V, ref, lens)
    w2 = w[:, :-1]
    dropped = (w2 / w2.sum(axis=1, keepdims=True)) @ V[:-1]
    assert np.any(np.abs(dropped - ref) > bound)

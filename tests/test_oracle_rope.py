"""Pins of the oracle's rotary embedding (GPT-NeoX architecture of the
paper's Pythia models, Section 4.2): identities, invariants and a closed form
that a pairing, sign or frequency mistake breaks.  CPU only."""
import math

import numpy as np
import pytest

import oracle
import synth


def _bf16_neighbours(x: float):
    """All bf16 values within a few ulps of x, by enumerating bit patterns."""
    b = synth.f32_to_bf16(np.array([x], dtype=np.float32))[0]
    cands = np.arange(max(int(b) - 4, 0), min(int(b) + 5, 0x7F80), dtype=np.uint16)
    if x < 0:
        cands = np.arange(max(int(b) - 4, 0x8000), min(int(b) + 5, 0xFF80), dtype=np.uint16)
    return cands, synth.bf16_to_f32(cands).astype(np.float64)


def _nearest_even(x: float) -> int:
    cands, vals = _bf16_neighbours(x)
    d = np.abs(vals - x)
    best = np.flatnonzero(d == d.min())
    if best.size == 1:
        return int(cands[best[0]])
    even = [int(cands[i]) for i in best if int(cands[i]) % 2 == 0]
    return even[0]


def test_bf16_rounding_is_nearest_ties_to_even():
    rng = np.random.default_rng(3)
    xs = list(rng.normal(0, 3, 400)) + [1.0, -2.5, 1e-3, 123.456]
    # exact midpoints between neighbouring bf16 values (ties)
    for bits in rng.integers(0x3C00, 0x4400, 100):
        lo, hi = synth.bf16_to_f32(np.array([bits, bits + 1], dtype=np.uint16)).astype(np.float64)
        xs.append((lo + hi) / 2)
        xs.append(-(lo + hi) / 2)
    for x in xs:
        assert oracle.bf16_from_double(x) == _nearest_even(float(x)), x


def test_position_zero_and_zero_channels_are_identity():
    x = synth.normal_bf16(5, 0, (64,))
    assert np.array_equal(oracle.rope(x, 0, 16), x)
    assert np.array_equal(oracle.rope(x, 123, 0), x)
    y = oracle.rope(x, 777, 16)
    assert np.array_equal(y[16:], x[16:])  # channels past rd untouched


def test_closed_form_of_a_four_channel_rotation():
    """D = rd = 4, base 10000, position 1: pair (0, 2) turns by 1 rad and pair
    (1, 3) by 10000^(-1/2) = 0.01 rad (rotate-half pairing)."""
    x = np.array([0.3, -1.2, 0.8, 2.0])
    y = oracle.rope_f64(x, 1.0, 4, 10000.0)
    t0, t1 = 1.0, 0.01
    want = [x[0] * math.cos(t0) - x[2] * math.sin(t0), x[1] * math.cos(t1) - x[3] * math.sin(t1),
            x[2] * math.cos(t0) + x[0] * math.sin(t0), x[3] * math.cos(t1) + x[1] * math.sin(t1)]
    assert np.allclose(y, want, rtol=0, atol=1e-15)


def test_pairs_keep_their_length():
    rng = np.random.default_rng(4)
    x = rng.normal(size=64)
    for pos in (1, 17, 4095, 32768):
        y = oracle.rope_f64(x, pos, 32, 10000.0)
        for j in range(16):
            assert math.isclose(x[j] ** 2 + x[j + 16] ** 2, y[j] ** 2 + y[j + 16] ** 2,
                                rel_tol=1e-12)


def test_scores_depend_only_on_the_position_difference():
    """The defining property: rope(q, m) . rope(k, n) is a function of m - n."""
    rng = np.random.default_rng(5)
    q, k = rng.normal(size=64), rng.normal(size=64)
    for rd in (16, 64):
        for m, n in ((10, 3), (2049, 2000), (32768, 1)):
            base = np.dot(oracle.rope_f64(q, m, rd), oracle.rope_f64(k, n, rd))
            for t in (1, 37, 1000):
                shifted = np.dot(oracle.rope_f64(q, m + t, rd), oracle.rope_f64(k, n + t, rd))
                assert math.isclose(base, shifted, rel_tol=1e-9, abs_tol=1e-9)
            rel = np.dot(oracle.rope_f64(q, m - n, rd), oracle.rope_f64(k, 0, rd))
            assert math.isclose(base, rel, rel_tol=1e-9, abs_tol=1e-9)


def test_bf16_rope_is_the_rounded_double_rotation():
    x = synth.normal_bf16(6, 0, (64,))
    xd = synth.bf16_to_f32(x).astype(np.float64)
    for pos in (1, 511, 2048, 32767):
        y = oracle.rope(x, pos, 16)
        yd = oracle.rope_f64(xd, pos, 16)
        assert np.array_equal(y, [oracle.bf16_from_double(v) for v in yd])


def test_step_with_rope_is_the_step_on_rotated_inputs():
    """decode_step_rope = decode_step on queries and new keys rotated at the
    new token's position (the cache holds keys rotated when appended)."""
    w = synth.Workload("rope_tiny", l=4, h=4, m=2, g=2, D=64, B=3, ctx=40, seed=8)
    inp = synth.step_inputs(w, fill=synth.BF16_NAN)
    ctx = np.array([0, 17, 40], np.int32)
    for arr in (inp["k_cache"], inp["v_cache"]):
        for b, c in enumerate(ctx):
            arr[:, b, c:] = synth.BF16_NAN
    kv_of, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
    q_rot = np.empty_like(inp["q"])
    for n in range(w.l):
        for b in range(w.B):
            for i in range(w.h):
                q_rot[n, b, i] = oracle.rope(inp["q"][n, b, i], ctx[b], 16)
    k_rot = np.empty_like(inp["k_new"])
    for b in range(w.B):
        for kv in range(w.n_kv):
            k_rot[b, kv] = oracle.rope(inp["k_new"][b, kv], ctx[b], 16)
    k1, v1 = inp["k_cache"].copy(), inp["v_cache"].copy()
    ref = oracle.decode_step(q_rot, k1, v1, k_rot, inp["v_new"], kv_of, owner_of, ctx)
    k2, v2 = inp["k_cache"].copy(), inp["v_cache"].copy()
    got = oracle.decode_step_rope(inp["q"], k2, v2, inp["k_new"], inp["v_new"], kv_of, owner_of,
                                  ctx, 16)
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
    assert np.array_equal(got, ref)

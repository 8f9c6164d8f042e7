"""Pins of the prefill oracle (T new tokens per sequence, causal).

Each pin ties the prefill to something other than its own formula: the decode
step it must reduce to (itself pinned in test_oracle.py), the same tokens fed
one decode step at a time, torch's scaled_dot_product_attention with an
explicit causal mask, causality itself, a two-token closed form, and the
cache rows the owners must write.
"""
import math

import numpy as np
import pytest

import oracle
import synth


def _f(x):
    return synth.bf16_to_f32(np.asarray(x, dtype=np.uint16)).astype(np.float64)


def _case(l=4, h=6, m=2, g=2, D=16, B=3, T=5, ctx=(0, 3, 9), seed=31, S=None):
    """Random prefill inputs; cache slots past each context are NaN-poisoned."""
    ctx = np.asarray(ctx, dtype=np.int32)
    assert ctx.size == B
    n_kv = m * g
    S = S or int(ctx.max()) + T + 2
    q = synth.normal_bf16(seed, 0, (l, B, T, h, D))
    k_new = synth.normal_bf16(seed, 3, (B, T, n_kv, D))
    v_new = synth.normal_bf16(seed, 4, (B, T, n_kv, D))
    lens = np.tile(ctx, n_kv)
    kc = synth.rows_bf16(seed, 1, n_kv * B, S, D, lens, fill=synth.BF16_NAN).reshape(n_kv, B, S, D)
    vc = synth.rows_bf16(seed, 2, n_kv * B, S, D, lens, fill=synth.BF16_NAN).reshape(n_kv, B, S, D)
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    return dict(q=q, k_new=k_new, v_new=v_new, kc=kc, vc=vc, ctx=ctx, kv_of=kv_of,
                owner_of=owner_of)


def _prefill(c):
    kc, vc = c["kc"].copy(), c["vc"].copy()
    out = oracle.prefill_step(c["q"], kc, vc, c["k_new"], c["v_new"], c["kv_of"], c["owner_of"],
                              c["ctx"])
    return out, kc, vc


def test_one_new_token_is_the_decode_step():
    """T = 1: the prefill is exactly the (separately pinned) decode step."""
    c = _case(T=1, ctx=(0, 4, 11))
    out, kc, vc = _prefill(c)
    kd, vd = c["kc"].copy(), c["vc"].copy()
    ref = oracle.decode_step(c["q"][:, :, 0], kd, vd, c["k_new"][:, 0], c["v_new"][:, 0],
                             c["kv_of"], c["owner_of"], c["ctx"])
    assert np.array_equal(out[:, :, 0], ref)
    assert np.array_equal(kc, kd) and np.array_equal(vc, vd)


@pytest.mark.parametrize("lmg", [(4, 6, 2, 2), (3, 6, 3, 1), (2, 4, 1, 4)])
def test_prompt_equals_decode_steps_one_token_at_a_time(lmg):
    """Feeding the T tokens one decode step at a time (context ctx + t for
    token t) gives the same outputs and the same cache, bit for bit."""
    l, h, m, g = lmg
    c = _case(l=l, h=h, m=m, g=g, T=6, ctx=(0, 2, 7))
    out, kc, vc = _prefill(c)
    kd, vd = c["kc"].copy(), c["vc"].copy()
    for t in range(6):
        ref = oracle.decode_step(np.ascontiguousarray(c["q"][:, :, t]), kd, vd,
                                 np.ascontiguousarray(c["k_new"][:, t]),
                                 np.ascontiguousarray(c["v_new"][:, t]), c["kv_of"],
                                 c["owner_of"], c["ctx"] + t)
        assert np.array_equal(out[:, :, t], ref), t
    assert np.array_equal(kc, kd) and np.array_equal(vc, vd)


def test_matches_torch_sdpa_with_a_causal_mask():
    """Every layer against torch's SDPA in fp64 over the full key/value rows
    of its KV heads (cached prefix then the new tokens, repeated over the
    query heads of a group) with a boolean mask: new token t sees positions
    up to ctx + t."""
    torch = pytest.importorskip("torch")
    l, h, m, g, D, B, T = 4, 6, 2, 3, 16, 3, 7
    c = _case(l=l, h=h, m=m, g=g, D=D, B=B, T=T, ctx=(0, 5, 12))
    out, _, _ = _prefill(c)
    for n in range(l):
        grp = n // (l // m)
        for b in range(B):
            L = int(c["ctx"][b]) + T
            K = np.empty((g, L, D))
            V = np.empty((g, L, D))
            for j in range(g):
                kv = grp * g + j
                K[j, :c["ctx"][b]] = _f(c["kc"][kv, b, :c["ctx"][b]])
                V[j, :c["ctx"][b]] = _f(c["vc"][kv, b, :c["ctx"][b]])
                K[j, c["ctx"][b]:] = _f(c["k_new"][b, :, kv])
                V[j, c["ctx"][b]:] = _f(c["v_new"][b, :, kv])
            K = np.repeat(K, h // g, axis=0)
            V = np.repeat(V, h // g, axis=0)
            Q = _f(c["q"][n, b]).transpose(1, 0, 2)  # [h][T][D]
            mask = np.arange(L)[None, :] <= (c["ctx"][b] + np.arange(T))[:, None]
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(np.ascontiguousarray(Q)), torch.from_numpy(K),
                torch.from_numpy(V), attn_mask=torch.from_numpy(mask))
            np.testing.assert_allclose(out[n, b], ref.numpy().transpose(1, 0, 2), rtol=0,
                                       atol=1e-12)


def test_later_tokens_do_not_change_earlier_outputs():
    """Causality: changing the queries, keys and values of tokens t >= 3
    leaves the outputs of tokens 0..2 unchanged in every layer."""
    c = _case(T=6, ctx=(1, 0, 4))
    out, _, _ = _prefill(c)
    c2 = dict(c)
    for name, stream in (("k_new", 7), ("v_new", 8)):
        a = c[name].copy()
        a[:, 3:] = synth.normal_bf16(99, stream, a[:, 3:].shape)
        c2[name] = a
    qq = c["q"].copy()
    qq[:, :, 3:] = synth.normal_bf16(99, 9, qq[:, :, 3:].shape)
    c2["q"] = qq
    out2, _, _ = _prefill(c2)
    assert np.array_equal(out[:, :, :3], out2[:, :, :3])
    assert not np.allclose(out[:, :, 3:], out2[:, :, 3:])


def test_two_new_tokens_closed_form():
    """Empty cache, two tokens: the first sees only itself (its own value),
    the second mixes the two values by sigmoid(s1 - s0), s = q.k / sqrt(D)."""
    D = 16
    c = _case(l=1, h=1, m=1, g=1, D=D, B=1, T=2, ctx=(0,), seed=12)
    out, _, _ = _prefill(c)
    v0, v1 = _f(c["v_new"][0, 0, 0]), _f(c["v_new"][0, 1, 0])
    k0, k1 = _f(c["k_new"][0, 0, 0]), _f(c["k_new"][0, 1, 0])
    q1 = _f(c["q"][0, 0, 1, 0])
    assert np.array_equal(out[0, 0, 0, 0], v0)
    s0, s1 = q1 @ k0 / math.sqrt(D), q1 @ k1 / math.sqrt(D)
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    np.testing.assert_allclose(out[0, 0, 1, 0], v0 + w1 * (v1 - v0), rtol=0, atol=1e-13)


def test_owners_write_the_new_rows_at_consecutive_slots():
    """After the prefill, slots ctx_b .. ctx_b + T - 1 of every KV head hold
    the new rows; the cached prefix is unchanged and every slot past the end
    is still NaN-poisoned."""
    c = _case(T=4, ctx=(0, 6, 2))
    _, kc, vc = _prefill(c)
    n_kv = kc.shape[0]
    for kv in range(n_kv):
        for b in range(3):
            cb = int(c["ctx"][b])
            assert np.array_equal(kc[kv, b, :cb], c["kc"][kv, b, :cb])
            assert np.array_equal(kc[kv, b, cb:cb + 4], c["k_new"][b, :, kv])
            assert np.array_equal(vc[kv, b, cb:cb + 4], c["v_new"][b, :, kv])
            assert np.all(kc[kv, b, cb + 4:] == synth.BF16_NAN)
            assert np.all(vc[kv, b, cb + 4:] == synth.BF16_NAN)


def test_non_owning_layer_appends_nothing():
    """append_rows in a layer that owns no KV head changes nothing."""
    c = _case(l=4, m=2, T=3)
    kc, vc = c["kc"].copy(), c["vc"].copy()
    assert oracle.append_rows(1, kc, vc, c["k_new"], c["v_new"], c["owner_of"], c["ctx"]) == 0
    assert np.array_equal(kc, c["kc"]) and np.array_equal(vc, c["vc"])

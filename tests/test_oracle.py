"""Pins of the oracle against facts the paper and the mathematics fix.

None of these re-types the oracle's own formulas: each checks a special case,
a closed form, an invariant, a library routine or a printed table.  A dropped
scale, a wrong group index, a transposed operand or a missing max-shift in the
oracle makes at least one of them fail (tests/test_oracle_mutants.py plants each
such mistake in a copy of the oracle and checks that a pin catches it).
"""
import math
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _bf16(x):
    return synth.f32_to_bf16(np.asarray(x, dtype=np.float32))


def _f(x):
    return synth.bf16_to_f32(np.asarray(x, dtype=np.uint16)).astype(np.float64)


# ----------------------------------------------------------------------- map --

@pytest.mark.parametrize("row", _read_table("table2_variants.txt"), ids=lambda r: r[0])
def test_map_matches_table2_head_counts(row):
    """Table 2 / Section 5.3: (l, h, m, g) -> mg total KV heads; every KV head is
    read, owned by the bottom layer of a contiguous block of l/m layers, and the
    query heads of a layer split into g contiguous blocks of h/g (Eq. 12)."""
    name, l, h, m, g, mg = row[0], *map(int, row[1:])
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    assert kv_of.shape == (l, h)
    assert len(np.unique(kv_of)) == mg
    assert sorted(np.unique(kv_of)) == list(range(mg))
    assert len(owner_of) == mg
    for kv in range(mg):
        readers = sorted({n for n in range(l) for i in range(h) if kv_of[n, i] == kv})
        # contiguous block of l/m layers; the owner is its bottom layer (Figure 2)
        assert readers == list(range(readers[0], readers[0] + l // m))
        assert owner_of[kv] == readers[0]
    for n in range(l):
        heads_of = {}
        for i in range(h):
            heads_of.setdefault(int(kv_of[n, i]), []).append(i)
        assert len(heads_of) == g
        for kv, heads in heads_of.items():
            assert heads == list(range(heads[0], heads[0] + h // g))


def test_map_special_cases():
    # MHA: every query head has its own KV head (Section 2.1).
    kv_of, owner_of = oracle.map_uniform(3, 4, 3, 4)
    assert sorted(kv_of.ravel()) == list(range(12))
    for n in range(3):
        for i in range(4):
            assert owner_of[kv_of[n, i]] == n
    # MQA: one KV head per layer shared by all its query heads (Section 2.2).
    kv_of, owner_of = oracle.map_uniform(5, 6, 5, 1)
    for n in range(5):
        assert len(set(kv_of[n])) == 1
        assert owner_of[kv_of[n, 0]] == n
    assert len(np.unique(kv_of)) == 5
    # Owners quoted for the decode workloads.
    assert list(oracle.map_uniform(12, 12, 2, 1)[1]) == [0, 6]
    assert list(oracle.map_uniform(12, 12, 4, 1)[1]) == [0, 3, 6, 9]
    own = oracle.map_uniform(32, 32, 8, 8)[1]
    assert list(own) == [4 * (k // 8) for k in range(64)]
    # Non-divisible shapes are rejected (the paper's configurations all divide).
    with pytest.raises(ValueError):
        oracle.map_uniform(12, 12, 5, 1)
    with pytest.raises(ValueError):
        oracle.map_uniform(12, 12, 4, 5)


def test_mlkv_two_heads_is_six_times_smaller_than_mqa():
    """Abstract / Section 6: MLKV reduces the cache up to 6x versus MQA
    (MQA-12 has 12 KV heads, MLKV-2 has 2)."""
    mqa = len(np.unique(oracle.map_uniform(12, 12, 12, 1)[0]))
    mlkv2 = len(np.unique(oracle.map_uniform(12, 12, 2, 1)[0]))
    assert mqa / mlkv2 == 6


def test_cache_size_ratios_match_table1():
    """Table 1 ratios for OPT-175B (b=8, s=1024, l=h=96, d_k=128)."""
    printed = {r[0]: float(r[1]) for r in _read_table("table1_cache_sizes.txt")}
    b, s, l, h, dk = 8, 1024, 96, 96, 128
    n = {
        "mha": oracle.cache_elements("mha", b, s, l, h, dk),
        "mqa": oracle.cache_elements("mqa", b, s, l, h, dk),
        "gqa": oracle.cache_elements("gqa", b, s, l, h, dk, g=24),
        "mlkv": oracle.cache_elements("mlkv", b, s, l, h, dk, m=24, g=1),
    }
    for a in n:
        for c in n:
            assert n[a] / n[c] == pytest.approx(printed[a] / printed[c], rel=1e-12)
    # absolute values: fp16 bytes in GiB are a quarter of the printed numbers
    for a in n:
        assert n[a] * 2 / 2**30 == pytest.approx(printed[a] / 4, rel=1e-12)
    # Section 3: with g = 1 the MLKV cache is m/l of the MQA cache
    for m in (1, 2, 3, 4, 6, 12):
        assert (oracle.cache_elements("mlkv", b, s, 12, 12, 64, m=m, g=1)
                / oracle.cache_elements("mqa", b, s, 12, 12, 64)) == pytest.approx(m / 12)


# ----------------------------------------------------------------- attention --

def _brute_force_head(q, K, V):
    """Independent per-head loops in pure Python floats."""
    D = len(q)
    s = [sum(float(q[d]) * float(K[t][d]) for d in range(D)) / math.sqrt(D)
         for t in range(len(K))]
    mx = max(s)
    w = [math.exp(x - mx) for x in s]
    z = math.fsum(w)
    return [math.fsum(w[t] * float(V[t][d]) for t in range(len(K))) / z for d in range(D)]


def _rand_case(seed, l, h, m, g, D, B, S, lens):
    n_kv = m * g
    q = synth.normal_bf16(seed, 0, (B, h, D))
    kc = synth.rows_bf16(seed, 1, n_kv * B, S, D, np.tile(lens, n_kv)).reshape(n_kv, B, S, D)
    vc = synth.rows_bf16(seed, 2, n_kv * B, S, D, np.tile(lens, n_kv)).reshape(n_kv, B, S, D)
    return q, kc, vc


@pytest.mark.parametrize("lmg", [(2, 4, 2, 4), (2, 4, 2, 1), (4, 4, 2, 2), (3, 6, 1, 3)])
def test_decode_attention_matches_brute_force(lmg):
    l, h, m, g = lmg
    D, B, S = 8, 3, 7
    lens = np.array([1, 5, 7], dtype=np.int32)
    q, kc, vc = _rand_case(11, l, h, m, g, D, B, S, lens)
    kv_of, _ = oracle.map_uniform(l, h, m, g)
    for layer in range(l):
        out = oracle.decode_attention(layer, q, kc, vc, kv_of, lens)
        for b in range(B):
            for i in range(h):
                kv = kv_of[layer, i]
                L = lens[b]
                ref = _brute_force_head(_f(q[b, i]), _f(kc[kv, b, :L]), _f(vc[kv, b, :L]))
                np.testing.assert_allclose(out[b, i], ref, rtol=0, atol=1e-13)


def test_identity_map_matches_torch_sdpa_fp64():
    """MHA (identity map) against torch's scaled_dot_product_attention in fp64."""
    torch = pytest.importorskip("torch")
    l, h, D, B, S = 2, 4, 16, 2, 40
    lens = np.array([40, 40], dtype=np.int32)
    q, kc, vc = _rand_case(5, l, h, l, h, D, B, S, lens)
    # MHA numbering: query head i of layer n has its own KV head n*h + i
    kv_of = np.arange(l * h, dtype=np.int32).reshape(l, h)
    for layer in range(l):
        out = oracle.decode_attention(layer, q, kc, vc, kv_of, lens)
        K = _f(kc[layer * h:(layer + 1) * h]).transpose(1, 0, 2, 3)  # [B][h][S][D]
        V = _f(vc[layer * h:(layer + 1) * h]).transpose(1, 0, 2, 3)
        K, V = np.ascontiguousarray(K), np.ascontiguousarray(V)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(_f(q)[:, :, None, :]), torch.from_numpy(K), torch.from_numpy(V))
        np.testing.assert_allclose(out, ref[:, :, 0, :].numpy(), rtol=0, atol=1e-12)


def test_gqa_matches_torch_sdpa_with_repeated_kv():
    """GQA/MLKV grouping: SDPA over K/V repeated h/g times (Eq. 12)."""
    torch = pytest.importorskip("torch")
    l, h, m, g, D, B, S = 4, 6, 2, 2, 8, 2, 33
    lens = np.array([33, 33], dtype=np.int32)
    q, kc, vc = _rand_case(6, l, h, m, g, D, B, S, lens)
    kv_of, _ = oracle.map_uniform(l, h, m, g)
    for layer in range(l):
        k_grp = layer // (l // m)
        K = _f(kc[k_grp * g:(k_grp + 1) * g]).transpose(1, 0, 2, 3)  # [B][g][S][D]
        V = _f(vc[k_grp * g:(k_grp + 1) * g]).transpose(1, 0, 2, 3)
        K = np.repeat(K, h // g, axis=1)
        V = np.repeat(V, h // g, axis=1)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(_f(q)[:, :, None, :]), torch.from_numpy(np.ascontiguousarray(K)),
            torch.from_numpy(np.ascontiguousarray(V)))
        out = oracle.decode_attention(layer, q, kc, vc, kv_of, lens)
        np.testing.assert_allclose(out, ref[:, :, 0, :].numpy(), rtol=0, atol=1e-12)


def test_two_tokens_closed_form():
    """L = 2: o = v0 + (v1 - v0) * sigmoid((s1 - s0)), s_t = q.k_t / sqrt(D)."""
    D = 16
    q = synth.normal_bf16(1, 0, (D,))
    K = synth.normal_bf16(1, 1, (2, D))
    V = synth.normal_bf16(1, 2, (2, D))
    o, alpha = oracle.attend_one(q, K, V)
    s = _f(K) @ _f(q) / 4.0
    sig = 1.0 / (1.0 + math.exp(-(s[1] - s[0])))
    np.testing.assert_allclose(o, _f(V[0]) + (_f(V[1]) - _f(V[0])) * sig, rtol=0, atol=1e-14)
    np.testing.assert_allclose(alpha, [1 - sig, sig], rtol=0, atol=1e-15)


def test_single_position_returns_v_exactly():
    for D in (8, 64, 128):
        q = synth.normal_bf16(2, 0, (D,))
        K = synth.normal_bf16(2, 1, (1, D), scale=50.0)
        V = synth.normal_bf16(2, 2, (1, D))
        o, alpha = oracle.attend_one(q, K, V)
        assert np.array_equal(o, _f(V[0]))
        assert alpha[0] == 1.0


def test_identical_keys_give_mean_of_values():
    D, L = 32, 37
    q = synth.normal_bf16(3, 0, (D,))
    k = synth.normal_bf16(3, 1, (1, D))
    K = np.repeat(k, L, axis=0)
    V = synth.normal_bf16(3, 2, (L, D))
    o, alpha = oracle.attend_one(q, K, V)
    np.testing.assert_allclose(alpha, np.full(L, 1.0 / L), rtol=1e-14)
    np.testing.assert_allclose(o, _f(V).mean(axis=0), rtol=0, atol=1e-14)


def test_weights_sum_to_one_and_are_nonnegative():
    D, L = 64, 1000
    q = synth.normal_bf16(4, 0, (D,))
    K = synth.normal_bf16(4, 1, (L, D), scale=3.0)
    V = synth.normal_bf16(4, 2, (L, D))
    _, alpha = oracle.attend_one(q, K, V)
    assert np.all(alpha >= 0)
    assert abs(math.fsum(alpha) - 1.0) < 1e-13


def test_shift_invariance_of_scores():
    """Adding c*q/|q|^2-like shifts: with q = e_0, K_t[0] += c shifts every score
    by c/sqrt(D); softmax is unchanged.  Values chosen exactly representable."""
    D, L = 16, 9
    q = np.zeros(D, dtype=np.float32)
    q[0] = 1.0
    rng = np.random.default_rng(0)
    K = rng.integers(-8, 8, size=(L, D)).astype(np.float32) * 0.25
    V = synth.normal_bf16(5, 2, (L, D))
    o1, a1 = oracle.attend_one(_bf16(q), _bf16(K), V)
    K2 = K.copy()
    K2[:, 0] += 6.0
    o2, a2 = oracle.attend_one(_bf16(q), _bf16(K2), V)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(a1, a2, rtol=0, atol=1e-15)


def test_token_permutation_invariance():
    D, L = 64, 300
    q = synth.normal_bf16(6, 0, (D,))
    K = synth.normal_bf16(6, 1, (L, D))
    V = synth.normal_bf16(6, 2, (L, D))
    perm = np.random.default_rng(1).permutation(L)
    o1, a1 = oracle.attend_one(q, K, V)
    o2, a2 = oracle.attend_one(q, K[perm], V[perm])
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(a1[perm], a2, rtol=0, atol=1e-15)


@pytest.mark.parametrize("pos", [0, 31, 32, 63, 199])
def test_needle_dominates_and_large_scores_stay_finite(pos):
    """A key aligned with q and scaled huge takes all the weight: o = v_needle.
    Scores near 1e4 would overflow exp() without the max shift."""
    D, L = 64, 200
    q = synth.normal_bf16(7, 0, (D,))
    K = synth.normal_bf16(7, 1, (L, D))
    V = synth.normal_bf16(7, 2, (L, D))
    K[pos] = _bf16(_f(q) * 200.0)
    o, alpha = oracle.attend_one(q, K, V)
    assert np.all(np.isfinite(o))
    assert alpha[pos] == pytest.approx(1.0, abs=1e-12)
    np.testing.assert_allclose(o, _f(V[pos]), rtol=0, atol=1e-12)


def test_empty_attention_is_zero():
    q = synth.normal_bf16(8, 0, (64,))
    o, alpha = oracle.attend_one(q, np.zeros((0, 64), np.uint16), np.zeros((0, 64), np.uint16))
    assert np.all(o == 0) and alpha.size == 0


# ------------------------------------------------------------ append / step --

def test_append_writes_only_owned_slots():
    l, h, m, g, D, B, S = 12, 12, 4, 1, 8, 3, 10
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    n_kv = m * g
    kc = np.full((n_kv, B, S, D), synth.BF16_NAN, np.uint16)
    vc = kc.copy()
    kn = synth.normal_bf16(9, 3, (B, n_kv, D))
    vn = synth.normal_bf16(9, 4, (B, n_kv, D))
    pos = np.array([0, 4, 9], np.int32)
    for layer in range(l):
        before_k, before_v = kc.copy(), vc.copy()
        owned = oracle.append(layer, kc, vc, kn, vn, owner_of, pos)
        assert owned == (1 if layer % 3 == 0 else 0)
        changed = np.argwhere(np.any(kc != before_k, axis=-1))
        if owned:
            kv = layer // 3
            assert sorted(map(tuple, changed)) == [(kv, b, pos[b]) for b in range(B)]
            for b in range(B):
                assert np.array_equal(kc[kv, b, pos[b]], kn[b, kv])
                assert np.array_equal(vc[kv, b, pos[b]], vn[b, kv])
        else:
            assert changed.size == 0 and np.array_equal(vc, before_v)
    # out-of-range positions write nothing
    before = kc.copy()
    oracle.append(0, kc, vc, kn, vn, owner_of, np.array([-1, S, S + 5], np.int32))
    assert np.array_equal(kc, before)


def test_step_mlkv2_empty_context_outputs_owner_values():
    """MLKV-2 with nothing cached: every layer of group k attends one position,
    the token its bottom layer appended this step, so o = v_new (Section 3 and
    Figure 2 ownership; L = 1 case)."""
    l, h, m, g, D, B = 12, 12, 2, 1, 64, 2
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    S = 64
    kc = np.full((2, B, S, D), synth.BF16_NAN, np.uint16)
    vc = kc.copy()
    q = synth.normal_bf16(10, 0, (l, B, h, D))
    kn = synth.normal_bf16(10, 3, (B, 2, D))
    vn = synth.normal_bf16(10, 4, (B, 2, D))
    out = oracle.decode_step(q, kc, vc, kn, vn, kv_of, owner_of, np.zeros(B, np.int32))
    for n in range(l):
        for b in range(B):
            for i in range(h):
                assert np.array_equal(out[n, b, i], _f(vn[b, n // 6]))


def test_step_non_owner_layer_sees_token_appended_this_step():
    """A needle in the new token of KV head 0, aligned with layer 2's query
    head 5 (a non-owning layer of the group): that head returns v_new."""
    l, h, m, g, D, B = 12, 12, 4, 1, 64, 1
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    S, ctx = 128, 100
    kc = synth.rows_bf16(12, 1, 4, S, D, np.full(4, ctx)).reshape(4, B, S, D)
    vc = synth.rows_bf16(12, 2, 4, S, D, np.full(4, ctx)).reshape(4, B, S, D)
    q = synth.normal_bf16(12, 0, (l, B, h, D))
    kn = synth.normal_bf16(12, 3, (B, 4, D))
    vn = synth.normal_bf16(12, 4, (B, 4, D))
    kn[0, 0] = _bf16(_f(q[2, 0, 5]) * 100.0)
    out = oracle.decode_step(q, kc, vc, kn, vn, kv_of, owner_of, np.array([ctx], np.int32))
    np.testing.assert_allclose(out[2, 0, 5], _f(vn[0, 0]), rtol=0, atol=1e-12)
    assert np.array_equal(kc[0, 0, ctx], kn[0, 0])


def test_golden_tiny_step_regression():
    """Stored outputs of a tiny seeded step, written by tests/golden/make_golden.py
    (which calls only the oracle); guards against unintended oracle drift."""
    path = os.path.join(GOLDEN, "tiny_step_outputs.txt")
    data = np.loadtxt(path)
    import importlib.util
    spec = importlib.util.spec_from_file_location("make_golden", os.path.join(GOLDEN, "make_golden.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    out = mod.tiny_step()
    np.testing.assert_allclose(out.ravel(), data, rtol=0, atol=1e-15)


# ----------------------------------------------------------------- generator --

def test_generator_is_deterministic_and_sliceable():
    a = synth.normal_bf16(123, 1, (1000,))
    b = synth.normal_bf16(123, 1, (400,), first=600)
    assert np.array_equal(a[600:], b)
    r = synth.rows_bf16(7, 1, 6, 50, 16)
    r2 = synth.rows_bf16(7, 1, 2, 50, 16, row0=3)
    assert np.array_equal(r[3:5], r2)
    # capacity does not change the values of valid tokens
    r3 = synth.rows_bf16(7, 1, 6, 80, 16, lens=np.full(6, 50), fill=synth.BF16_NAN)
    assert np.array_equal(r3[:, :50], r)
    assert np.all(r3[:, 50:] == synth.BF16_NAN)
    x = synth.bf16_to_f32(synth.normal_bf16(1, 0, (200000,)))
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01
    n = synth.uniform_int(3, 5, 10000, 512, 2048)
    assert n.min() >= 512 and n.max() <= 2048 and len(np.unique(n)) > 1000

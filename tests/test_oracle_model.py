"""Pins of the model-level oracle (oracle/model.py): one decode step of a
GPT-NeoX model with an MLKV map.

- layer norm and GELU against torch's own routines in float64;
- the whole step with a one-KV-head-per-query-head map (plain multi-head
  attention) against an independent implementation of the architecture,
  transformers' GPTNeoXModel in float64: the prefix's keys and values come
  from that model's cache, the new token's last-layer output must match its
  full-sequence forward pass;
- with an MLKV map, the attention of every layer reduces to the separately
  pinned decode-step oracle (oracle.decode_step) fed with the model's own
  rotated queries and the owners' rows.
"""
import numpy as np
import pytest

import oracle
import oracle.model as om
import synth

torch = pytest.importorskip("torch")


def _bits(x):
    return synth.f32_to_bf16(np.asarray(x, dtype=np.float32))


def test_layer_norm_and_gelu_match_torch():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 48)) * 3 + 1
    w, b = rng.standard_normal(48), rng.standard_normal(48)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(w),
                                         torch.from_numpy(b), eps=1e-5).numpy()
    np.testing.assert_allclose(om.layer_norm(x, w, b, 1e-5), ref, rtol=0, atol=1e-13)
    g = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(om.gelu(x), g, rtol=0, atol=1e-14)


def test_to_bf16_is_nearest_even():
    x = np.random.default_rng(4).standard_normal(5000) * 10
    bits = np.array([oracle.bf16_from_double(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(om.to_bf16(x), om._f64(bits))


def _hf_model(l, d, h, d_ff, rd, seed):
    transformers = pytest.importorskip("transformers")
    cfg = transformers.GPTNeoXConfig(
        vocab_size=8, hidden_size=d, num_hidden_layers=l, num_attention_heads=h,
        intermediate_size=d_ff, rotary_pct=rd / (d // h), rotary_emb_base=10000,
        max_position_embeddings=64, use_parallel_residual=True, hidden_act="gelu",
        layer_norm_eps=1e-5, attn_implementation="eager")
    m = transformers.GPTNeoXModel(cfg).double().eval()
    gen = torch.Generator().manual_seed(seed)
    with torch.no_grad():
        for name, p in m.named_parameters():
            scale = 0.5 if "layernorm" in name else 0.08
            base = 1.0 if name.endswith("layernorm.weight") else 0.0
            r = base + scale * torch.randn(p.shape, generator=gen, dtype=torch.float64)
            p.copy_(torch.from_numpy(om.to_bf16(r.numpy())))  # bf16-representable
    # transformers evaluates the rotary angles and their sine and cosine in
    # float32 whatever the model's precision; the same formula in float64:
    inv_freq = 10000.0 ** (-torch.arange(0, rd, 2, dtype=torch.float64) / rd)

    def rotary64(x, position_ids):
        freqs = position_ids[:, :, None].to(torch.float64) * inv_freq[None, None, :]
        emb = torch.cat((freqs, freqs), dim=-1)
        return emb.cos().to(x.dtype), emb.sin().to(x.dtype)

    m.rotary_emb.forward = rotary64
    return m


def _weights_from_hf(m, h, D):
    layers = []
    for layer in m.layers:
        W = layer.attention.query_key_value.weight.detach().numpy()   # [h*3D][d]
        bqkv = layer.attention.query_key_value.bias.detach().numpy()
        rows = lambda part: np.concatenate([np.arange(i * 3 * D + part * D, i * 3 * D + (part + 1) * D)
                                            for i in range(h)])
        pick = lambda part: (_bits(W[rows(part)].T), _bits(bqkv[rows(part)]))
        (wq, bq), (wk, bk), (wv, bv) = pick(0), pick(1), pick(2)
        layers.append(dict(
            ln1_w=_bits(layer.input_layernorm.weight.detach().numpy()),
            ln1_b=_bits(layer.input_layernorm.bias.detach().numpy()),
            ln2_w=_bits(layer.post_attention_layernorm.weight.detach().numpy()),
            ln2_b=_bits(layer.post_attention_layernorm.bias.detach().numpy()),
            w_q=wq, b_q=bq, w_k=wk, b_k=bk, w_v=wv, b_v=bv,
            w_o=_bits(layer.attention.dense.weight.detach().numpy().T),
            b_o=_bits(layer.attention.dense.bias.detach().numpy()),
            w_fc1=_bits(layer.mlp.dense_h_to_4h.weight.detach().numpy().T),
            b_fc1=_bits(layer.mlp.dense_h_to_4h.bias.detach().numpy()),
            w_fc2=_bits(layer.mlp.dense_4h_to_h.weight.detach().numpy().T),
            b_fc2=_bits(layer.mlp.dense_4h_to_h.bias.detach().numpy())))
    return layers


def _eager_attention_fp64(module, query, key, value, attention_mask, scaling, dropout=0.0,
                          **kwargs):
    """transformers' eager attention with its softmax kept in float64 (the
    library forces float32 there)."""
    w = torch.matmul(query, key.transpose(2, 3)) * scaling
    if attention_mask is not None:
        w = w + attention_mask
    w = torch.nn.functional.softmax(w, dim=-1, dtype=torch.float64)
    return torch.matmul(w, value).transpose(1, 2).contiguous(), w


def _check_mha_against_transformers(model_oracle, monkeypatch):
    l, d, h, d_ff, rd, B, P = 3, 64, 4, 160, 4, 2, 6
    D = d // h
    m = _hf_model(l, d, h, d_ff, rd, seed=5)
    import transformers.models.gpt_neox.modeling_gpt_neox as neox
    monkeypatch.setattr(neox, "eager_attention_forward", _eager_attention_fp64)
    x = torch.randn(B, P + 1, d, dtype=torch.float64, generator=torch.Generator().manual_seed(6))
    captured = {}
    hook = m.layers[-1].register_forward_hook(
        lambda mod, inp, out: captured.__setitem__("x", out[0] if isinstance(out, tuple) else out))
    with torch.no_grad():
        m(inputs_embeds=x)
        full = captured["x"][:, P].numpy()
        pre = m(inputs_embeds=x[:, :P], use_cache=True)
    hook.remove()
    n_kv = l * h
    S = P + 2
    kc = np.zeros((n_kv, B, S, D))
    vc = np.zeros((n_kv, B, S, D))
    for n in range(l):
        keys = pre.past_key_values.layers[n].keys.numpy()
        vals = pre.past_key_values.layers[n].values.numpy()
        for i in range(h):
            kc[n * h + i, :, :P] = keys[:, i]
            vc[n * h + i, :, :P] = vals[:, i]
    kv_of = np.arange(n_kv).reshape(l, h)
    owner_of = np.repeat(np.arange(l), h)
    ctx = np.full(B, P)
    out = model_oracle.decode_step_model(x[:, P].numpy(), _weights_from_hf(m, h, D), kv_of,
                                         owner_of, kc, vc, ctx, h, D, rd, round_bf16=False)
    np.testing.assert_allclose(out, full, rtol=0, atol=1e-10)


def test_mha_step_matches_transformers_gpt_neox(monkeypatch):
    _check_mha_against_transformers(om, monkeypatch)


# Planted mistakes in copies of oracle/model.py, each caught by the pin above.
MODEL_MUTANTS = [
    ("attention_added_twice", "x = x + a + m", "x = x + a + m + a"),
    ("gelu_tanh_form", "return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))",
     "return 0.5 * x * (1.0 + np.tanh(0.7978845608 * (x + 0.044715 * x ** 3)))"),
    ("norm_without_eps", "return (x - mu) / np.sqrt(var + eps) * w + b",
     "return (x - mu) / np.sqrt(var) * w + b"),
    ("mlp_from_first_norm", "f = rb(gelu(h2 @ g[\"w_fc1\"] + g[\"b_fc1\"]))",
     "f = rb(gelu(h1 @ g[\"w_fc1\"] + g[\"b_fc1\"]))"),
    ("query_not_rotated", "q = rb(np.stack([np.stack([rope_f64(q[b, i], int(ctx[b]), rd, base)",
     "q = rb(np.stack([np.stack([rope_f64(q[b, i], 0, rd, base)"),
    ("key_rotated_at_next_position", "k = rb(np.stack([np.stack([rope_f64(k[b, c], int(ctx[b]), rd, base)",
     "k = rb(np.stack([np.stack([rope_f64(k[b, c], int(ctx[b]) + 1, rd, base)"),
]


@pytest.mark.parametrize("name,old,new", MODEL_MUTANTS, ids=[m[0] for m in MODEL_MUTANTS])
def test_planted_model_mistake_is_caught(name, old, new, monkeypatch):
    import importlib.util
    import os
    import sys

    src = open(os.path.join(os.path.dirname(oracle.__file__), "model.py")).read()
    assert src.count(old) == 1, f"anchor of {name} not found exactly once"
    spec = importlib.util.spec_from_loader("oracle._mutant_model", loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"
    sys.modules["oracle._mutant_model"] = mod
    try:
        exec(compile(src.replace(old, new), "mutant_model.py", "exec"), mod.__dict__)
        with pytest.raises(AssertionError):
            _check_mha_against_transformers(mod, monkeypatch)
    finally:
        del sys.modules["oracle._mutant_model"]


def test_mlkv_attention_reduces_to_the_decode_step_oracle():
    """MLKV-2 over four layers (owners 0 and 2): rerun the model oracle one
    layer at a time and check each layer's attention against oracle.decode_step
    on the same bf16 queries and owners' rows."""
    l, h, m_, g, D, d, d_ff, B, rd = 4, 4, 2, 1, 16, 64, 96, 3, 4
    kv_of, owner_of = oracle.map_uniform(l, h, m_, g)
    rng = np.random.default_rng(7)
    n_kv = m_ * g
    S, ctx = 12, np.array([0, 5, 9], dtype=np.int32)
    layers = []
    for n in range(l):
        owned = int((owner_of == n).sum())
        mk = lambda *shape: _bits(rng.standard_normal(shape) * 0.1)
        lw = dict(ln1_w=_bits(1 + 0.2 * rng.standard_normal(d)), ln1_b=mk(d),
                  ln2_w=_bits(1 + 0.2 * rng.standard_normal(d)), ln2_b=mk(d),
                  w_q=mk(d, h * D), b_q=mk(h * D), w_k=None, b_k=None, w_v=None, b_v=None,
                  w_o=mk(h * D, d), b_o=mk(d), w_fc1=mk(d, d_ff), b_fc1=mk(d_ff),
                  w_fc2=mk(d_ff, d), b_fc2=mk(d))
        if owned:
            lw.update(w_k=mk(d, owned * D), b_k=mk(owned * D), w_v=mk(d, owned * D),
                      b_v=mk(owned * D))
        layers.append(lw)
    kc_bits = synth.rows_bf16(1, 1, n_kv * B, S, D, np.tile(ctx, n_kv)).reshape(n_kv, B, S, D)
    vc_bits = synth.rows_bf16(1, 2, n_kv * B, S, D, np.tile(ctx, n_kv)).reshape(n_kv, B, S, D)
    x = rng.standard_normal((B, d))
    kc, vc = om._f64(kc_bits), om._f64(vc_bits)
    for n in range(l):
        # the model oracle's layer n alone, with its queries and owners' rows exposed
        lw = layers[n]
        gw = {k: (om._f64(v) if v is not None else None) for k, v in lw.items()}
        h1 = om.to_bf16(om.layer_norm(x, gw["ln1_w"], gw["ln1_b"], 1e-5))
        q = (h1 @ gw["w_q"] + gw["b_q"]).reshape(B, h, D)
        q = om.to_bf16(np.stack([[oracle.rope_f64(q[b, i], int(ctx[b]), rd) for i in range(h)]
                                 for b in range(B)]))
        k_new = np.zeros((B, n_kv, D))
        v_new = np.zeros((B, n_kv, D))
        owned = [kv for kv in range(n_kv) if owner_of[kv] == n]
        if owned:
            k = (h1 @ gw["w_k"] + gw["b_k"]).reshape(B, len(owned), D)
            v = om.to_bf16((h1 @ gw["w_v"] + gw["b_v"]).reshape(B, len(owned), D))
            k = om.to_bf16(np.stack([[oracle.rope_f64(k[b, c], int(ctx[b]), rd)
                                      for c in range(len(owned))] for b in range(B)]))
            for c, kv in enumerate(owned):
                k_new[:, kv], v_new[:, kv] = k[:, c], v[:, c]
        # the pinned decode-step oracle restricted to layer n (a one-layer map)
        k_bits = kc_bits.copy()
        v_bits = vc_bits.copy()
        ref = oracle.decode_step(_bits(q)[None], k_bits, v_bits, _bits(k_new), _bits(v_new),
                                 kv_of[n:n + 1], np.where(owner_of == n, 0, -1).astype(np.int32),
                                 ctx)[0]
        # the model oracle, one layer, same inputs
        kc_m, vc_m = kc.copy(), vc.copy()
        x_next = om.decode_step_model(x, [lw], kv_of[n:n + 1],
                                      np.where(owner_of == n, 0, -1), kc_m, vc_m, ctx, h, D, rd)
        assert np.array_equal(kc_m, om._f64(k_bits)) and np.array_equal(vc_m, om._f64(v_bits))
        o = om.to_bf16(ref).reshape(B, h * D)
        h2 = om.to_bf16(om.layer_norm(x, gw["ln2_w"], gw["ln2_b"], 1e-5))
        mlp = om.to_bf16(om.gelu(h2 @ gw["w_fc1"] + gw["b_fc1"])) @ gw["w_fc2"] + gw["b_fc2"]
        np.testing.assert_allclose(x_next, x + o @ gw["w_o"] + gw["b_o"] + mlp, rtol=0, atol=1e-12)
        # carry the state on
        kc, vc, kc_bits, vc_bits, x = kc_m, vc_m, k_bits, v_bits, x_next

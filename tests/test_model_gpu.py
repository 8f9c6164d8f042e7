"""GPU parity of the model-level decode step (GPT-NeoX layers around the MLKV
attention, mlkv_model_decode_step) against the float64 model oracle
(oracle/model.py) in both its forms: the plain float64 form (the one pinned
against transformers' GPT-NeoX), with a bar derived from bf16 storage at the
path's rounding points (storage_error_scale), and the form that rounds to
bf16 at those same points, with a tighter regression bar.

Tolerance of the rounded form.  The attention kernels round the softmax weights to bf16 before
the value product (relative error up to 2^-8 per weight, the decode path's
documented arithmetic) where the oracle keeps them exact, so each layer's
attention output differs from the oracle's by up to about one bf16 step in
many elements; through W_o that adds a perturbation of order 2^-8 |a| to the
residual stream per layer, and over the layers these add up; the fp32
products also flip some stored bf16 values against the oracle's float64 ones.
Bars: max |diff| <= 5e-3 * max(1, max |x|) and mean |diff| <= 5e-3 * mean |x|
after the last layer; a cache row appended by layer 0
(computed from the step's input, before any attention) within one bf16 step
of the oracle's, widened where an input of its product may round either way
(layer0_row_allowance), later owners' rows within 1e-2 * max(1, max |row|).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import oracle.model as om  # noqa: E402
import synth  # noqa: E402
from gpu_util import say  # noqa: E402
from layout_ref import unpack_k, unpack_v  # noqa: E402

pytestmark = pytest.mark.gpu

mlkv = pytest.importorskip("paper_2406_09297_amd")

# Regression bars against the form with the same bf16 storage points:
# 0.5 % of max |x| and of mean |x| (measured up to 0.24 % after 12 layers).
MAX_REL = 5e-3
MEAN_REL = 5e-3
ROW_REL = 1e-2  # later owners' appended rows (see above)
# Bars against the plain float64 form, in units of the storage error scale E
# (storage_error_scale): mean |diff| <= 1.7 E (measured 0.48 - 1.02 E; the
# model counts each rounding once, and errors carried through later layers'
# layer norms add to it); max |diff| <= the largest of the N = B*d roughly
# normal deviations at that mean bar (sigma = 1.25 mean), sqrt(2 ln N) sigma:
# 8.9 E for the benchmark's 6144 (measured max 2.4 - 5.6 E there; over 1282
# random shapes, maps and batches the largest max reached 0.99 of this bar,
# its tails being somewhat heavier than normal).
PLAIN_MEAN_E = 1.7


def plain_max_bar(n: int) -> float:
    """The max |diff| bar against the plain form, in units of E, for n outputs."""
    return 1.25 * PLAIN_MEAN_E * np.sqrt(2.0 * np.log(max(n, 2)))
# rms relative error of rounding to bf16 (8 significant bits, nearest even):
# an error uniform within half a spacing, 2^-8 of the binade's base, over
# values spread log-uniformly in the binade gives 2^-8 / sqrt(8 ln 2)
RMS_BF16 = 2.0 ** -8 / np.sqrt(8.0 * np.log(2.0))


def storage_error_scale(updates) -> float:
    """Expected rms deviation of the final residual stream from the plain
    float64 form caused by bf16 storage at the path's rounding points: each
    rounding is a relative error of rms RMS_BF16 that a following matrix
    product carries into the update it feeds at the same relative size.  The attention update a of a layer sits behind five
    roundings (h1, q, k or v, the softmax weights, o), the MLP update m
    behind two (h2, the GELU output); layers add independently:
        E = RMS_BF16 * sqrt(sum_n 5 rms(a_n)^2 + 2 rms(m_n)^2)."""
    tot = sum(5.0 * float(np.mean(a * a)) + 2.0 * float(np.mean(m * m)) for a, m in updates)
    return RMS_BF16 * np.sqrt(tot)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mlkv.lib()
    yield


# A layer-norm output y = z w + b within AMBIGUOUS_REL (|y| + |w|) of a bf16
# rounding midpoint may round either way: the kernels form it in fp32, the
# oracle in float64.  fp32 puts y within a few ulps of |y|, plus the error the
# mean carries (a 768-term sum: about 10 ulps of the mean |x|, times |w| and
# the inverse standard deviation, both about 1 for the step's input); the
# bound is about four times that.
AMBIGUOUS_REL = 2.0 ** -19


def _bf16_neighbours(v: np.ndarray):
    """The bf16 values just above and below each bf16 value v (finite)."""
    bits = synth.f32_to_bf16(v.astype(np.float32)).astype(np.int64)
    pos = (bits & 0x8000) == 0  # +0 and positive values
    up = np.where(pos, bits + 1, np.where(bits == 0x8000, 1, bits - 1))
    dn = np.where(pos, np.where(bits == 0, 0x8001, bits - 1), bits + 1)
    return (synth.bf16_to_f32(up.astype(np.uint16)).astype(np.float64),
            synth.bf16_to_f32(dn.astype(np.uint16)).astype(np.float64))


def layer0_row_allowance(x0, w, cols, bias, rd, D):
    """Per (row, channel) widening of the layer-0 cache-row bar, for what the
    arithmetic before the final rounding may move.  h = bf16(LN1(x)) is a
    storage point of both forms, reached in fp32 by the kernels and in
    float64 by the oracle; an element of LN1(x) within AMBIGUOUS_REL
    (|y| + |w|) of the midpoint between two bf16 values may round to either,
    and the other choice moves the product's output c by the rounding step
    times |W[k, c]|.  The product itself sums exact bf16 products in fp32: at
    most 32 roundings inside a matrix-core step, one per k-block a wave
    chains, eight for the waves' sum and one for the bias, each at most
    u sum_k |h_k W[k, c]| (u = 2^-24), which matters only where the output
    nearly cancels.  A rotated channel takes its partner's terms too (the
    rotation mixes the pair with a unit-norm matrix).  x0 [B][d]; w the
    layer's weights; cols the product's weight columns [d][D], bias [D]."""
    scale = om._f64(w["ln1_w"])
    ln = om.layer_norm(x0.astype(np.float64), scale, om._f64(w["ln1_b"]), 1e-5)
    hb = om.to_bf16(ln)
    up, dn = _bf16_neighbours(hb)
    step = np.zeros_like(ln)
    margin = AMBIGUOUS_REL * (np.abs(ln) + np.abs(scale))
    for nb in (up, dn):
        mid = 0.5 * (hb + nb)
        near = np.isfinite(nb) & (np.abs(ln - mid) <= margin)
        step = np.maximum(step, np.where(near, np.abs(nb - hb), 0.0))
    d = cols.shape[0]
    u = 2.0 ** -24
    du = step @ np.abs(cols)  # [B][D]
    du += (32 + d // 32 + 10) * u * (np.abs(hb) @ np.abs(cols)) + u * np.abs(bias)[None, :]
    if rd:
        half = rd // 2
        pair = du.copy()
        pair[:, :half] += du[:, half:rd]
        pair[:, half:rd] += du[:, :half]
        du = pair
    return du


def _offset_view(t):
    """The same values at a 2-byte offset (not 16-byte aligned)."""
    buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=t.device)
    buf[1:].copy_(t.reshape(-1))
    return buf[1:].view(t.shape)


def _run_case(l, h, D, d_ff, m, g, B, ctx, seed, rd=16, kv_of=None, owner_of=None, label="",
              misalign_ln=False, fused=True):
    ctx = np.asarray(ctx, dtype=np.int32)
    if kv_of is None:
        kv_of, owner_of = oracle.map_uniform(l, h, m, g)
        mp = mlkv.Map.uniform(l, h, m, g)
    else:
        mp = mlkv.Map.from_tables(kv_of, owner_of)
    n_kv = len(owner_of)
    owned = [int((np.asarray(owner_of) == n).sum()) for n in range(l)]
    weights = synth.model_weights(seed, l, h, D, d_ff, owned)
    dev = [{k: (None if v is None else mlkv.bf16_tensor(v, "cuda")) for k, v in lw.items()}
           for lw in weights]
    if misalign_ln:
        for lw in dev:
            for k in ("ln1_w", "ln1_b", "ln2_w", "ln2_b"):
                lw[k] = _offset_view(lw[k])
    d = h * D
    model = mlkv.Model(mp, d, d_ff, D, dev, rotary_dims=rd)
    assert model.fused_path(B) == fused, f"{label}: fused path expected {fused}"
    S = (int(ctx.max()) + 1 + 63) // 64 * 64
    lens = np.tile(ctx, n_kv)
    kc = synth.rows_bf16(seed, 1, n_kv * B, S, D, lens, fill=synth.BF16_NAN).reshape(n_kv, B, S, D)
    vc = synth.rows_bf16(seed, 2, n_kv * B, S, D, lens, fill=synth.BF16_NAN).reshape(n_kv, B, S, D)
    cache = mlkv.Cache.empty(n_kv, B, S, D)
    cache.load_rows(kc, vc)
    x_bits = synth.normal_bf16(seed, 0, (B, d))
    x0 = synth.bf16_to_f32(x_bits)
    x = torch.from_numpy(x0.copy()).cuda()
    ctx_dev = torch.from_numpy(ctx).cuda()
    ws = model.workspace(B, S)
    say(f"model step {label}")
    model.decode_step(x, cache, ctx_dev, ws)
    torch.cuda.synchronize()
    out = x.cpu().numpy().astype(np.float64)
    k_gpu = unpack_k(mlkv.bf16_bits(cache.k), n_kv, B, S, D)
    v_gpu = unpack_v(mlkv.bf16_bits(cache.v), n_kv, B, S, D)
    kr, vr = om._f64(kc), om._f64(vc)
    ref = om.decode_step_model(x0.astype(np.float64), weights, kv_of, owner_of, kr, vr, ctx, h, D,
                               rd)
    # The plain float64 form (no bf16 storage; the form pinned against
    # transformers' GPT-NeoX), with the storage error scale of this run.
    updates = []
    plain = om.decode_step_model(x0.astype(np.float64), weights, kv_of, owner_of, om._f64(kc),
                                 om._f64(vc), ctx, h, D, rd, round_bf16=False, updates=updates)
    E = storage_error_scale(updates)
    diff = np.abs(out - ref)
    scale = max(1.0, float(np.abs(ref).max()))
    mean_x = float(np.abs(ref).mean())
    dp = np.abs(out - plain)
    say(f"  {label}: vs rounded form max|d|={diff.max():.3e} ({diff.max() / scale:.2e} of max|x|) "
        f"mean|d|={diff.mean():.3e} ({diff.mean() / mean_x:.2e} of mean|x|); "
        f"vs plain form max|d|={dp.max():.3e} ({dp.max() / E:.2f} E) mean|d|={dp.mean():.3e} "
        f"({dp.mean() / E:.2f} E), E={E:.3e}; max|x|={np.abs(ref).max():.3f} mean|x|={mean_x:.3f}")
    assert np.all(np.isfinite(out))
    assert dp.mean() <= PLAIN_MEAN_E * E and dp.max() <= plain_max_bar(dp.size) * E, \
        f"{label}: vs plain form"
    assert diff.max() <= MAX_REL * scale and diff.mean() <= MEAN_REL * mean_x, label
    # cache: untouched slots bit-exact.  The rows appended by layer 0 come
    # from the step's input x: within one bf16 step of the oracle's, plus
    # what an input of their product rounding the other way can move.  Later
    # owners' rows come from a residual stream already carrying the earlier
    # layers' attention error: within the output bar.
    appended = np.zeros((n_kv, B, S), dtype=bool)
    for kv in range(n_kv):
        appended[kv, np.arange(B), ctx] = True
    first = np.asarray(owner_of) == 0
    own0 = [kv for kv in range(n_kv) if first[kv]]
    for name, got, orig, r in (("w_k", k_gpu, kc, kr), ("w_v", v_gpu, vc, vr)):
        assert np.array_equal(got[~appended], orig[~appended]), f"{label}: untouched slots changed"
        for kv in range(n_kv):
            g64 = om._f64(got[kv, np.arange(B), ctx])
            rr = r[kv, np.arange(B), ctx]
            if first[kv]:
                j = own0.index(kv)
                cols = om._f64(weights[0][name])[:, j * D:(j + 1) * D]
                bias = om._f64(weights[0]["b" + name[1:]])[j * D:(j + 1) * D]
                allow = layer0_row_allowance(x0, weights[0], cols, bias,
                                             rd if name == "w_k" else 0, D)
                assert np.all(np.abs(g64 - rr) <= np.abs(rr) * 2.0 ** -7 + 2.0 * allow + 1e-30), \
                    f"{label}: layer-0 row of KV head {kv} off by more than one bf16 step"
                # Most values are bit-exact; an input rounding the other way
                # changes about a fifth of its row, a systematic rounding
                # error (truncation for nearest) about half of them.
                assert np.mean(g64 != rr) <= 0.25, f"{label}: too many layer-0 values differ"
            else:
                assert np.abs(g64 - rr).max() <= ROW_REL * max(1.0, float(np.abs(rr).max())), \
                    f"{label}: row of KV head {kv} outside the bar"
    return diff.max() / scale, diff.mean()


def test_model_step_pythia160m_shape_mlkv4():
    """Pythia-160M layer shapes (12 layers, 12 heads of 64, d_ff 3072, rotary
    on 16 channels) with MLKV-4 (owners 0, 3, 6, 9): ragged contexts."""
    _run_case(12, 12, 64, 3072, 4, 1, B=4, ctx=[0, 33, 100, 257], seed=91, label="pythia MLKV-4")


@pytest.mark.parametrize("m,g", [(4, 12), (1, 1), (2, 3)])
def test_model_step_maps(m, g):
    """Plain multi-head attention (every layer owns its 12 heads), MLKV-1 (one
    KV head for the whole model) and a grouped map (3 KV heads per owning layer)."""
    _run_case(4, 12, 64, 512, m, g, B=3, ctx=[5, 64, 130], seed=92, label=f"m{m} g{g}")


def test_model_step_head_dim_128_and_full_rotation():
    _run_case(2, 4, 128, 640, 2, 2, B=2, ctx=[31, 96], seed=93, rd=128, label="D128 rd128")


def test_model_step_full_size_benchmark_configuration():
    """The whole-model benchmark's configuration: Pythia-160M shapes, MLKV-4,
    batch 8, 2000 cached tokens per sequence (capacity 2048)."""
    _run_case(12, 12, 64, 3072, 4, 1, B=8, ctx=[2000] * 8, seed=90, label="model_b8 full size")


def test_model_step_library_gemm_path(monkeypatch):
    """The library-GEMM path (forced here; taken by itself when d_ff is not a
    multiple of 32 or the layer-norm vectors are not 16-byte aligned) against
    the same oracle."""
    monkeypatch.setenv("MLKV_MODEL_GEMM", "library")
    _run_case(12, 12, 64, 3072, 4, 1, B=4, ctx=[0, 33, 100, 257], seed=91, label="library MLKV-4",
              fused=False)
    _run_case(2, 4, 128, 640, 2, 2, B=2, ctx=[31, 96], seed=93, rd=128, label="library D128",
              fused=False)


def test_model_step_batch_tiles_ragged():
    """Fused path over two 16-row batch tiles, the second with 4 rows."""
    ctx = [int(c) for c in np.random.default_rng(96).integers(0, 200, 20)]
    _run_case(3, 4, 64, 256, 3, 2, B=20, ctx=ctx, seed=96, label="B20")


def test_model_step_mlp_product_beside_attention_with_offset_k_blocks():
    """Six heads of 64 (h D / 32 = 12 k-blocks of W_o): the MLP's second
    product, carried by the attention launch, starts its k-blocks in the
    middle of the eight-wave round, over two batch tiles."""
    ctx = [int(c) for c in np.random.default_rng(95).integers(0, 300, 19)]
    _run_case(3, 6, 64, 384, 3, 1, B=19, ctx=ctx, seed=95, label="h6 B19")


@pytest.mark.parametrize("B", [65, 130, 256])
def test_model_step_serving_batches_on_the_fused_kernels(B):
    """Batches above 64 rows (five, nine and sixteen 16-row tiles, the last
    two ragged) run on the fused kernels too: no library GEMM."""
    ctx = [int(c) for c in np.random.default_rng(97 + B).integers(0, 90, B)]
    _run_case(2, 4, 64, 256, 2, 1, B=B, ctx=ctx, seed=97, label=f"B{B}", fused=True)


def test_model_step_re_reading_layers_on_a_workgroup_per_unit():
    """MLKV-2 at 100 sequences: the layers that re-read the owner's KV heads
    (1 and 3) run one eight-wave attention workgroup per (sequence, KV head)
    inside the model step, the owning layers split runs on a recorded plan."""
    ctx = [int(c) for c in np.random.default_rng(101).integers(0, 120, 100)]
    mp = mlkv.Map.uniform(4, 4, 2, 1)
    S = (max(ctx) + 1 + 63) // 64 * 64
    assert mp.plan(1, 100, S, 64, S)[0] == 100 and mp.plan(0, 100, S, 64, S)[0] > 100
    _run_case(4, 4, 64, 256, 2, 1, B=100, ctx=ctx, seed=102, label="B100 MLKV-2", fused=True)


def test_model_step_ragged_ff_takes_the_library_path():
    """d_ff = 400 (not a multiple of 32, so no packed weights): library GEMMs."""
    _run_case(2, 4, 64, 400, 1, 1, B=3, ctx=[3, 40, 77], seed=98, label="ff400", fused=False)


def test_model_step_unaligned_layer_norm_vectors_take_the_library_path():
    """The fused kernels read the layer-norm vectors 16 bytes at a time; a
    model whose vectors are not 16-byte aligned keeps no packed weights and
    runs on library GEMMs."""
    _run_case(2, 4, 64, 256, 2, 1, B=3, ctx=[3, 40, 77], seed=99, label="unaligned ln",
              misalign_ln=True, fused=False)


def test_model_step_general_map_owner_not_reading_its_head():
    """Layer 0 owns KV heads 0 and 1 but reads only head 0 (its append runs
    separately); layer 1 reads head 1."""
    kv_of = np.array([[0] * 4, [1] * 4, [0] * 4, [1] * 4], np.int32)
    owner_of = np.array([0, 0], np.int32)
    _run_case(4, 4, 64, 384, None, None, B=2, ctx=[7, 70], seed=94, kv_of=kv_of,
              owner_of=owner_of, label="general map")


def test_model_rejects_missing_or_extra_key_weights():
    mp = mlkv.Map.uniform(2, 4, 1, 1)  # layer 0 owns the KV head, layer 1 none
    weights = synth.model_weights(95, 2, 4, 64, 256, [1, 0])
    dev = [{k: (None if v is None else mlkv.bf16_tensor(v, "cuda")) for k, v in lw.items()}
           for lw in weights]
    bad = [dict(dev[0]), dict(dev[1])]
    bad[1]["w_k"] = dev[0]["w_k"]  # a non-owner with key weights
    with pytest.raises(mlkv.MLKVError):
        mlkv.Model(mp, 256, 256, 64, bad)
    bad = [dict(dev[0]), dict(dev[1])]
    bad[0]["w_v"] = None  # the owner without value weights
    with pytest.raises(mlkv.MLKVError):
        mlkv.Model(mp, 256, 256, 64, bad)


@pytest.mark.parametrize("mg", [(4, 1), (12, 12)])
def test_model_step_captured_in_a_hip_graph_replays_like_eager(mg):
    """The benchmark replays a captured model step (torch's graph capture on
    the library's stream, rocBLAS included).  Every replay, with eager steps
    between replays, must give the eager step's residual stream and cache
    rows bit for bit."""
    m, g = mg
    w = synth.get_workload("model_b8").with_map(m, g).scaled(B=4, ctx=300)
    say(f"model graph {w.name}: building")
    mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
    _, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
    owned = [int((owner_of == n).sum()) for n in range(w.l)]
    weights = synth.model_weights(w.seed, w.l, w.h, w.D, w.d_ff, owned)
    dev = [{k: (None if v is None else mlkv.bf16_tensor(v, "cuda")) for k, v in lw.items()}
           for lw in weights]
    d = w.h * w.D
    model = mlkv.Model(mp, d, w.d_ff, w.D, dev, rotary_dims=16)
    inp = synth.step_inputs(w, fill=0)
    S = inp["capacity"]
    cache = mlkv.Cache.empty(w.n_kv, w.B, S, w.D)
    cache.load_rows(inp["k_cache"], inp["v_cache"])
    k0, v0 = cache.k.clone(), cache.v.clone()
    x0 = torch.from_numpy(synth.bf16_to_f32(synth.normal_bf16(w.seed, 0, (w.B, d))).copy()).cuda()
    x = x0.clone()
    ctx = torch.from_numpy(inp["ctx"]).cuda()
    ws = model.workspace(w.B, S)

    def step():
        model.decode_step(x, cache, ctx, ws)

    step()  # first call outside capture (library and rocBLAS set-up)
    torch.cuda.synchronize()

    def reset():
        x.copy_(x0)
        cache.k.copy_(k0)
        cache.v.copy_(v0)
        torch.cuda.synchronize()

    reset()
    step()
    torch.cuda.synchronize()
    x_ref, k_ref, v_ref = x.clone(), cache.k.clone(), cache.v.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    reset()
    say(f"model graph {w.name}: capturing")
    with torch.cuda.graph(graph, stream=side):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        reset()
        say(f"model graph {w.name}: replay {rep}")
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(x, x_ref), f"replay {rep}: residual stream differs"
        assert torch.equal(cache.k, k_ref) and torch.equal(cache.v, v_ref), f"replay {rep}: cache"
        step()  # eager work between replays
        torch.cuda.synchronize()

"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Cache writes are compared bit for bit; attention outputs within the
tolerances stated in gpu_util.  Every case prints its name before touching the
GPU so that a failure names it.
"""
import contextlib
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from gpu_util import (BOUND_MAX_POSITIONS, DeviceWorkload, check_close, f64,  # noqa: E402
                      layer_rounding_bound, say, step_rounding_bound)
from layout_ref import unpack_k, unpack_v  # noqa: E402

pytestmark = pytest.mark.gpu

mlkv = pytest.importorskip("paper_2406_09297_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mlkv.lib()
    yield


def small(name, **kw):
    return synth.get_workload(name).scaled(**kw)


@contextlib.contextmanager
def plan_env(workgroups="", merge="", wide=""):
    """Launch-plan overrides read by the library on every call:
    MLKV_WORKGROUPS (workgroup budget), MLKV_COMBINE=kernel/fused (merge
    split runs in a separate kernel / in place even at a cost in
    workgroups), MLKV_WIDE=0/1 (one run per unit on a wide
    workgroup: in no layer / in every layer; unset: in the layers that
    re-read KV heads, when there are enough units)."""
    names = {"MLKV_WORKGROUPS": workgroups, "MLKV_COMBINE": merge, "MLKV_WIDE": wide}
    for k, v in names.items():
        if v:
            os.environ[k] = v
        else:
            os.environ.pop(k, None)
    try:
        yield
    finally:
        for k in names:
            os.environ.pop(k, None)


# ------------------------------------------------------------------ append --

@pytest.mark.parametrize("wname,kw", [
    ("mlkv4_b128_ragged", dict(B=5, ctx=300)),
    ("7b_mlkv8x8", dict(B=3, ctx=100)),
    ("sweep_b32", dict(B=2, ctx=70)),
])
def test_append_bit_exact(wname, kw):
    w = small(wname, **kw)
    say(f"append {w.name} B={w.B} D={w.D} n_kv={w.n_kv}")
    dw = DeviceWorkload(w, fill=synth.BF16_NAN)
    k_ref, v_ref = dw.host["k_cache"].copy(), dw.host["v_cache"].copy()
    pos = dw.host["ctx"].copy()
    pos[0] = -1           # skipped
    if w.B > 1:
        pos[1] = dw.S     # skipped (out of range)
    pos_d = torch.from_numpy(pos).cuda()
    for layer in range(w.l):
        begin, count = dw.map.layer_owned(layer)
        if count:
            kn = dw.k_new[:, begin:begin + count].contiguous()
            vn = dw.v_new[:, begin:begin + count].contiguous()
            mlkv.cache_append(layer, dw.map, dw.cache, kn, vn, pos_d)
        oracle.append(layer, k_ref, v_ref, dw.host["k_new"], dw.host["v_new"], dw.owner_of, pos)
    k_gpu, v_gpu = dw.read_cache()
    assert np.array_equal(k_gpu, k_ref)
    assert np.array_equal(v_gpu, v_ref)


@pytest.mark.parametrize("n_kv,B,S,D", [(3, 2, 96, 64), (2, 3, 64, 128)])
def test_cache_rows_through_the_library(n_kv, B, S, D):
    """mlkv_cache_write_rows stores plain row-major rows in the documented
    plane layout (checked against the tests' own statement of it), touching
    only the named KV heads; mlkv_cache_read_rows returns them unchanged."""
    import layout_ref

    say(f"cache rows n_kv={n_kv} B={B} S={S} D={D}")
    rng = np.random.default_rng(n_kv * 1000 + D)
    rows_k = rng.integers(0, 0x7F00, size=(n_kv, B, S, D), dtype=np.uint16)
    rows_v = rng.integers(0, 0x7F00, size=(n_kv, B, S, D), dtype=np.uint16)
    cache = mlkv.Cache.empty(n_kv, B, S, D)
    cache.k.fill_(float("nan"))
    cache.v.fill_(float("nan"))
    lo = 1  # heads 1.. written; head 0 stays as filled
    cache.write_rows(mlkv.bf16_tensor(rows_k[lo:], "cuda"), mlkv.bf16_tensor(rows_v[lo:], "cuda"), lo)
    torch.cuda.synchronize()
    k_plane = mlkv.bf16_bits(cache.k).reshape(n_kv, B, S, D)
    v_plane = mlkv.bf16_bits(cache.v).reshape(n_kv, B, S // 32, D, 32)
    nan = mlkv.bf16_bits(torch.tensor([float("nan")], dtype=torch.bfloat16))[0]
    assert np.all(k_plane[:lo] == nan) and np.all(v_plane[:lo] == nan), "other heads written"
    assert np.array_equal(k_plane[lo:], layout_ref.pack_k(rows_k[lo:]))
    assert np.array_equal(v_plane[lo:], layout_ref.pack_v(rows_v[lo:]))
    k_back, v_back = cache.read_rows(lo)
    torch.cuda.synchronize()
    assert np.array_equal(mlkv.bf16_bits(k_back), rows_k[lo:])
    assert np.array_equal(mlkv.bf16_bits(v_back), rows_v[lo:])


# ----------------------------------------------------------- one layer ------

@pytest.mark.parametrize("wname,kw,layers", [
    ("mlkv2_b1", {}, [0, 5, 6, 11]),
    ("mlkv4_b128_ragged", dict(B=16, ctx=700), [0, 1, 4]),
    ("mlkv4_b8_long", dict(B=2, ctx=3000), [0, 7]),
    ("7b_mlkv8x8", dict(B=4, ctx=600), [0, 3, 29]),
])
def test_decode_attention_matches_oracle(wname, kw, layers):
    w = small(wname, **kw)
    dw = DeviceWorkload(w)
    lens = dw.host["ctx"].copy()
    lens_d = torch.from_numpy(lens).cuda()
    for n in layers:
        say(f"decode_attention {w.name} layer={n} B={w.B} D={w.D} G={w.h // w.g}")
        out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
        mlkv.decode_attention(n, dw.q[n], dw.cache, dw.map, lens_d, out, ws=dw.ws)
        torch.cuda.synchronize()
        ref = oracle.decode_attention(n, dw.host["q"][n], dw.host["k_cache"], dw.host["v_cache"],
                                      dw.kv_of, lens)
        check_close(out.cpu().numpy(), ref, f"{w.name} L{n}",
                    bound=_layer_bound(dw, n, dw.host["k_cache"], lens, ref))


def _layer_bound(dw, n, k_cache, lens, ref):
    """Rounding bound of layer n's outputs (None for rows too long for it)."""
    if int(np.max(lens, initial=0)) > BOUND_MAX_POSITIONS:
        return None
    return layer_rounding_bound(dw.host["q"][n], k_cache, dw.host["v_cache"], dw.kv_of[n], lens,
                                ref)


def _sweep_workload(D, m, g, lens, h=12, l=4, k_scale=1.0, seed=99):
    B = len(lens)
    w = synth.Workload("sweep", l=l, h=h, m=m, g=g, D=D, B=B, ctx=int(max(lens)), k_scale=k_scale,
                       seed=seed)
    return w


LEN_SWEEP = [1, 2, 7, 31, 32, 33, 63, 64, 65, 96, 127, 128, 129, 160, 191, 255, 256, 257, 300]


@pytest.mark.parametrize("D,m,g", [(64, 4, 1), (64, 4, 3), (128, 2, 4), (64, 2, 12)])
def test_length_sweep_across_tile_boundaries(D, m, g):
    w = _sweep_workload(D, m, g, LEN_SWEEP)
    dw = DeviceWorkload(w)
    lens = np.array(LEN_SWEEP, dtype=np.int32)
    lens_d = torch.from_numpy(lens).cuda()
    refs = {n: oracle.decode_attention(n, dw.host["q"][n], dw.host["k_cache"],
                                       dw.host["v_cache"], dw.kv_of, lens) for n in (0, w.l - 1)}
    bounds = {n: _layer_bound(dw, n, dw.host["k_cache"], lens, refs[n]) for n in refs}
    for wg, comb, wide in (("", "", ""), ("3", "", ""), ("40", "", ""), ("", "fused", ""),
                           ("40", "fused", ""), ("", "kernel", ""), ("40", "kernel", ""),
                           ("", "", "1"), ("", "", "0")):
        with plan_env(wg, comb, wide):
            for n in (0, w.l - 1):
                say(f"length sweep D={D} m={m} g={g} layer={n} workgroups={wg or 'auto'} "
                    f"merge={comb or 'kernel'} wide={wide or 'auto'}")
                out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
                mlkv.decode_attention(n, dw.q[n], dw.cache, dw.map, lens_d, out, ws=dw.ws)
                torch.cuda.synchronize()
                check_close(out.cpu().numpy(), refs[n],
                            f"sweep D{D} g{g} L{n} wg{wg} {comb} {wide}", bound=bounds[n])


@pytest.mark.parametrize("workgroups", ["", "600", "1500"])
def test_schedule_path_with_many_short_runs(workgroups):
    """The in-kernel schedule (decode_attention, and the first layer of a
    step) with short ragged sequences, so that many runs have fewer tiles
    than the workgroup has waves: waves with no tile of their own reach the
    LDS merge early while their siblings still read the schedule tables,
    which share that LDS (the schedule is read into registers and a barrier
    separates the two)."""
    rng = np.random.default_rng(31)
    lens = rng.integers(1, 130, size=300).astype(np.int32)
    lens[:4] = [1, 32, 33, 96]
    w = _sweep_workload(64, 4, 1, lens, h=12, l=4, seed=131)
    dw = DeviceWorkload(w)
    lens_d = torch.from_numpy(lens).cuda()
    with plan_env(workgroups=workgroups):
        for n in (0, 2):
            say(f"short runs workgroups={workgroups or 'auto'} layer={n}")
            out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
            mlkv.decode_attention(n, dw.q[n], dw.cache, dw.map, lens_d, out, ws=dw.ws)
            torch.cuda.synchronize()
            ref = oracle.decode_attention(n, dw.host["q"][n], dw.host["k_cache"],
                                          dw.host["v_cache"], dw.kv_of, lens)
            check_close(out.cpu().numpy(), ref, f"short runs wg{workgroups} L{n}",
                        bound=_layer_bound(dw, n, dw.host["k_cache"], lens, ref))
        say(f"short runs workgroups={workgroups or 'auto'}: step")
        _with_contexts(dw, lens - 1)
        out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, f"short runs step wg{workgroups}")


def test_schedule_path_at_the_table_limit():
    """The in-kernel schedule at its table size: 2048 sequences, eight per
    thread, under a workgroup budget of 4096, so the per-thread loops, the
    packed run-count scans (about 3700 runs) and the run lookup across
    thread slices all run, with units split into up to three runs merged in
    place; ragged lengths (0..400 positions, a few sequences attending
    nothing), then a whole step (its first layer records the plan, the
    others follow it)."""
    rng = np.random.default_rng(37)
    lens = rng.integers(0, 401, size=2048).astype(np.int32)
    lens[:4] = [0, 1, 400, 33]
    lens[-3:] = [0, 32, 64]
    w = _sweep_workload(64, 4, 1, np.maximum(lens, 1), h=12, l=4, seed=137)
    dw = DeviceWorkload(w)
    lens_d = torch.from_numpy(lens).cuda()
    with plan_env(workgroups="4096"):
        assert dw.map.plan(0, w.B, dw.S, w.D, int(lens.max()))[0] == 4096  # > units: scheduled
        # The default plan gives each of the 2048 units its own workgroup and
        # needs no workspace; this budget's plan does.
        dw.ws = mlkv.workspace(dw.map, w.B, dw.S, w.D)
        for n in (0, 1):
            say(f"table limit B={w.B} layer={n}")
            out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
            mlkv.decode_attention(n, dw.q[n], dw.cache, dw.map, lens_d, out, ws=dw.ws)
            torch.cuda.synchronize()
            ref = oracle.decode_attention(n, dw.host["q"][n], dw.host["k_cache"],
                                          dw.host["v_cache"], dw.kv_of, lens)
            got = out.cpu().numpy()
            assert np.all(got[lens == 0] == 0.0), "sequences attending nothing must be zero"
            check_close(got, ref, f"table limit L{n}",
                        bound=_layer_bound(dw, n, dw.host["k_cache"], lens, ref))
        say("table limit: step")
        _with_contexts(dw, np.maximum(lens, 1) - 1)
        out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, "table limit step")


def test_split_count_invariance_and_determinism():
    """Results do not depend on how many workgroups share the tiles (up to
    rounding), and a repeated call is bitwise identical."""
    w = small("mlkv4_b8_long", B=2, ctx=5000)
    dw = DeviceWorkload(w)
    lens_d = torch.from_numpy(dw.host["ctx"]).cuda()
    outs = {}
    for wg, comb, wide in (("1", "", ""), ("7", "", ""), ("64", "", ""), ("300", "", ""),
                           ("", "", ""), ("", "fused", ""), ("300", "fused", ""),
                           ("", "kernel", ""), ("300", "kernel", ""), ("", "", "1")):
        with plan_env(wg, comb, wide):
            say(f"workgroup invariance workgroups={wg or 'auto'} merge={comb or 'kernel'} "
                f"wide={wide or 'auto'}")
            o = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
            mlkv.decode_attention(2, dw.q[2], dw.cache, dw.map, lens_d, o, ws=dw.ws)
            o2 = torch.empty_like(o)
            mlkv.decode_attention(2, dw.q[2], dw.cache, dw.map, lens_d, o2, ws=dw.ws)
            torch.cuda.synchronize()
            assert torch.equal(o, o2), "run-to-run results differ"
            outs[wg + comb + wide] = o.cpu().numpy().astype(np.float64)
    ref = oracle.decode_attention(2, dw.host["q"][2], dw.host["k_cache"], dw.host["v_cache"],
                                  dw.kv_of, dw.host["ctx"])
    for k, o in outs.items():
        check_close(o, ref, f"workgroups {k or 'auto'}")


def test_single_position_and_empty():
    """L = 1 returns v exactly (one weight of exactly 1); L = 0 returns zeros."""
    w = _sweep_workload(64, 2, 3, [1, 0, 1, 0], h=6, l=2)
    dw = DeviceWorkload(w)
    lens = np.array([1, 0, 1, 0], np.int32)
    say("single position / empty")
    out = torch.full((w.B, w.h, w.D), 7.0, dtype=torch.float32, device="cuda")
    mlkv.decode_attention(1, dw.q[1], dw.cache, dw.map, torch.from_numpy(lens).cuda(), out,
                          ws=dw.ws)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    for b in range(w.B):
        for i in range(w.h):
            kv = dw.kv_of[1, i]
            if lens[b] == 1:
                assert np.array_equal(out[b, i], f64(dw.host["v_cache"][kv, b, 0]).astype(np.float32))
            else:
                assert np.all(out[b, i] == 0)


def test_non_finite_inputs_propagate_as_in_the_definition():
    """A NaN key inside the attended range makes every output of the heads
    reading it NaN, and an infinite value makes their outputs in that
    channel infinite, as Eq. 3 evaluated in IEEE arithmetic (the oracle)
    gives; only a row that attends nothing (zero weight sum) is zero.
    Every plan: one run per unit, split runs merged in place or by the
    merge kernel, a wide workgroup per unit."""
    lens = np.array([300, 300, 300, 0, 70], np.int32)
    w = _sweep_workload(64, 4, 1, lens, h=12, l=4, seed=61)
    dw = DeviceWorkload(w)
    kc, vc = dw.host["k_cache"], dw.host["v_cache"]
    kc[0, 1, 131] = synth.BF16_NAN      # sequence 1: a NaN key (KV head 0)
    vc[0, 2, 40, 5] = 0x7F80            # sequence 2: +inf in channel 5 of one value
    kc[0, 4, 200] = synth.BF16_NAN      # sequence 4: past its length, never read
    dw.cache.load_rows(kc, vc)
    lens_d = torch.from_numpy(lens).cuda()
    ref = oracle.decode_attention(0, dw.host["q"][0], kc, vc, dw.kv_of, lens)
    assert np.all(np.isnan(ref[1])) and np.all(np.isposinf(ref[2][:, 5]))
    clean = [0, 2, 3, 4]  # sequence 2 without its channel 5
    with np.errstate(invalid="ignore"):
        bound = layer_rounding_bound(dw.host["q"][0][clean], kc[:, clean], vc[:, clean],
                                     dw.kv_of[0], lens[clean], ref[clean])
    keep = np.ones(ref[clean].shape, bool)
    keep[1, :, 5] = False
    for wg, comb, wide in (("", "", ""), ("40", "fused", ""), ("40", "kernel", ""), ("", "", "1")):
        with plan_env(wg, comb, wide):
            say(f"non-finite inputs workgroups={wg or 'auto'} merge={comb or 'auto'} "
                f"wide={wide or 'auto'}")
            out = torch.full((w.B, w.h, w.D), 7.0, dtype=torch.float32, device="cuda")
            mlkv.decode_attention(0, dw.q[0], dw.cache, dw.map, lens_d, out, ws=dw.ws)
            torch.cuda.synchronize()
        got = out.cpu().numpy()
        assert np.all(np.isnan(got[1])), "a NaN key must make its rows NaN"
        assert np.all(np.isposinf(got[2][:, 5])), "an infinite value must give +inf"
        check_close(got[clean][keep], ref[clean][keep], "non-finite: the finite outputs",
                    bound=bound[keep])


@pytest.mark.parametrize("pos_kind", ["first", "tile_end", "tile_start", "split_edge", "last"])
def test_needle_token(pos_kind):
    """A key aligned with q and scaled up takes (almost) all weight: o = v_needle
    to bf16 weight precision.  Catches dropped or duplicated tokens."""
    L = 1200
    w = _sweep_workload(64, 1, 1, [L, L], h=12, l=1, seed=123)
    dw = DeviceWorkload(w)
    pos = {"first": 0, "tile_end": 31, "tile_start": 32, "split_edge": 511, "last": L - 1}[pos_kind]
    b, head = 1, 7
    q = dw.host["q"][0, b, head]
    kc = dw.host["k_cache"]
    kc[0, b, pos] = synth.f32_to_bf16(synth.bf16_to_f32(q) * 4.0)
    dw.cache.load_rows(kc, dw.host["v_cache"])
    with plan_env(workgroups="5"):
        say(f"needle at {pos} ({pos_kind})")
        out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
        lens = np.array([L, L], np.int32)
        mlkv.decode_attention(0, dw.q[0], dw.cache, dw.map, torch.from_numpy(lens).cuda(), out,
                              ws=dw.ws)
        torch.cuda.synchronize()
    ref = oracle.decode_attention(0, dw.host["q"][0], kc, dw.host["v_cache"], dw.kv_of, lens)
    _, alpha = oracle.attend_one(q, kc[0, b, :L], dw.host["v_cache"][0, b, :L])
    assert alpha[pos] > 0.99
    check_close(out.cpu().numpy(), ref, f"needle {pos_kind}",
                bound=_layer_bound(dw, 0, kc, lens, ref))


def test_bf16_output_is_the_rounded_fp32_result():
    """bf16 output mode returns exactly the RNE rounding of the fp32 result of the
    same (deterministic) computation, and stays within the tolerances of the
    oracle once its own rounding (half a bf16 ulp) is allowed for."""
    w = small("mlkv4_b128_ragged", B=8, ctx=900)
    dw = DeviceWorkload(w)
    lens = torch.from_numpy(dw.host["ctx"]).cuda()
    say("bf16 output")
    out16 = torch.empty((w.B, w.h, w.D), dtype=torch.bfloat16, device="cuda")
    out32 = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    mlkv.decode_attention(3, dw.q[3], dw.cache, dw.map, lens, out16, ws=dw.ws)
    mlkv.decode_attention(3, dw.q[3], dw.cache, dw.map, lens, out32, ws=dw.ws)
    torch.cuda.synchronize()
    bits = mlkv.bf16_bits(out16)
    assert np.array_equal(bits, synth.f32_to_bf16(out32.cpu().numpy()))
    ref = oracle.decode_attention(3, dw.host["q"][3], dw.host["k_cache"], dw.host["v_cache"],
                                  dw.kv_of, dw.host["ctx"])
    got = f64(bits)
    d = np.abs(got - ref)
    assert np.all(d <= 1e-2 + np.abs(ref) * 2.0**-8), d.max()
    assert d.mean() <= 1e-3


# -------------------------------------------------------------- whole step --

def _run_step(dw, out_dtype=torch.float32):
    w = dw.w
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=out_dtype, device="cuda")
    mlkv.decode_step(dw.q, dw.k_new, dw.v_new, dw.cache, dw.map, dw.ctx, out, ws=dw.ws)
    torch.cuda.synchronize()
    return out


def _oracle_step(dw):
    k, v = dw.host["k_cache"].copy(), dw.host["v_cache"].copy()
    out = oracle.decode_step(dw.host["q"], k, v, dw.host["k_new"], dw.host["v_new"], dw.kv_of,
                             dw.owner_of, dw.host["ctx"])
    return out, k, v


def _check_step(dw, out, ref, k_ref, v_ref, tag):
    """A step's outputs against the oracle's, each within its rounding bound
    (computed from the caches after the step) where the rows are short enough
    for it to be tight."""
    ctx = dw.host["ctx"]
    bound = None
    if int(ctx.max(initial=0)) + 1 <= BOUND_MAX_POSITIONS:
        bound = step_rounding_bound(dw.host["q"], k_ref, v_ref, dw.kv_of, ctx, ref)
    check_close(out, ref, tag, bound=bound)


def test_step_mlkv2_empty_context_outputs_new_value_exactly():
    w = synth.Workload("mlkv2_ctx0", l=12, h=12, m=2, g=1, D=64, B=3, ctx=0, seed=5)
    dw = DeviceWorkload(w)
    say("step MLKV-2 ctx=0")
    out = _run_step(dw).cpu().numpy()
    for n in range(12):
        for b in range(3):
            for i in range(12):
                assert np.array_equal(out[n, b, i],
                                      f64(dw.host["v_new"][b, n // 6]).astype(np.float32))


@pytest.mark.parametrize("wname,wide", [("mlkv2_b1", ""), ("mlkv4_b128_ragged", ""),
                                        ("mlkv4_b128_ragged", "1"), ("mlkv4_b128_ragged", "0"),
                                        ("mlkv4_b8_long", "")])
def test_full_size_step_matches_oracle(wname, wide):
    """Full-size workloads in the launch configuration the benchmark times
    (and the ragged batch also with one wide workgroup per sequence in every
    layer, and with split runs in every layer)."""
    w = synth.get_workload(wname)
    say(f"full step {wname} wide={wide or 'auto'}: uploading")
    dw = DeviceWorkload(w)
    say(f"full step {wname}: running")
    with plan_env(wide=wide):
        out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    say(f"full step {wname}: oracle")
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, f"step {wname}")


@pytest.mark.parametrize("mg", [(12, 12), (12, 4), (12, 1), (6, 1), (4, 1), (1, 1)])
def test_map_sweep_full_size(mg):
    w = synth.get_workload("sweep_b32").with_map(*mg)
    say(f"sweep step {w.name}: uploading")
    dw = DeviceWorkload(w)
    say(f"sweep step {w.name}: running")
    out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    say(f"sweep step {w.name}: oracle")
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, f"step {w.name}")


@pytest.mark.parametrize("merge", ["", "kernel"])
def test_full_size_step_twice_on_one_workspace(merge):
    """The ragged 128-sequence step, run twice on one workspace (the in-place
    merge's arrival counters must return to zero), with the default merge
    (in place where it fits) and with the separate merge kernel."""
    w = synth.get_workload("mlkv4_b128_ragged")
    with plan_env(merge=merge):
        say(f"full step twice merge={merge or 'auto'}: uploading")
        dw = DeviceWorkload(w)
        say("full step twice: running")
        _run_step(dw)
        dw2 = DeviceWorkload(w)  # fresh cache, same workspace
        dw2.ws = dw.ws
        out = _run_step(dw2).cpu().numpy()
    k_gpu, v_gpu = dw2.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw2)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw2, out, ref, k_ref, v_ref, f"step twice merge={merge or 'auto'}")


def test_one_workspace_shared_by_steps_of_different_batches():
    """A workspace sized for the largest of several steps serves them in
    turn: a large batch, a smaller one with another map, then the large one
    again.  The arrival counters keep one place in every call's layout, so
    the smaller step's run list and partials never land where the larger
    step's counters are (each step is checked against the oracle)."""
    big = synth.Workload("ws_big", l=12, h=12, m=4, g=1, D=64, B=96, ctx_range=(200, 2000),
                         seed=0x5C1)
    small = synth.Workload("ws_small", l=4, h=12, m=2, g=3, D=64, B=9, ctx_range=(1, 300),
                           seed=0x5C2)
    need = 0
    for w in (big, small):
        mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
        need = max(need, mp.workspace_bytes(w.B, w.ctx_range[1] + 64, w.D))
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    mlkv.lib().mlkv_workspace_init(ws.data_ptr(), need, torch.cuda.current_stream().cuda_stream)
    for w in (big, small, big):
        say(f"shared workspace {w.name} B={w.B}")
        dw = DeviceWorkload(w)
        dw.ws = ws
        out = _run_step(dw).cpu().numpy()
        k_gpu, v_gpu = dw.read_cache()
        ref, k_ref, v_ref = _oracle_step(dw)
        assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
        _check_step(dw, out, ref, k_ref, v_ref, f"shared workspace {w.name}")


# ---------------------------------------------------- fused append in step --

def _with_contexts(dw, ctx):
    """Give a device workload explicit per-sequence contexts: slots at or past
    each context are NaN-poisoned again on host and device."""
    ctx = np.asarray(ctx, dtype=np.int32)
    assert ctx.size == dw.w.B and ctx.max() < dw.S
    for arr in (dw.host["k_cache"], dw.host["v_cache"]):
        for b, c in enumerate(ctx):
            arr[:, b, max(c, 0):] = synth.BF16_NAN
    dw.host["ctx"] = ctx
    dw.ctx = torch.from_numpy(ctx).cuda()
    dw.cache.load_rows(dw.host["k_cache"], dw.host["v_cache"])
    return dw


APPEND_CTX = [0, 1, 30, 31, 32, 33, 63, 64, 95, 96, 127, 128, 200, 254, 255]


@pytest.mark.parametrize("D,m,g,workgroups,wide", [
    (64, 4, 1, "", ""), (64, 4, 1, "7", ""), (64, 4, 1, "", "1"),
    (64, 4, 3, "40", ""), (128, 2, 4, "", ""), (128, 2, 4, "", "1"), (128, 2, 4, "7", "")])
def test_step_fused_append_across_tile_boundaries(D, m, g, workgroups, wide):
    """The owning layers append inside their attention launch: the new token
    lands at every offset of a 32-token tile (and in the last slot of the
    cache), is attended by the owner in the same launch and by the later
    layers of its group; the whole cache matches the oracle bit for bit."""
    w = synth.Workload("append_sweep", l=4, h=12, m=m, g=g, D=D, B=len(APPEND_CTX),
                       ctx=max(APPEND_CTX), seed=77)
    dw = _with_contexts(DeviceWorkload(w), APPEND_CTX)
    assert dw.S == 256  # the last context appends into the last slot
    say(f"fused append D={D} m={m} g={g} workgroups={workgroups or 'auto'} wide={wide or 'auto'}")
    with plan_env(workgroups=workgroups, wide=wide):
        out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, f"fused append D{D} m{m} g{g} wg{workgroups} {wide}")


def test_step_mixing_split_runs_and_a_workgroup_per_unit():
    """By default a step gives the layers that only re-read KV heads (here
    layers 1 and 3 of MLKV-2) one eight-wave workgroup per (sequence, KV
    head), while the owning layers split runs on a recorded plan; the cache
    and every layer's output match the oracle, with and without rotation."""
    rng = np.random.default_rng(41)
    ctx = rng.integers(0, 400, size=100).astype(np.int32)
    ctx[:3] = [0, 31, 399]
    w = synth.Workload("mixed", l=4, h=12, m=2, g=1, D=64, B=100, ctx=int(ctx.max()), seed=141)
    dw = _with_contexts(DeviceWorkload(w), ctx)
    S = dw.S
    with plan_env():
        p0 = dw.map.plan(0, w.B, S, w.D, S)[0]
        p1 = dw.map.plan(1, w.B, S, w.D, S)[0]
        assert p0 > w.B and p1 == w.B, (p0, p1)  # layer 0 splits runs, layer 1 one per unit
        say("mixed plans: step")
        out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, "mixed plans step")
    _check_rope_step(dw, 16, "mixed plans rope")


def test_step_owner_that_does_not_read_its_head():
    """A general map where layer 0 owns KV heads 0 and 1 but reads only head 0:
    head 1 is appended by a separate launch before layer 0 attends, and layer
    1 reads it."""
    w = synth.Workload("general", l=4, h=4, m=2, g=1, D=64, B=3, ctx=100, seed=11)
    dw = DeviceWorkload(w)
    kv_of = np.array([[0] * 4, [1] * 4, [0] * 4, [1] * 4], np.int32)
    owner_of = np.array([0, 0], np.int32)
    dw.map = mlkv.Map.from_tables(kv_of, owner_of)
    dw.kv_of, dw.owner_of = kv_of, owner_of
    _with_contexts(dw, [0, 37, 100])
    say("general map: owner not reading its head")
    out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    _check_step(dw, out, ref, k_ref, v_ref, "general map")


# ------------------------------------------------------ rotary embedding --

def _check_rope_step(dw, rd, label, base=10000.0):
    """The step with rotary embedding against the oracle: the cache (rotated
    keys) matches bit for bit and the outputs within tolerance; the caller's
    queries and new keys are left unchanged, so a second call on the same
    buffers gives the same outputs and cache bit for bit."""
    w = dw.w
    ws = mlkv.workspace(dw.map, w.B, dw.S, w.D, rotary_dims=rd)
    q0, kn0 = dw.q.clone(), dw.k_new.clone()
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    mlkv.decode_step(dw.q, dw.k_new, dw.v_new, dw.cache, dw.map, dw.ctx, out, ws=ws,
                     rotary_dims=rd, rotary_base=base)
    torch.cuda.synchronize()
    assert torch.equal(dw.q, q0) and torch.equal(dw.k_new, kn0), f"{label}: inputs written"
    k_gpu, v_gpu = dw.read_cache()
    out2 = torch.full_like(out, float("nan"))
    mlkv.decode_step(dw.q, dw.k_new, dw.v_new, dw.cache, dw.map, dw.ctx, out2, ws=ws,
                     rotary_dims=rd, rotary_base=base)
    torch.cuda.synchronize()
    assert torch.equal(out, out2), f"{label}: a repeated call differs"
    k2, v2 = dw.read_cache()
    assert np.array_equal(k2, k_gpu) and np.array_equal(v2, v_gpu), f"{label}: cache changed"
    out = out.cpu().numpy()
    k, v = dw.host["k_cache"].copy(), dw.host["v_cache"].copy()
    ref, q_rot, _ = oracle.decode_step_rope(dw.host["q"], k, v, dw.host["k_new"],
                                            dw.host["v_new"], dw.kv_of, dw.owner_of,
                                            dw.host["ctx"], rd, base, return_rotated=True)
    bad = np.argwhere(k_gpu != k)
    assert bad.size == 0, f"{label}: cached (rotated) keys differ at {bad[:4].tolist()}"
    assert np.array_equal(v_gpu, v), f"{label}: cached values differ"
    ctx = dw.host["ctx"]
    bound = None
    if int(ctx.max(initial=0)) + 1 <= BOUND_MAX_POSITIONS:  # rows of the rotated queries
        bound = step_rounding_bound(q_rot, k, v, dw.kv_of, ctx, ref)
    check_close(out, ref, label, bound=bound)


@pytest.mark.parametrize("D,m,g,rd,wide", [
    (64, 4, 1, 16, ""), (64, 4, 1, 64, ""), (64, 4, 3, 32, "1"),
    (128, 2, 4, 128, ""), (128, 2, 4, 32, "1"), (128, 2, 4, 64, "")])
def test_step_rope_across_tile_boundaries(D, m, g, rd, wide):
    """Rotary embedding of the newest token inside the step: its queries are
    rotated as each layer's attention loads them and its keys as the owner
    appends them, at every offset of a 32-token tile; the cache (rotated keys)
    matches the oracle bit for bit and the outputs within tolerance."""
    w = synth.Workload("rope_sweep", l=4, h=12, m=m, g=g, D=D, B=len(APPEND_CTX),
                       ctx=max(APPEND_CTX), seed=78)
    dw = _with_contexts(DeviceWorkload(w), APPEND_CTX)
    say(f"rope step D={D} m={m} g={g} rd={rd} wide={wide or 'auto'}")
    with plan_env(wide=wide):
        _check_rope_step(dw, rd, f"rope D{D} m{m} g{g} rd{rd} {wide}")


def test_step_rope_general_map_separate_append():
    """Rotated keys through the separate append launch (an owner that does
    not read its head), with a base other than the default."""
    w = synth.Workload("general_rope", l=4, h=4, m=2, g=1, D=64, B=3, ctx=100, seed=12)
    dw = DeviceWorkload(w)
    kv_of = np.array([[0] * 4, [1] * 4, [0] * 4, [1] * 4], np.int32)
    owner_of = np.array([0, 0], np.int32)
    dw.map = mlkv.Map.from_tables(kv_of, owner_of)
    dw.kv_of, dw.owner_of = kv_of, owner_of
    _with_contexts(dw, [0, 37, 100])
    say("rope general map")
    _check_rope_step(dw, 32, "rope general map", base=500.0)


@pytest.mark.parametrize("wname,rd", [("mlkv4_b8_long", 16), ("mlkv4_b128_ragged", 16),
                                      ("mlkv4_b128_ragged", 64)])
def test_full_size_step_rope(wname, rd):
    """Full-size steps with the Pythia-160M rotary (16 of 64 channels, base
    10000) and with every channel rotated; the long contexts put the new
    token at positions near 32768."""
    w = synth.get_workload(wname)
    say(f"full rope step {wname} rd={rd}: uploading")
    dw = DeviceWorkload(w)
    say(f"full rope step {wname} rd={rd}: running")
    _check_rope_step(dw, rd, f"full rope {wname} rd{rd}")


# ------------------------------------------------------------ edge cases --

def test_step_bf16_output_is_the_rounded_fp32_step():
    """decode_step in bf16 output mode returns the RNE rounding of its fp32
    output (the append is idempotent, so the step can run twice)."""
    w = small("mlkv4_b128_ragged", B=6, ctx=700)
    dw = DeviceWorkload(w)
    say("step bf16 output")
    out32 = _run_step(dw, torch.float32)
    out16 = _run_step(dw, torch.bfloat16)
    assert np.array_equal(mlkv.bf16_bits(out16), synth.f32_to_bf16(out32.cpu().numpy()))


def test_step_sequence_with_nothing_cached_before_nothing_to_attend():
    """A context of -1 (no token, nothing to append: L = 0) gives zero output
    in every layer and leaves the cache untouched; the other sequences of the
    batch are unaffected."""
    w = synth.Workload("neg_ctx", l=4, h=12, m=2, g=1, D=64, B=3, ctx=80, seed=21)
    dw = _with_contexts(DeviceWorkload(w), [-1, 5, 80])
    say("step with a -1 context")
    out = _run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = _oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    assert np.all(out[:, 0] == 0)
    _check_step(dw, out, ref, k_ref, v_ref, "step with -1 context")


def test_lengths_above_the_hint_are_truncated_to_it():
    """max_len_hint bounds the attended positions: a sequence longer than the
    hint attends to its first max_len_hint positions."""
    w = _sweep_workload(64, 2, 1, [50, 300, 150], h=12, l=2)
    dw = DeviceWorkload(w)
    lens = np.array([50, 300, 150], np.int32)
    hint = 100
    say("lengths truncated by max_len_hint")
    out = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    mlkv.decode_attention(1, dw.q[1], dw.cache, dw.map, torch.from_numpy(lens).cuda(), out,
                          max_len_hint=hint, ws=dw.ws)
    torch.cuda.synchronize()
    ref = oracle.decode_attention(1, dw.host["q"][1], dw.host["k_cache"], dw.host["v_cache"],
                                  dw.kv_of, np.minimum(lens, hint))
    check_close(out.cpu().numpy(), ref, "hint truncation",
                bound=_layer_bound(dw, 1, dw.host["k_cache"], np.minimum(lens, hint), ref))


def test_length_check_rejects_out_of_range_lengths(monkeypatch):
    """MLKV_CHECK=1 reads the device lengths back and rejects any above the
    capacity before launching anything."""
    w = _sweep_workload(64, 2, 1, [10, 20], h=12, l=2)
    dw = DeviceWorkload(w)
    monkeypatch.setenv("MLKV_CHECK", "1")
    out = torch.zeros((w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    say("MLKV_CHECK rejects a length above capacity")
    bad = torch.tensor([10, dw.S + 1], dtype=torch.int32, device="cuda")
    with pytest.raises(mlkv.MLKVError, match="MLKV_ERR_CAPACITY"):
        mlkv.decode_attention(0, dw.q[0], dw.cache, dw.map, bad, out, ws=dw.ws)
    with pytest.raises(mlkv.MLKVError, match="MLKV_ERR_CAPACITY"):
        mlkv.decode_step(dw.q, dw.k_new, dw.v_new, dw.cache, dw.map,
                         torch.tensor([3, dw.S], dtype=torch.int32, device="cuda"),
                         torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda"),
                         ws=dw.ws)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0  # nothing ran


# ------------------------------------------------------------- HIP graphs --

@pytest.mark.parametrize("wname,kw", [("mlkv4_b128_ragged", dict(B=24, ctx=900)),
                                      ("mlkv4_b8_long", dict(B=2, ctx=4000))])
def test_step_captured_in_a_hip_graph_replays_like_eager(wname, kw):
    """The whole decode step (appends, attention, in-place or separate merge)
    captured in one HIP graph: every replay, with eager steps in between,
    gives the eager output bit for bit and leaves the same cache (the step
    allocates nothing and records no memset, so it can be captured)."""
    w = small(wname, **kw)
    dw = DeviceWorkload(w)
    say(f"graph step {w.name}")
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda")

    def step():
        mlkv.decode_step(dw.q, dw.k_new, dw.v_new, dw.cache, dw.map, dw.ctx, out, ws=dw.ws)

    step()
    torch.cuda.synchronize()
    ref = out.clone()
    k_ref, v_ref = dw.read_cache()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for _ in range(3):
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
        step()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, ref)
    k, v = dw.read_cache()
    assert np.array_equal(k, k_ref) and np.array_equal(v, v_ref)
    ref64, k64, v64 = _oracle_step(dw)
    _check_step(dw, ref.cpu().numpy(), ref64, k64, v64, f"graph step {w.name}")


# --------------------------------------------------- 7B-like, full size --

def test_full_size_7b_step_sampled_sequences():
    """The 7B-like workload at full size (32 layers x 32 heads, head dim 128,
    64 KV heads owned by 8 layers, batch 64, context 8192: a 17 GB cache,
    filled on the device from a seeded generator).  Eight sampled sequences
    are checked whole: their cache rows after the step equal the rows before
    it plus the owners' new rows, and their outputs in every layer and head
    match the oracle run on their rows (sequences are independent)."""
    w = synth.get_workload("7b_mlkv8x8")
    S = w.capacity
    say("7b full: filling the cache on the device")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0x7B)
    cache = mlkv.Cache.empty(w.n_kv, w.B, S, w.D)
    cache.k.normal_(generator=gen)
    cache.v.normal_(generator=gen)
    inp = synth.step_inputs(w, with_cache=False)
    mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
    kv_of, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
    sample = [0, 9, 21, 33, 42, 50, 58, w.B - 1]
    sel = torch.tensor(sample, device="cuda")

    def rows():
        k = unpack_k(mlkv.bf16_bits(cache.k.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        v = unpack_v(mlkv.bf16_bits(cache.v.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        return k, v

    k0, v0 = rows()
    ws = mlkv.workspace(mp, w.B, S, w.D)
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    say("7b full: running the step")
    mlkv.decode_step(mlkv.bf16_tensor(inp["q"], "cuda"), mlkv.bf16_tensor(inp["k_new"], "cuda"),
                     mlkv.bf16_tensor(inp["v_new"], "cuda"), cache, mp,
                     torch.from_numpy(inp["ctx"]).cuda(), out, ws=ws)
    torch.cuda.synchronize()
    k1, v1 = rows()
    out = out.cpu().numpy()[:, sample]
    say("7b full: oracle on the sampled sequences")
    ref = oracle.decode_step(np.ascontiguousarray(inp["q"][:, sample]), k0, v0,
                             np.ascontiguousarray(inp["k_new"][sample]),
                             np.ascontiguousarray(inp["v_new"][sample]), kv_of, owner_of,
                             inp["ctx"][sample])
    assert np.array_equal(k1, k0) and np.array_equal(v1, v0), "cache rows differ"
    check_close(out, ref, "7b full, sampled sequences")


# ------------------------------------ batches above the schedule's tables --

@pytest.mark.parametrize("m,g,B", [(1, 1, 4096), (4, 1, 3000), (12, 12, 2100)])
def test_large_batch_step_sampled_sequences(m, g, B):
    """Batches above 2048 sequences (the in-kernel schedule's table size) run
    with one workgroup per (sequence, KV head).  The cache (ragged contexts
    0..300, some sequences attending only their new token) is filled on the
    device from a seeded generator; eight sampled sequences are checked
    whole against the oracle run on their rows."""
    w = synth.Workload(f"large_b{B}_m{m}g{g}", l=12, h=12, m=m, g=g, D=64, B=B,
                       ctx_range=(0, 300), seed=0x4D4C + B)
    inp = synth.step_inputs(w, with_cache=False)
    S = inp["capacity"]
    say(f"large batch {w.name}: filling the cache on the device")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(B)
    cache = mlkv.Cache.empty(w.n_kv, w.B, S, w.D)
    cache.k.normal_(generator=gen)
    cache.v.normal_(generator=gen)
    mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
    assert mp.plan(0, B, S, w.D, S)[0] == B * w.g  # a workgroup per (sequence, KV head)
    assert mp.workspace_bytes(B, S, w.D) == 0
    kv_of, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
    sample = sorted({0, 1, B // 3, B // 2, 2047, 2048, B - 2, B - 1})
    sel = torch.tensor(sample, device="cuda")

    def rows():
        k = unpack_k(mlkv.bf16_bits(cache.k.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        v = unpack_v(mlkv.bf16_bits(cache.v.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        return k, v

    k0, v0 = rows()
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    say(f"large batch {w.name}: running the step")
    mlkv.decode_step(mlkv.bf16_tensor(inp["q"], "cuda"), mlkv.bf16_tensor(inp["k_new"], "cuda"),
                     mlkv.bf16_tensor(inp["v_new"], "cuda"), cache, mp,
                     torch.from_numpy(inp["ctx"]).cuda(), out, ws=None)
    torch.cuda.synchronize()
    k1, v1 = rows()
    out = out.cpu().numpy()[:, sample]
    say(f"large batch {w.name}: oracle on the sampled sequences")
    k_ref, v_ref = k0.copy(), v0.copy()
    ref = oracle.decode_step(np.ascontiguousarray(inp["q"][:, sample]), k_ref, v_ref,
                             np.ascontiguousarray(inp["k_new"][sample]),
                             np.ascontiguousarray(inp["v_new"][sample]), kv_of, owner_of,
                             inp["ctx"][sample])
    assert np.array_equal(k1, k_ref) and np.array_equal(v1, v_ref), "cache rows differ"
    bound = step_rounding_bound(np.ascontiguousarray(inp["q"][:, sample]), k_ref, v_ref, kv_of,
                                inp["ctx"][sample], ref)
    check_close(out, ref, f"large batch {w.name}, sampled sequences", bound=bound)


def test_capacity_batch_step_sampled_sequences():
    """The capacity experiment's configuration (bench.py --workload
    capacity_ctx2048, MLKV-2): the largest batch whose 2048-token cache fits
    the free device memory (about 2.6e5 sequences, a cache of ~270 GB with
    sequences at offsets beyond 2^37 bytes), 2000 cached tokens each.  Six
    sampled sequences, the last ones included, are checked whole against the
    oracle run on their rows."""
    import bench

    w = synth.get_workload("capacity_ctx2048")
    say("capacity batch: sizing and filling the cache on the device")
    B, cache, q, kn, vn, ctx, out = bench.capacity_setup(w, "cuda", seed=0xCA9)
    S = w.capacity
    assert B > 100_000, B
    say(f"capacity batch: B={B}")
    mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
    kv_of, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
    sample = [0, 1, B // 2, B - 3, B - 2, B - 1]
    sel = torch.tensor(sample, device="cuda")

    def rows():
        k = unpack_k(mlkv.bf16_bits(cache.k.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        v = unpack_v(mlkv.bf16_bits(cache.v.index_select(1, sel)), w.n_kv, len(sample), S, w.D)
        return k, v

    k0, v0 = rows()
    say("capacity batch: running the step")
    mlkv.decode_step(q, kn, vn, cache, mp, ctx, out, max_len_hint=w.ctx + 1, ws=None)
    torch.cuda.synchronize()
    k1, v1 = rows()
    got = out.index_select(1, sel).float().cpu().numpy().astype(np.float64)
    q_h = mlkv.bf16_bits(q.index_select(1, sel))
    kn_h = mlkv.bf16_bits(kn.index_select(0, sel))
    vn_h = mlkv.bf16_bits(vn.index_select(0, sel))
    del cache, q, kn, vn, out
    torch.cuda.empty_cache()
    say("capacity batch: oracle on the sampled sequences")
    k_ref, v_ref = k0.copy(), v0.copy()
    ref = oracle.decode_step(q_h, k_ref, v_ref, kn_h, vn_h, kv_of, owner_of,
                             np.full(len(sample), w.ctx, dtype=np.int32))
    assert np.array_equal(k1, k_ref) and np.array_equal(v1, v_ref), "cache rows differ"
    # bf16 output (the benchmark's): its rounding (at most 2^-8 relative) fits
    # inside the same bars as the fp32 output
    check_close(got, ref, "capacity batch, sampled sequences (bf16 out)")

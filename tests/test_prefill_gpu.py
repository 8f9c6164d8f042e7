"""GPU parity of the prefill path (T new tokens per sequence, causal) against
the fp64 oracle, through the C ABI.

The cache after the owners' row appends is compared bit for bit; outputs
within the tolerances of gpu_util.  Every case prints its name before it
touches the GPU.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import synth  # noqa: E402
from gpu_util import (check_close, f64, prefill_rounding_bound, say,  # noqa: E402
                      softmax_rounding_bound, step_rounding_bound)
from layout_ref import unpack_k, unpack_v  # noqa: E402

pytestmark = pytest.mark.gpu

mlkv = pytest.importorskip("paper_2406_09297_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mlkv.lib()
    yield


class PrefillCase:
    """Seeded prefill inputs on host (logical order) and device."""

    def __init__(self, w: synth.Workload, ctx=None, fill=synth.BF16_NAN, kv_of=None,
                 owner_of=None, device="cuda"):
        self.w = w
        inp = synth.prefill_inputs(w, fill=fill)
        if ctx is not None:  # explicit contexts: slots at or past each are poisoned again
            ctx = np.asarray(ctx, dtype=np.int32)
            assert ctx.size == w.B and ctx.max() + w.T <= inp["capacity"]
            for arr in (inp["k_cache"], inp["v_cache"]):
                for b, c in enumerate(ctx):
                    arr[:, b, c:] = fill
            inp["ctx"] = ctx
        self.host = inp
        self.S = inp["capacity"]
        if kv_of is None:
            self.map = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
            self.kv_of, self.owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
        else:
            self.map = mlkv.Map.from_tables(kv_of, owner_of)
            self.kv_of, self.owner_of = kv_of, owner_of
        self.cache = mlkv.Cache.empty(w.n_kv, w.B, self.S, w.D, device)
        self.cache.load_rows(inp["k_cache"], inp["v_cache"])
        self.q = mlkv.bf16_tensor(inp["q"], device)
        self.k_new = mlkv.bf16_tensor(inp["k_new"], device)
        self.v_new = mlkv.bf16_tensor(inp["v_new"], device)
        self.ctx = torch.from_numpy(inp["ctx"]).to(device)

    def run(self, out_dtype=torch.float32):
        w = self.w
        out = torch.empty((w.l, w.B, w.T, w.h, w.D), dtype=out_dtype, device="cuda")
        mlkv.prefill_step(self.q, self.k_new, self.v_new, self.cache, self.map, self.ctx, out)
        torch.cuda.synchronize()
        return out

    def read_cache(self):
        torch.cuda.synchronize()
        w = self.w
        k = unpack_k(mlkv.bf16_bits(self.cache.k), w.n_kv, w.B, self.S, w.D)
        v = unpack_v(mlkv.bf16_bits(self.cache.v), w.n_kv, w.B, self.S, w.D)
        return k, v

    def oracle(self):
        k, v = self.host["k_cache"].copy(), self.host["v_cache"].copy()
        out = oracle.prefill_step(self.host["q"], k, v, self.host["k_new"], self.host["v_new"],
                                  self.kv_of, self.owner_of, self.host["ctx"])
        return out, k, v


def _check_case(c: PrefillCase, label: str):
    out = c.run().cpu().numpy()
    k_gpu, v_gpu = c.read_cache()
    ref, k_ref, v_ref = c.oracle()
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), f"{label}: cache differs"
    bound = prefill_rounding_bound(c.host["q"], k_ref, v_ref, c.kv_of, c.host["ctx"], ref)
    check_close(out, ref, label, bound=bound)


PROMPTS = [1, 2, 5, 15, 16, 17, 31, 32, 33, 70]


@pytest.mark.parametrize("T", PROMPTS)
def test_prefill_mlkv4_across_tile_and_block_edges(T):
    """Pythia-160M head shape with MLKV-4 (12 query heads per KV head): T new
    tokens on top of ragged contexts (0, 1, 31, 32, 95); query blocks of 64
    rows end mid-token and mid-tile."""
    w = synth.Workload("prefill_sweep", l=4, h=12, m=4, g=1, D=64, B=5, ctx=96, T=T, seed=81)
    say(f"prefill MLKV-4 T={T}")
    _check_case(PrefillCase(w, ctx=[0, 1, 31, 32, 95]), f"prefill T={T}")


@pytest.mark.parametrize("D,h,m,g,T", [(64, 4, 4, 4, 50), (128, 12, 2, 4, 40),
                                       (64, 16, 2, 1, 9), (64, 24, 2, 1, 10),
                                       (128, 8, 1, 1, 37)])
def test_prefill_group_sizes_and_head_dims(D, h, m, g, T):
    """One query head per KV head (MHA), three, sixteen (a whole MFMA block
    per token), twenty-four (beyond the decode path's 16-head limit) and
    eight with head dimension 128."""
    w = synth.Workload("prefill_groups", l=4 if m < 4 else m, h=h, m=m, g=g, D=D, B=3, ctx=40,
                       T=T, seed=82)
    say(f"prefill D={D} h={h} m={m} g={g} T={T}")
    _check_case(PrefillCase(w, ctx=[0, 17, 40]), f"prefill D{D} h{h} m{m} g{g} T{T}")


def test_prefill_long_prompt_empty_cache():
    """A 300-token prompt into an empty cache (ten tiles on the diagonal)."""
    w = synth.Workload("prefill_long", l=2, h=12, m=1, g=1, D=64, B=2, ctx=0, T=300, seed=83)
    say("prefill T=300")
    _check_case(PrefillCase(w), "prefill T=300")


@pytest.mark.parametrize("ctx,T,D,seed", [(64, 80, 64, 84), (0, 160, 64, 85), (100, 300, 64, 86),
                                          (31, 33, 64, 87), (64, 80, 128, 88), (500, 257, 64, 89)])
def test_prefill_peaked_scores(ctx, T, D, seed):
    """Keys x3 before rounding (peaked softmax, as in the long decode case),
    over prompt lengths and contexts that put the causal edge at different
    tile and block offsets."""
    w = synth.Workload("prefill_peaked", l=2, h=12, m=2, g=1, D=D, B=2, ctx=ctx, T=T,
                       k_scale=3.0, seed=seed)
    say(f"prefill peaked ctx={ctx} T={T} D={D}")
    _check_case(PrefillCase(w), f"prefill peaked ctx={ctx} T={T} D={D}")


def test_prefill_general_map_owner_not_reading_its_head():
    """Layer 0 owns KV heads 0 and 1 but reads only head 0: both get their
    rows, and layer 1 reads head 1."""
    w = synth.Workload("prefill_general", l=4, h=4, m=2, g=1, D=64, B=2, ctx=20, T=12, seed=85)
    kv_of = np.array([[0] * 4, [1] * 4, [0] * 4, [1] * 4], np.int32)
    owner_of = np.array([0, 0], np.int32)
    say("prefill general map")
    _check_case(PrefillCase(w, ctx=[3, 20], kv_of=kv_of, owner_of=owner_of), "prefill general")


def test_prefill_bf16_output_is_the_rounded_fp32_output():
    """prefill_attention in bf16 output mode is the RNE rounding of its fp32
    output (same cache, same call otherwise)."""
    w = synth.Workload("prefill_bf16", l=1, h=12, m=1, g=1, D=64, B=2, ctx=10, T=45, seed=86)
    c = PrefillCase(w, ctx=[0, 10])
    say("prefill bf16 output")
    c.run()  # appends the rows
    q0 = c.q[0]
    o32 = torch.empty((w.B, w.T, w.h, w.D), dtype=torch.float32, device="cuda")
    o16 = torch.empty((w.B, w.T, w.h, w.D), dtype=torch.bfloat16, device="cuda")
    mlkv.prefill_attention(0, q0, c.cache, c.map, c.ctx, o32)
    mlkv.prefill_attention(0, q0, c.cache, c.map, c.ctx, o16)
    torch.cuda.synchronize()
    assert np.array_equal(mlkv.bf16_bits(o16), synth.f32_to_bf16(o32.cpu().numpy()))


@pytest.mark.parametrize("D", [64, 128])
def test_prefill_repeats_bit_for_bit(D):
    """Repeated launches on the same cache give identical outputs, at both head
    sizes (a read of matrix-core results without the wait states the hardware
    requires once made the softmax reference, and so the rounding of some
    rows, vary from launch to launch)."""
    w = synth.Workload("prefill_repeat", l=1, h=12, m=1, g=1, D=D, B=2, ctx=20, T=70, seed=88)
    c = PrefillCase(w, ctx=[3, 20])
    say(f"prefill repeats D={D}")
    c.run()
    outs = []
    for _ in range(8):
        o = torch.empty((w.B, w.T, w.h, w.D), dtype=torch.float32, device="cuda")
        mlkv.prefill_attention(0, c.q[0], c.cache, c.map, c.ctx, o)
        torch.cuda.synchronize()
        outs.append(o.cpu().numpy())
    for o in outs[1:]:
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))


def test_prefill_of_zero_tokens_changes_nothing():
    w = synth.Workload("prefill_zero", l=2, h=12, m=1, g=1, D=64, B=2, ctx=10, T=1, seed=87)
    c = PrefillCase(w)
    say("prefill T=0")
    k0, v0 = c.read_cache()
    out = torch.full((w.l, w.B, 1, w.h, w.D), 7.0, dtype=torch.float32, device="cuda")
    assert mlkv.lib().mlkv_prefill_step(c.q.data_ptr(), c.k_new.data_ptr(), c.v_new.data_ptr(),
                                        c.cache.struct, c.map.handle, c.ctx.data_ptr(), 0,
                                        out.data_ptr(), mlkv.OUT_F32, None) == 0
    torch.cuda.synchronize()
    k1, v1 = c.read_cache()
    assert np.array_equal(k0, k1) and np.array_equal(v0, v1)
    assert torch.all(out == 7.0)


def test_prefill_then_decode_continues_the_sequence():
    """A 40-token prefill followed by one decode step at context ctx + 40
    matches the oracle's prefill then decode step."""
    w = synth.Workload("prefill_then_decode", l=4, h=12, m=2, g=1, D=64, B=3, ctx=30, T=40,
                       seed=88)
    c = PrefillCase(w, ctx=[0, 7, 30])
    say("prefill then decode")
    c.run()
    ref_p, k_ref, v_ref = c.oracle()
    ctx2 = c.host["ctx"] + w.T
    q2 = synth.normal_bf16(89, 0, (w.l, w.B, w.h, w.D))
    kn2 = synth.normal_bf16(89, 3, (w.B, w.n_kv, w.D))
    vn2 = synth.normal_bf16(89, 4, (w.B, w.n_kv, w.D))
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device="cuda")
    ws = mlkv.workspace(c.map, w.B, c.S, w.D)
    mlkv.decode_step(mlkv.bf16_tensor(q2, "cuda"), mlkv.bf16_tensor(kn2, "cuda"),
                     mlkv.bf16_tensor(vn2, "cuda"), c.cache, c.map,
                     torch.from_numpy(ctx2).cuda(), out, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.decode_step(q2, k_ref, v_ref, kn2, vn2, c.kv_of, c.owner_of, ctx2)
    k_gpu, v_gpu = c.read_cache()
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref)
    bound = step_rounding_bound(q2, k_ref, v_ref, c.kv_of, ctx2, ref)
    check_close(out.cpu().numpy(), ref, "decode after prefill", bound=bound)


def test_full_size_prefill_sampled_rows():
    """The benchmark's prefill (Pythia-160M shape, MLKV-4, batch 8, a
    2000-token prompt into an empty cache): the whole cache bit for bit, and
    sampled output rows (every layer, first/last sequence, tokens at the
    start, across tile edges and at the end) against the oracle row by row."""
    w = synth.get_workload("prefill_b8_2000")
    say("full prefill: uploading")
    c = PrefillCase(w, fill=0)
    say("full prefill: running")
    out = c.run().cpu().numpy()
    k_gpu, v_gpu = c.read_cache()
    h = c.host
    k_ref, v_ref = h["k_cache"].copy(), h["v_cache"].copy()
    for n in range(w.l):
        oracle.append_rows(n, k_ref, v_ref, h["k_new"], h["v_new"], c.owner_of, h["ctx"])
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), "cache differs"
    say("full prefill: oracle rows")
    rows, refs, bounds = [], [], []
    for n in range(w.l):
        for b in (0, w.B - 1):
            for t in (0, 1, 31, 32, 63, 64, 1000, w.T - 2, w.T - 1):
                for i in (0, w.h - 1):
                    kv = c.kv_of[n, i]
                    L = int(h["ctx"][b]) + t + 1
                    o, _ = oracle.attend_one(h["q"][n, b, t, i], k_ref[kv, b, :L], v_ref[kv, b, :L])
                    rows.append(out[n, b, t, i])
                    refs.append(o)
                    bounds.append(softmax_rounding_bound(
                        f64(h["q"][n, b, t, i])[None], f64(k_ref[kv, b, :L]), f64(v_ref[kv, b, :L]),
                        o[None], np.array([L]))[0])
    check_close(np.array(rows), np.array(refs), "full prefill sampled rows", bound=np.array(bounds))

"""Seeded random cases on the GPU against the oracle, with the helpers and
bars of the other parity tests: maps (l, h, m, g), head sizes, batches and
ragged lengths within the filled cache, launch-plan overrides (workgroup
budget, merge in place or by the merge kernel, wide workgroups), rotary
widths, prompt lengths on top of cached tokens, and whole model steps.  Each
case draws its parameters from its own index, prints them first, and so
names itself when it fails.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402
import test_decode_gpu as td  # noqa: E402
import test_model_gpu as tm  # noqa: E402
import test_prefill_gpu as tp  # noqa: E402
from gpu_util import DeviceWorkload, say  # noqa: E402

pytestmark = pytest.mark.gpu

mlkv = pytest.importorskip("paper_2406_09297_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mlkv.lib()
    yield


def _divisors(n):
    return [d for d in range(1, n + 1) if n % d == 0]


def _map(rng):
    l = int(rng.choice([2, 3, 4, 6, 8, 12]))
    h = int(rng.choice([4, 8, 12, 16]))
    return l, h, int(rng.choice(_divisors(l))), int(rng.choice(_divisors(h)))


def _plan(rng):
    return dict(workgroups=str(int(rng.integers(1, 700))) if rng.random() < 0.3 else "",
                merge=str(rng.choice(["", "", "kernel", "fused"])),
                wide=str(rng.choice(["", "", "0", "1"])))


def _step_case(i, rotary):
    rng = np.random.default_rng(0x57E9 + 1000 * rotary + i)
    l, h, m, g = _map(rng)
    D = int(rng.choice([64, 128]))
    B = int(rng.integers(1, 25))
    filled = int(rng.choice([40, 100, 300]))
    env = _plan(rng)
    seed = int(rng.integers(1 << 30))
    w = synth.Workload("random", l=l, h=h, m=m, g=g, D=D, B=B, ctx=filled, seed=seed)
    dw = DeviceWorkload(w)
    top = min(filled, dw.S - 1)  # contexts within the filled slots
    pool = [0, 1, 31, 32, 33, 63, 64, top]
    ctx = np.where(rng.random(B) < 0.3, rng.choice(pool, B), rng.integers(0, top + 1, B))
    ctx = np.minimum(ctx, top).astype(np.int32)
    rd = int(rng.choice([16, 32, D])) if rotary else 0
    tag = f"l{l} h{h} m{m} g{g} D{D} B{B} filled{filled} rd{rd} plan={env} seed={seed}"
    say(f"random {'rotary ' if rotary else ''}step {i}: {tag}")
    td._with_contexts(dw, ctx)
    with td.plan_env(**env):
        if rotary:
            td._check_rope_step(dw, rd, tag)
            return
        out = td._run_step(dw).cpu().numpy()
    k_gpu, v_gpu = dw.read_cache()
    ref, k_ref, v_ref = td._oracle_step(dw)
    assert np.array_equal(k_gpu, k_ref) and np.array_equal(v_gpu, v_ref), f"{tag}: cache differs"
    td._check_step(dw, out, ref, k_ref, v_ref, tag)


@pytest.mark.parametrize("i", range(12))
def test_random_decode_step(i):
    _step_case(i, rotary=False)


@pytest.mark.parametrize("i", range(6))
def test_random_rotary_step(i):
    _step_case(i, rotary=True)


@pytest.mark.parametrize("i", range(8))
def test_random_prefill(i):
    rng = np.random.default_rng(0x9F11 + i)
    l, h, m, g = _map(rng)
    D = int(rng.choice([64, 128]))
    B = int(rng.integers(1, 5))
    T = int(rng.integers(1, 90))
    filled = int(rng.choice([0, 20, 100]))
    seed = int(rng.integers(1 << 30))
    w = synth.Workload("random_pf", l=l, h=h, m=m, g=g, D=D, B=B, ctx=filled, T=T, seed=seed)
    ctx = rng.integers(0, filled + 1, B)  # within the filled slots
    tag = f"l{l} h{h} m{m} g{g} D{D} B{B} T{T} ctx={ctx.tolist()} seed={seed}"
    say(f"random prefill {i}: {tag}")
    tp._check_case(tp.PrefillCase(w, ctx=ctx.tolist()), tag)


@pytest.mark.parametrize("i", range(6))
def test_random_model_step(i):
    rng = np.random.default_rng(0x30DE + i)
    l = int(rng.choice([2, 3, 4, 6]))
    h = int(rng.choice([2, 4, 6, 8, 12]))
    m = int(rng.choice(_divisors(l)))
    g = int(rng.choice(_divisors(h)))
    D = int(rng.choice([64, 64, 128]))
    d_ff = 32 * int(rng.integers(4, 40))
    B = int(rng.integers(1, 25))
    ctx = [int(c) for c in rng.integers(0, 300, B)]
    rd = int(rng.choice([16, 32]))
    seed = int(rng.integers(1 << 20))
    tm._run_case(l, h, D, d_ff, m, g, B, ctx, seed, rd=rd,
                 label=f"random model {i}: l{l} h{h} m{m} g{g} D{D} ff{d_ff} B{B} rd{rd} seed{seed}")

"""mlkv_decode_step_noalloc (the step on the library's static device scratch,
for callers that cannot allocate) against mlkv_decode_step (the same step on
a caller's workspace), through the C ABI: outputs and caches identical, on
calls in a row over one device's scratch, the second with a smaller batch and
shorter contexts, the third the first again (so the scratch's arrival
counters must have returned to zero)."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402
from gpu_util import DeviceWorkload, say  # noqa: E402

pytestmark = pytest.mark.gpu

mlkv = pytest.importorskip("paper_2406_09297_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    mlkv.lib()
    yield


def _step_both(dw, label):
    """The step through both entry points on two copies of the same cache."""
    w = dw.w
    L = mlkv.lib()
    k0, v0 = dw.cache.k.clone(), dw.cache.v.clone()
    stream = torch.cuda.current_stream().cuda_stream
    out_ws = torch.full((w.l, w.B, w.h, w.D), float("nan"), dtype=torch.float32, device="cuda")
    out_na = torch.full_like(out_ws, float("nan"))
    max_len = int(dw.host["ctx"].max()) + 1
    args = (dw.q.data_ptr(), dw.k_new.data_ptr(), dw.v_new.data_ptr(), dw.cache.struct,
            dw.map.handle, dw.ctx.data_ptr())
    say(f"noalloc {label}: workspace step")
    st = L.mlkv_decode_step(*args, out_ws.data_ptr(), mlkv.OUT_F32, max_len, dw.ws.data_ptr(),
                            dw.ws.numel(), stream)
    assert st == mlkv.MLKV_OK, L.mlkv_last_error().decode()
    torch.cuda.synchronize()
    k_ws, v_ws = dw.cache.k.clone(), dw.cache.v.clone()
    dw.cache.k.copy_(k0)
    dw.cache.v.copy_(v0)
    say(f"noalloc {label}: static-scratch step")
    st = L.mlkv_decode_step_noalloc(*args, out_na.data_ptr(), mlkv.OUT_F32, max_len, stream)
    assert st == mlkv.MLKV_OK, L.mlkv_last_error().decode()
    torch.cuda.synchronize()
    assert torch.equal(out_na, out_ws), f"{label}: outputs differ"
    # bit patterns: the slots past each context hold NaN
    same = (torch.equal(dw.cache.k.view(torch.int16), k_ws.view(torch.int16)) and
            torch.equal(dw.cache.v.view(torch.int16), v_ws.view(torch.int16)))
    assert same, f"{label}: caches differ"
    assert bool(torch.isfinite(out_na).all())


def test_noalloc_step_matches_the_workspace_step_on_consecutive_calls():
    big = synth.Workload("noalloc_big", l=12, h=12, m=4, g=1, D=64, B=96, ctx_range=(200, 2000),
                         seed=0x5C1)
    small = synth.Workload("noalloc_small", l=4, h=12, m=2, g=3, D=64, B=9, ctx_range=(1, 300),
                           seed=0x5C2)
    d128 = synth.Workload("noalloc_d128", l=4, h=8, m=2, g=2, D=128, B=5, ctx_range=(30, 900),
                          seed=0x5C3)
    for w in (big, small, d128, big):
        _step_both(DeviceWorkload(w), f"{w.name} B={w.B} D={w.D}")


def test_noalloc_rejects_a_step_above_the_scratch_size():
    """A step whose split-run partials need more than the 16 MiB scratch is
    refused before anything is launched (the workspace entry point takes it)."""
    mp = mlkv.Map.uniform(12, 12, 4, 1)
    B, S, D = 511, 16384, 64
    assert mp.workspace_bytes(B, S, D) > (16 << 20)
    cache = mlkv._Cache(0x10000, 0x20000, 4, B, S, D)
    L = mlkv.lib()
    st = L.mlkv_decode_step_noalloc(0x30000, 0x30000, 0x30000, ctypes.byref(cache), mp.handle,
                                    0x40000, 0x50000, mlkv.OUT_F32, 0, None)
    assert mlkv.STATUS_NAMES[st] == "MLKV_ERR_WORKSPACE"
    assert "static scratch" in L.mlkv_last_error().decode()

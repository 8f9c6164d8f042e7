"""Host checks of the integer arithmetic the attention kernel's run schedule
does in float32: ceil(t / R) as floor((t - 1/2) * rcp(R)) + 1 and floor(rem /
nb) as floor((rem + 1/2) * rcp(nb)), where rcp is the hardware reciprocal
(within one ulp of 1/R).  Each is emulated in numpy float32 with the
reciprocal rounded to nearest and moved one ulp either way, and compared with
exact integer division over the ranges the kernel uses (tiles of a unit below
2^15, run lengths up to the same, run indices below 2^20)."""
import numpy as np
import pytest


def _recips(y):
    r = (np.float32(1.0) / y.astype(np.float32)).astype(np.float32)
    return [np.nextafter(r, np.float32(0.0)), r, np.nextafter(r, np.float32(np.inf))]


@pytest.mark.parametrize("r_lo,r_hi", [(1, 512), (512, 4096), (4096, 32769)])
def test_ceil_div_half(r_lo, r_hi):
    rng = np.random.default_rng(r_lo)
    t = np.arange(0, 1 << 15, dtype=np.int64)
    Rs = np.arange(r_lo, r_hi) if r_hi - r_lo <= 512 else np.unique(rng.integers(r_lo, r_hi, 400))
    for R in Rs:
        Rv = np.full(t.shape, R, dtype=np.int64)
        want = -(-t // Rv)
        th = (t.astype(np.float32) - np.float32(0.5)).astype(np.float32)
        for rR in _recips(Rv):
            got = np.floor((th * rR).astype(np.float32)).astype(np.int64) + 1
            assert np.array_equal(got, want), f"R = {R}"


def test_floor_div_half():
    rng = np.random.default_rng(7)
    rem = np.concatenate([np.arange(0, 1 << 14), rng.integers(0, 1 << 20, 1 << 16)]).astype(np.int64)
    for nb in list(range(1, 300)) + list(rng.integers(300, 1 << 15, 200)):
        nbv = np.full(rem.shape, nb, dtype=np.int64)
        want = rem // nbv
        x = (rem.astype(np.float32) + np.float32(0.5)).astype(np.float32)
        for r in _recips(nbv):
            got = np.floor((x * r).astype(np.float32)).astype(np.int64)
            assert np.array_equal(got, want), f"nb = {nb}"


def test_packed_halves_do_not_carry():
    """Per-candidate run counts are packed two to a 32-bit word and scanned;
    with every prefix at most 2^15 the halves add and subtract independently."""
    rng = np.random.default_rng(3)
    a = rng.integers(0, 16, 2048)
    b = rng.integers(0, 16, 2048)
    a[-1] = (1 << 15) - a[:-1].sum()  # the low half's total at its bound 2^15
    b[-1] = (1 << 15) - b[:-1].sum()
    assert a[-1] >= 0 and b[-1] >= 0
    packed = (a | (b << 16)).astype(np.int64)
    incl = np.cumsum(packed) & 0xFFFFFFFF
    excl = (incl - packed) & 0xFFFFFFFF
    assert np.array_equal(incl & 0xFFFF, np.cumsum(a) & 0xFFFF)
    assert np.array_equal(incl >> 16, np.cumsum(b))
    assert np.array_equal(excl & 0xFFFF, np.cumsum(a) - a)
    assert np.array_equal(excl >> 16, np.cumsum(b) - b)

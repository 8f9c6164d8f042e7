"""Host checks of the tests' own statement of the cache layout (layout_ref):
the key plane's chunk order inside a 32-token tile is a permutation of the
tile's 4*D chunks, each load instruction's 1 KB run holds exactly the
matrix-core operands its 64 lanes need (lane 16 g + r: row r of the 16-token
half, channels 8 g .. 8 g + 7 of the 32-channel step), and packing and
unpacking are inverse to each other and agree with the element index."""
import numpy as np
import pytest

import layout_ref


@pytest.mark.parametrize("D", [64, 128])
def test_key_chunks_form_a_permutation_matching_the_operand_lanes(D):
    KK = D // 32
    chunks = {layout_ref.k_chunk(u, c, D) for u in range(32) for c in range(D // 8)}
    assert chunks == set(range(4 * D))
    for sb in range(2):
        for kk in range(KK):
            for lane in range(64):
                r, g = lane & 15, lane >> 4
                token = (r >> 2) * 8 + sb * 4 + (r & 3)  # the half's row r
                assert layout_ref.k_chunk(token, g + 4 * kk, D) == (sb * KK + kk) * 64 + lane


@pytest.mark.parametrize("D", [64, 128])
def test_pack_unpack_and_index(D):
    rng = np.random.default_rng(D)
    rows = rng.integers(0, 0xFFFF, size=(2, 3, 96, D), dtype=np.uint16)
    plane = layout_ref.pack_k(rows)
    assert np.array_equal(layout_ref.unpack_k(plane, 2, 3, 96, D), rows)
    flat = plane.reshape(-1)
    for kv, b, t, d in zip(rng.integers(0, 2, 500), rng.integers(0, 3, 500),
                           rng.integers(0, 96, 500), rng.integers(0, D, 500)):
        assert flat[layout_ref.k_index(kv, b, t, d, 3, 96, D)] == rows[kv, b, t, d]
    vflat = layout_ref.pack_v(rows).reshape(-1)
    for kv, b, t, d in zip(rng.integers(0, 2, 200), rng.integers(0, 3, 200),
                           rng.integers(0, 96, 200), rng.integers(0, D, 200)):
        assert vflat[layout_ref.v_index(kv, b, t, d, 3, 96, D)] == rows[kv, b, t, d]

"""Writes tiny_step_outputs.txt: the oracle's outputs for a tiny seeded MLKV
decode step.  Calls only oracle/ and synth/ (never the HIP library).

    python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402


def tiny_step():
    """MLKV with l=4, h=4, m=2, g=2 (two KV heads per owning layer, two query
    heads per KV head), D=8, B=2, contexts (3, 6), capacity 8."""
    l, h, m, g, D, B, S = 4, 4, 2, 2, 8, 2, 8
    ctx = np.array([3, 6], np.int32)
    n_kv = m * g
    kv_of, owner_of = oracle.map_uniform(l, h, m, g)
    q = synth.normal_bf16(77, synth.STREAM_Q, (l, B, h, D))
    kn = synth.normal_bf16(77, synth.STREAM_K_NEW, (B, n_kv, D))
    vn = synth.normal_bf16(77, synth.STREAM_V_NEW, (B, n_kv, D))
    lens = np.tile(ctx, n_kv)
    kc = synth.rows_bf16(77, synth.STREAM_K_CACHE, n_kv * B, S, D, lens).reshape(n_kv, B, S, D)
    vc = synth.rows_bf16(77, synth.STREAM_V_CACHE, n_kv * B, S, D, lens).reshape(n_kv, B, S, D)
    return oracle.decode_step(q, kc, vc, kn, vn, kv_of, owner_of, ctx)


if __name__ == "__main__":
    out = tiny_step()
    path = os.path.join(HERE, "tiny_step_outputs.txt")
    header = ("oracle outputs [l=4][B=2][h=4][D=8] (row-major) of tests/golden/make_golden.py "
              "tiny_step(); written by that script from oracle/ only")
    np.savetxt(path, out.ravel(), fmt="%.17g", header=header)
    print("wrote", path, out.size, "values")

"""Decode-step benchmark of MLKV decode attention on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
for every layer, the owning layers append the newest token's K/V, then every
query head attends over its (shared) KV head through split-K decode attention
(mlkv_decode_step through the C ABI).  Inputs are resident in HBM before the
timed region starts.

Prints ONE JSON line:
  value = algorithmic decode-attention bytes per step / step time (GB/s),
  plus steps/s, the roofline object of the dominant kernel (split-K
  attention, timed per launch with HIP events on the launch stream) and the
  CPU-oracle baseline on the host cores.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--cold]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
DEFAULT_WORKLOAD = "mlkv4_b128_ragged"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def step_bytes(w, ctx, kv_count, owned_count, out_bytes=4):
    """Algorithmic HBM bytes of one step, by layer: every cached K/V byte of the
    KV heads a layer reads, read once per layer; q read; output written; the
    appended rows read and written in owning layers."""
    L = ctx.astype(np.int64) + 1
    per_layer = []
    for n in range(w.l):
        kv = kv_count[n] * int(L.sum()) * w.D * 2 * 2
        q = w.B * w.h * w.D * 2
        out = w.B * w.h * w.D * out_bytes
        app = owned_count[n] * w.B * w.D * 2 * 2 * 2
        per_layer.append(dict(kv=kv, q=q, out=out, append=app))
    return per_layer


def cpu_baseline(w, inp, kv_of, owner_of, bytes_per_step, budget_s=12.0):
    """The oracle, as it stands, on the host cores: whole decode steps on the
    same host inputs, repeated until the time budget is used (at least once)."""
    import oracle

    threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    runs, t0 = 0, time.perf_counter()
    while True:
        k, v = inp["k_cache"].copy(), inp["v_cache"].copy()
        ts = time.perf_counter()
        oracle.decode_step(inp["q"], k, v, inp["k_new"], inp["v_new"], kv_of, owner_of, inp["ctx"])
        runs += 1
        if runs == 1:
            spent = time.perf_counter() - ts
        else:
            spent += time.perf_counter() - ts
        if time.perf_counter() - t0 >= budget_s:
            break
    return {"value": bytes_per_step * runs / spent / 1e9, "unit": "GB/s", "cores": threads,
            "kind": "oracle", "steps_per_s": runs / spent,
            "sample": f"{runs} whole decode step(s) of the same workload (fp64 oracle, "
                      f"OpenMP over (sequence, head)), {spent:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cold", action="store_true",
                    help="flush caches (512 MB write) before each timed attention launch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the decode path is "
                                   "single-GPU (multi-GPU sharding is a design note, not built)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    import synth
    import paper_2406_09297_amd as mlkv

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = synth.get_workload(args.workload)
    if w.sweep:
        m, g = w.sweep[-1]
        w = w.with_map(m, g)
    log(f"[bench] workload {w.name}: generating inputs")
    inp = synth.step_inputs(w, fill=0)
    S = inp["capacity"]
    mp = mlkv.Map.uniform(w.l, w.h, w.m, w.g)
    cache = mlkv.Cache.empty(w.n_kv, w.B, S, w.D, dev)
    log("[bench] uploading")
    for kv in range(w.n_kv):
        cache.load_rows(inp["k_cache"][kv:kv + 1], inp["v_cache"][kv:kv + 1], (kv, kv + 1))
    q = mlkv.bf16_tensor(inp["q"], dev)
    kn = mlkv.bf16_tensor(inp["k_new"], dev)
    vn = mlkv.bf16_tensor(inp["v_new"], dev)
    ctx = torch.from_numpy(inp["ctx"]).to(dev)
    out = torch.empty((w.l, w.B, w.h, w.D), dtype=torch.float32, device=dev)
    ws = mlkv.workspace(mp, w.B, S, w.D, dev)
    max_len = int(inp["ctx"].max()) + 1
    stream = torch.cuda.current_stream()

    kv_count = [mp.layer_kv_count(n) for n in range(w.l)]
    owned = [mp.layer_owned(n)[1] for n in range(w.l)]
    per_layer = step_bytes(w, inp["ctx"], kv_count, owned)
    step_total = sum(sum(x.values()) for x in per_layer)
    kv_total = sum(x["kv"] for x in per_layer)

    def one_step():
        mlkv.decode_step(q, kn, vn, cache, mp, ctx, out, max_len_hint=max_len, ws=ws)

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        one_step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps

    # Per-launch duration of the dominant kernel (split-K attention; the
    # combine is launched only when a sequence spans several splits), HIP
    # events on the launch stream around each call, natural layer order.
    log("[bench] per-launch attention timing")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev) if args.cold else None
    reps = max(3, min(20, args.steps // 5))
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(reps * w.l)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(reps * w.l)]
    lens_attn = (ctx + 1).to(torch.int32)
    out_l = torch.empty((w.B, w.h, w.D), dtype=torch.float32, device=dev)
    i = 0
    for _ in range(reps):
        for n in range(w.l):
            if flush is not None:
                flush.fill_(i & 0xFF)
            starts[i].record(stream)
            mlkv.decode_attention(n, q[n], cache, mp, lens_attn, out_l, max_len_hint=max_len,
                                  ws=ws)
            ends[i].record(stream)
            i += 1
    torch.cuda.synchronize()
    durs = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)]) * 1e-3  # seconds
    attn_bytes = np.mean([x["kv"] + x["q"] + x["out"] for x in per_layer])
    avg = float(durs.mean())
    achieved = attn_bytes / avg / 1e9
    tps, ns = mp.plan_splits(0, w.B, S, w.D, max_len)

    result = {
        "metric": "decode-attention HBM GB/s (% of peak) + decode steps/s, MLKV Pythia-160M shape",
        "value": round(step_total / (ms_step * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "steps_per_s": round(1e3 / ms_step, 1),
        "pct_of_hbm_peak": round(100 * step_total / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 2),
        "kv_gbs": round(kv_total / (ms_step * 1e-3) / 1e9, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 q/K/V; no weights)",
        "config": {"workload": w.name, "l": w.l, "h": w.h, "m": w.m, "g": w.g, "head_dim": w.D,
                   "batch": w.B, "ctx": w.ctx if w.ctx is not None else list(w.ctx_range),
                   "ctx_sum": int(inp["ctx"].sum()), "capacity": S,
                   "bytes_per_step": int(step_total), "kv_bytes_per_step": int(kv_total),
                   "split_tokens_layer0": tps, "splits_layer0": ns},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "attn_partial_kernel (+ combine when split)",
                     "avg_launch_us": round(avg * 1e6, 3),
                     "bytes_per_launch": int(attn_bytes),
                     "cache_state": "cold (512 MB flush before each launch)" if args.cold
                     else "warm (natural layer order)"},
    }
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        import oracle

        kv_of, owner_of = oracle.map_uniform(w.l, w.h, w.m, w.g)
        result["cpu_baseline"] = cpu_baseline(w, inp, kv_of, owner_of, step_total)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

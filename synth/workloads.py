"""Shapes and seeds of the decode workloads (synthetic, no weights, no data).

Every workload is one decode step of a model with ``l`` layers and ``h`` query
heads of dimension ``D``, a uniform MLKV map (``m`` layers own ``g`` KV heads
each), batch ``B`` and per-sequence cached context ``ctx_b`` (tokens already in
the cache before the step; the step appends one token, so attention covers
``ctx_b + 1`` positions).  q, K, V are i.i.d. N(0,1) in bf16 from the seed;
``k_scale`` multiplies the keys before rounding (a peaked softmax).

The five shapes follow the paper's own inference experiment (Pythia-160M:
12 layers, 12 heads, head dim 64, decode against a cache of about 2000
tokens, Section 4.5) and the Table 2 sharing variants, plus a long-context
case and a 7B-like shape.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    l: int
    h: int
    m: int
    g: int
    D: int
    B: int
    ctx: int | None = None            # uniform context, or None if ragged
    ctx_range: tuple | None = None    # inclusive [lo, hi] for ragged contexts
    k_scale: float = 1.0
    seed: int = 0x4D4C4B56
    note: str = ""
    sweep: tuple = field(default_factory=tuple)   # (m, g) points of a map sweep
    T: int = 1                        # new tokens per sequence (prefill when > 1)
    d_ff: int = 0                     # > 0: a whole-model decode step (MLP width)

    @property
    def n_kv(self) -> int:
        return self.m * self.g

    @property
    def max_ctx(self) -> int:
        return self.ctx if self.ctx is not None else self.ctx_range[1]

    @property
    def capacity(self) -> int:
        """Cache capacity: the longest attended length rounded up to 64."""
        need = self.max_ctx + self.T
        return (need + 63) // 64 * 64

    def with_map(self, m: int, g: int) -> "Workload":
        return Workload(self.name + f"-m{m}g{g}", self.l, self.h, m, g, self.D, self.B,
                        self.ctx, self.ctx_range, self.k_scale, self.seed, self.note, T=self.T,
                        d_ff=self.d_ff)

    def scaled(self, B: int | None = None, ctx: int | None = None,
               T: int | None = None) -> "Workload":
        """Same map and statistics with a smaller batch / context / prompt (test sizes)."""
        c, cr = self.ctx, self.ctx_range
        if ctx is not None:
            if cr is not None:
                cr = (min(cr[0], ctx), ctx)
            else:
                c = ctx
        return Workload(self.name + "-small", self.l, self.h, self.m, self.g, self.D,
                        B or self.B, c, cr, self.k_scale, self.seed, self.note, T=T or self.T,
                        d_ff=self.d_ff)


WORKLOADS = {
    "mlkv2_b1": Workload(
        "mlkv2_b1", l=12, h=12, m=2, g=1, D=64, B=1, ctx=128, seed=0x4D4C4B56 + 0,
        note="Pythia-160M shape, MLKV-2 (KV heads owned by layers 0 and 6), batch 1, "
             "128 cached tokens + the new one"),
    "sweep_b32": Workload(
        "sweep_b32", l=12, h=12, m=12, g=12, D=64, B=32, ctx=2048, seed=0x4D4C4B56 + 1,
        note="Pythia-160M shape, batch 32, context 2048, map sweep",
        sweep=((12, 12), (12, 4), (12, 1), (6, 1), (4, 1), (1, 1))),
    "mlkv4_b128_ragged": Workload(
        "mlkv4_b128_ragged", l=12, h=12, m=4, g=1, D=64, B=128, ctx_range=(512, 2048),
        seed=0x4D4C4B56 + 2,
        note="Pythia-160M shape, MLKV-4 (owners 0,3,6,9), batch 128, ragged context "
             "U{512..2048}, append in owning layers"),
    "mlkv4_b8_long": Workload(
        "mlkv4_b8_long", l=12, h=12, m=4, g=1, D=64, B=8, ctx=32768, k_scale=3.0,
        seed=0x4D4C4B56 + 3,
        note="Pythia-160M shape, MLKV-4, batch 8, context 32768, keys x3 (peaked softmax)"),
    "7b_mlkv8x8": Workload(
        "7b_mlkv8x8", l=32, h=32, m=8, g=8, D=128, B=64, ctx=8192, seed=0x4D4C4B56 + 4,
        note="7B-like shape, 32 layers x 32 heads, head dim 128, 8 owning layers with 8 KV "
             "heads each (64 KV heads, 4 query heads per KV head), batch 64, context 8192"),
    "prefill_b8_2000": Workload(
        "prefill_b8_2000", l=12, h=12, m=4, g=1, D=64, B=8, ctx=0, T=2000,
        seed=0x4D4C4B56 + 5,
        note="Pythia-160M shape, MLKV-4, batch 8: a 2000-token prompt prefilled into an "
             "empty cache (the paper's inference runs first fill a 2000-token cache)"),
    "model_b8": Workload(
        "model_b8", l=12, h=12, m=4, g=1, D=64, B=8, ctx=2000, d_ff=3072, seed=0x4D4C4B56 + 6,
        note="whole Pythia-160M-shaped decode step (synthetic weights, rotary on 16 channels) "
             "at batch 8 on a 2000-token cache, the shape of the paper's throughput "
             "measurement; map sweep over the Table 2 variants",
        sweep=((12, 12), (12, 4), (4, 12), (12, 1), (4, 3), (6, 1), (2, 1), (1, 1), (4, 1))),
    "capacity_ctx2048": Workload(
        "capacity_ctx2048", l=12, h=12, m=2, g=1, D=64, B=0, ctx=2000, seed=0x4D4C4B56 + 7,
        note="Pythia-160M shape: the largest batch whose 2048-token cache (2000 cached tokens "
             "plus 48 decode steps, the paper's memory protocol) and step buffers fit in the "
             "GPU's free memory, per Table 2 map; B is set at run time",
        sweep=((12, 12), (12, 4), (4, 12), (12, 1), (4, 3), (6, 1), (4, 1), (2, 1), (1, 1))),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def step_bytes_per_sequence(w: Workload, capacity: int, out_bytes: int = 2) -> int:
    """Device bytes one sequence of a decode step occupies: its cache rows (keys
    and values of every KV head, ``capacity`` slots, bf16: the per-sequence
    share of the cache size 2*b*s*m*g*d_k), the queries and outputs of every
    layer, the new token's key and value rows, and its length."""
    cache = 2 * w.n_kv * capacity * w.D * 2
    q_out = w.l * w.h * w.D * (2 + out_bytes)
    new_rows = 2 * w.n_kv * w.D * 2
    return cache + q_out + new_rows + 4


def capacity_batch(w: Workload, budget_bytes: int, capacity: int, out_bytes: int = 2) -> int:
    """The largest batch whose decode-step buffers fit in ``budget_bytes``."""
    return max(0, int(budget_bytes) // step_bytes_per_sequence(w, capacity, out_bytes))

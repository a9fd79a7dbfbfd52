"""The five workload shapes of the per-loop step (Ouro-like 16 heads x 128, 4-8 loops, 4K-32K context).

Budgets the paper gives as fractions (its loop-wise sparsity table, Appendix E) are turned into row
counts as k = floor(f * N + 0.5), at least 1 and never more than the previous loop's k (the active sets
are nested, Appendix D.1).  The column budget c of a layer is split into n_sink leading columns that are
always kept, a per-row causal band of `window` columns, and t = c - n_sink - window ranked columns.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int          # independent layers, each with its own seed stream
    loops: int           # R; loop 1 is dense, loops 2..R are sparse
    batch: int
    seq: int             # N prompt rows
    heads: int
    head_dim: int
    hot_frac: tuple      # per sparse loop r = 2..R: fraction of rows that get the large delta
    topk_frac: tuple     # per sparse loop r = 2..R: token budget as a fraction of N
    col_budget: int      # c = n_sink + window + t
    n_sink: int
    window: int
    bits: tuple          # residual bit width per sparse loop r = 2..R
    base_bits: int       # bit width of the loop-1 base
    group: int           # quantization group size G
    seed: int
    delta: str = "normal"     # "normal" (std hot_scale) or "student_t" (df, scale hot_scale)
    col_decay: tuple = ()     # optional per sparse loop r = 2..R: column budget c_r (c_2 = col_budget); a
                              # smaller budget prunes the list after the loop before (Section 4.2)
    tail: int = 0             # the most recent `tail` positions are stored exactly in bf16 (Appendix E: 64)
    hot_scale: float = 0.5
    cold_std: float = 0.01
    df: float = 3.0

    def __post_init__(self):
        nl = self.loops - 1
        if not (len(self.hot_frac) == len(self.topk_frac) == len(self.bits) == nl):
            raise ValueError(f"{self.name}: per-loop tuples must have R-1 = {nl} entries")
        if self.col_decay and (len(self.col_decay) != nl or self.col_decay[0] != self.col_budget):
            raise ValueError(f"{self.name}: col_decay needs R-1 = {nl} budgets starting at col_budget")

    # ---- derived sizes -------------------------------------------------------------------------
    def n_hot(self, r: int) -> int:
        """Rows of loop r (2..R) drawn from the large-delta distribution (nested across loops)."""
        n = self.seq
        for rr in range(2, r + 1):
            n = min(n, max(1, math.floor(self.hot_frac[rr - 2] * self.seq + 0.5)))
        return n

    def k(self, r: int) -> int:
        """Token budget k_r of sparse loop r (2..R), nested: k_r <= k_{r-1}, k_1 = N."""
        n = self.seq
        for rr in range(2, r + 1):
            n = min(n, max(1, math.floor(self.topk_frac[rr - 2] * self.seq + 0.5)))
        return n

    def bits_at(self, r: int) -> int:
        return self.bits[r - 2]

    @property
    def top_cols(self) -> int:
        """t: ranked columns beyond the sinks and the band, clamped to the available columns."""
        return max(0, min(self.col_budget - self.n_sink - self.window, self.seq - self.n_sink))

    def top_cols_at(self, r: int) -> int:
        """t_r of sparse loop r (2..R): ranked list entries under that loop's budget, never more than the
        loop before (pruned lists are nested)."""
        t = self.top_cols
        for rr in range(3, r + 1):
            if self.col_decay:
                t = min(t, max(0, min(self.col_decay[rr - 2] - self.n_sink - self.window, self.seq - self.n_sink)))
        return t

    @property
    def n_sink_eff(self) -> int:
        return min(self.n_sink, self.seq)

    @property
    def c_list(self) -> int:
        """Length of the per-(batch, head) column list: sinks plus ranked columns."""
        return self.n_sink_eff + self.top_cols

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _geom(a: float, b: float, n: int) -> tuple:
    """n fractions decaying geometrically from a to b (inclusive)."""
    if n == 1:
        return (a,)
    q = (b / a) ** (1.0 / (n - 1))
    return tuple(a * q ** t for t in range(n))


CONFIGS = {
    # Tiny: 1 layer, R=2, batch 1, seq 256, 2 heads x 64; 25 % hot rows; top-k 64; c = 32 (sink + top);
    # int4 residual, G = 32.
    "C1": Workload("C1-tiny", 1, 2, 1, 256, 2, 64,
                   hot_frac=(0.25,), topk_frac=(0.25,), col_budget=32, n_sink=4, window=0,
                   bits=(4,), base_bits=4, group=32, seed=0),
    # Ouro-1.4B-shaped single layer: R=4, seq 4096, 16 x 128; hot fraction halves each loop; top-k 10 %;
    # c = 512; int4 residual, G = 64.
    "C2": Workload("C2-ouro1.4b-4k", 1, 4, 1, 4096, 16, 128,
                   hot_frac=(0.10, 0.05, 0.025), topk_frac=(0.10, 0.10, 0.10), col_budget=512,
                   n_sink=4, window=0, bits=(4, 4, 4), base_bits=4, group=64, seed=1),
    # Ouro-2.6B-shaped stack: 48 layers x R=4, seq 8192; update fraction 15 % -> 3 % (geometric); c = 1024.
    "C3": Workload("C3-ouro2.6b-8k-48L", 48, 4, 1, 8192, 16, 128,
                   hot_frac=_geom(0.15, 0.03, 3), topk_frac=_geom(0.15, 0.03, 3), col_budget=1024,
                   n_sink=4, window=0, bits=(4, 4, 4), base_bits=4, group=64, seed=2),
    # Long-context prefill: R=4, seq 32768; 5 % hot rows; c = 2048 = sink + band 512 + ranked;
    # int2 residual (int4 base), G = 64.
    "C4": Workload("C4-long-32k", 1, 4, 1, 32768, 16, 128,
                   hot_frac=(0.05, 0.05, 0.05), topk_frac=(0.05, 0.05, 0.05), col_budget=2048,
                   n_sink=4, window=512, bits=(2, 2, 2), base_bits=4, group=64, seed=3),
    # Deep-loop batch: R=8, batch 4, seq 16384; update fraction 20 % -> 2 % geometric; c = 1024;
    # int4 for loops 2-3, int2 after; Student-t(df=3) x 0.3 deltas on updated rows.
    "C5": Workload("C5-deep-b4-16k", 1, 8, 4, 16384, 16, 128,
                   hot_frac=_geom(0.20, 0.02, 7), topk_frac=_geom(0.20, 0.02, 7), col_budget=1024,
                   n_sink=4, window=0, bits=(4, 4, 2, 2, 2, 2, 2), base_bits=4, group=64, seed=4,
                   delta="student_t", hot_scale=0.3),
}


def get(name: str) -> Workload:
    return CONFIGS[name]


def scaled(name: str, **kw) -> Workload:
    """A smaller variant of a named workload with the same structure (for parity at small sizes)."""
    w = CONFIGS[name]
    return w.replace(name=w.name + "-scaled", **kw)

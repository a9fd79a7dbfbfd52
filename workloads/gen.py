"""Seeded lazy-update states for one layer of a looped block.

Recipe (one layer, numpy PCG64 seeded with SeedSequence([seed, layer]), fixed draw order):

* loop 1: Q, K, V ~ N(0, 1) in fp32, rounded to bf16 (round to nearest even), layout [B, N, H, d];
* each sparse loop r = 2..R, for each batch element: a hot set T_r drawn without replacement from
  T_{r-1} (T_1 = all rows), so hot sets are nested like the paper's active sets (Section 3.1);
* then for Q, K, V in that order: a delta with std cold_std on every row, whose hot rows are redrawn from
  N(0, hot_scale) or hot_scale * Student-t(df); X^(r) = bf16(fp32(X^(r-1)) + delta).

Arrays hold raw bf16 bit patterns as uint16.  Nothing here scores, selects, quantizes or attends.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .configs import Workload


def _round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    out = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    return out


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class LoopStates:
    """Raw per-loop states of one layer; index 0 is loop 1."""
    workload: Workload
    layer: int
    q: list = field(default_factory=list)   # R arrays uint16 [B, N, H, d]
    k: list = field(default_factory=list)
    v: list = field(default_factory=list)
    hot: list = field(default_factory=list)  # per loop r>=2: list over batch of sorted int64 row ids

    def state(self, name: str, r: int) -> np.ndarray:
        """Raw state X^(r) (r is 1-based)."""
        return getattr(self, name)[r - 1]


def make_layer(w: Workload, layer: int = 0) -> LoopStates:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, layer])))
    shape = (w.batch, w.seq, w.heads, w.head_dim)
    out = LoopStates(w, layer)
    for name in ("q", "k", "v"):
        getattr(out, name).append(_round_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32)))
    prev_hot = [np.arange(w.seq, dtype=np.int64) for _ in range(w.batch)]
    for r in range(2, w.loops + 1):
        n_hot = w.n_hot(r)
        hot = []
        for b in range(w.batch):
            pick = rng.choice(prev_hot[b].size, size=n_hot, replace=False)
            hot.append(np.sort(prev_hot[b][pick]))
        out.hot.append(hot)
        prev_hot = hot
        for name in ("q", "k", "v"):
            delta = rng.standard_normal(shape, dtype=np.float32)
            delta *= np.float32(w.cold_std)
            for b in range(w.batch):
                hshape = (n_hot, w.heads, w.head_dim)
                if w.delta == "normal":
                    hd = rng.standard_normal(hshape, dtype=np.float32) * np.float32(w.hot_scale)
                elif w.delta == "student_t":
                    hd = (rng.standard_t(w.df, size=hshape) * w.hot_scale).astype(np.float32)
                else:
                    raise ValueError(w.delta)
                delta[b, hot[b]] = hd
            prev = _bf16_bits_to_f32(getattr(out, name)[-1])
            delta += prev
            getattr(out, name).append(_round_to_bf16_bits(delta))
            del delta, prev
    return out

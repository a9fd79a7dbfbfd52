"""The same lazy-update states as gen.make_layer, drawn on the GPU (for measurements only).

The host generator draws every state with numpy in a fixed order, which the CPU oracle and the parity
tests need bit for bit; at the 16K x 4 x 8-loop shape that takes minutes.  Throughput does not depend on
the particular values (the work of each call is set by the budgets), so the benchmark's secondary
workloads draw the same distributions on the device instead:

* loop 1: Q, K, V ~ N(0, 1) in fp32, rounded to bf16 (round to nearest even), layout [B, N, H, d];
* each sparse loop r = 2..R, per batch element: a hot set drawn without replacement from the previous one
  (nested), of the size gen.make_layer uses;
* Q, K, V deltas: std cold_std on every row, hot rows redrawn from N(0, hot_scale) or hot_scale * Student-t(df)
  (t = Z / sqrt(chi2_df / df), chi2_df a sum of df squared normals for integer df);
  X^(r) = bf16(fp32(X^(r-1)) + delta).

Seeded with torch's default device generator (seed, layer).  Nothing here scores, selects, quantizes or
attends.
"""
from __future__ import annotations

from .configs import Workload


def _student_t(torch, shape, df, device):
    z = torch.randn(shape, device=device)
    if float(df).is_integer():
        chi2 = torch.zeros(shape, device=device)
        for _ in range(int(df)):
            chi2 += torch.randn(shape, device=device) ** 2
    else:
        chi2 = torch.distributions.Chi2(torch.tensor(float(df), device=device)).sample(shape)
    return z / torch.sqrt(chi2 / df)


def make_layer_device(w: Workload, layer: int = 0, device="cuda"):
    """Dict name -> list over loops of bf16 tensors [B, N, H, d] on `device`."""
    import torch

    torch.cuda.manual_seed(w.seed * 1000003 + layer)
    shape = (w.batch, w.seq, w.heads, w.head_dim)
    out = {n: [torch.randn(shape, device=device).to(torch.bfloat16)] for n in "qkv"}
    prev_hot = [torch.arange(w.seq, device=device) for _ in range(w.batch)]
    for r in range(2, w.loops + 1):
        n_hot = w.n_hot(r)
        hot = []
        for b in range(w.batch):
            pick = torch.randperm(prev_hot[b].numel(), device=device)[:n_hot]
            hot.append(torch.sort(prev_hot[b][pick]).values)
        prev_hot = hot
        for name in "qkv":
            delta = torch.randn(shape, device=device) * w.cold_std
            for b in range(w.batch):
                hshape = (n_hot, w.heads, w.head_dim)
                if w.delta == "normal":
                    hd = torch.randn(hshape, device=device) * w.hot_scale
                elif w.delta == "student_t":
                    hd = _student_t(torch, hshape, w.df, device) * w.hot_scale
                else:
                    raise ValueError(w.delta)
                delta[b, hot[b]] = hd
            out[name].append((out[name][-1].float() + delta).to(torch.bfloat16))
            del delta
    return out

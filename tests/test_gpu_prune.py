"""GPU parity of the list pruning for a smaller budget (fl_prune_columns) against the oracle.

Both sides get the same state: bf16 queries and keys, ascending lists whose first entries are the sinks,
ascending updated rows, and fp32 reference log-normalisers (the fp64 row normalisers of a mass-corrected
loop rounded to fp32, as the state keeps them).  Keys: within one fp32 ulp of the oracle's fp64 statistic
rounded to fp32.  Bit-exact: the kept lists.  Shapes: several 128-entry workgroups with a ragged tail,
rows in several 32-row tiles with a ragged tail, rows before the first entry, budgets of none, some and
all entries, no updated rows, a list of sinks only.
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_keys_close, down, say, up_bf16
from oracle import attention as att
from oracle import prune
from oracle.numerics import bf16_to_f64, f32_to_bf16

pytestmark = pytest.mark.gpu


def _state(seed, B, N, H, d, ns, t_list, k):
    rng = np.random.default_rng(seed)
    q = f32_to_bf16(rng.standard_normal((B, N, H, d)).astype(np.float32))
    kc = f32_to_bf16(rng.standard_normal((B, N, H, d)).astype(np.float32))
    sc = 1.0 / np.sqrt(d)
    cols = np.zeros((B, H, ns + t_list), dtype=np.int32)
    rows = np.zeros((B, k), dtype=np.int32)
    lse = np.zeros((B, N, H), dtype=np.float32)
    for b in range(B):
        rows[b] = np.sort(rng.choice(N, k, replace=False))
        for h in range(H):
            cols[b, h] = att.select_columns(rng.random(N).astype(np.float32), ns, t_list)
            q64, k64 = bf16_to_f64(q[b, :, h]), bf16_to_f64(kc[b, :, h])
            for i in rows[b]:
                S = att.row_columns(cols[b, h], int(i), 32)
                lg = sc * (k64[S] @ q64[i])
                m = rng.uniform(0.3, 1.0)                     # a cached mass below 1
                lse[b, i, h] = lg.max() + np.log(np.exp(lg - lg.max()).sum()) - np.log(m)
    return q, kc, cols, rows, lse, sc


def _check(F, seed, B, N, H, d, ns, t_list, k, budgets):
    q, kc, cols, rows, lse, sc = _state(seed, B, N, H, d, ns, t_list, k)
    say(f"prune B={B} N={N} H={H} d={d} list={ns}+{t_list} rows={k} budgets={budgets}")
    dq, dk = up_bf16(q), up_bf16(kc)
    dcols = torch.from_numpy(cols).cuda()
    drows = torch.from_numpy(rows).cuda() if k > 0 else None
    dlse = torch.from_numpy(lse).cuda()
    for t in budgets:
        got_cols, got_key = F.prune_columns(dq, dk, drows, dcols, dlse, ns, t)
        torch.cuda.synchronize()
        got_cols, got_key = down(got_cols), down(got_key)
        for b in range(B):
            for h in range(H):
                stat = prune.column_mass(cols[b, h], rows[b], bf16_to_f64(q[b, :, h]), bf16_to_f64(kc[b, :, h]),
                                         lse[b, :, h].astype(np.float64), sc, ns)
                want = prune.prune_columns(cols[b, h], stat, ns, t)
                if t_list > 0:
                    assert_keys_close(got_key[b, h], stat.astype(np.float32), f"keys b={b} h={h}")
                assert np.array_equal(got_cols[b, h], want), f"kept list b={b} h={h} t={t}"


@pytest.mark.parametrize("d", [64, 128])
def test_prune_matches_oracle(F, d):
    # 333 entries after the sinks: three 128-entry workgroups, the last ragged; 150 rows: five 32-row tiles
    _check(F, seed=d, B=2, N=1200, H=2, d=d, ns=4, t_list=333, k=150, budgets=[200, 1, 333, 0])


def test_prune_edges(F):
    _check(F, seed=1, B=1, N=500, H=2, d=64, ns=4, t_list=60, k=0, budgets=[20])      # no updated rows
    _check(F, seed=2, B=1, N=300, H=1, d=128, ns=3, t_list=0, k=40, budgets=[0])      # sinks only
    _check(F, seed=3, B=1, N=4000, H=2, d=128, ns=4, t_list=1500, k=400, budgets=[1000])


def test_prune_32k_shape(F):
    # the 32K shape's list (4 sinks + 1532 ranked columns) shrinking to 1024 entries, 1638 updated rows,
    # checked on two of the 16 heads (the oracle statistic is O(rows x entries x d) per head)
    B, N, H, d, ns, t_list, k = 1, 32768, 16, 128, 4, 1532, 1638
    rng = np.random.default_rng(9)
    q = f32_to_bf16(rng.standard_normal((B, N, H, d)).astype(np.float32))
    kc = f32_to_bf16(rng.standard_normal((B, N, H, d)).astype(np.float32))
    sc = 1.0 / np.sqrt(d)
    rows = np.sort(rng.choice(N, k, replace=False)).astype(np.int32)[None]
    cols = np.stack([att.select_columns(rng.random(N).astype(np.float32), ns, t_list) for _ in range(H)])[None]
    lse = (rng.standard_normal((B, N, H)) * 0.5 + 4.0).astype(np.float32)   # plausible normalisers
    got_cols, got_key = F.prune_columns(up_bf16(q), up_bf16(kc), torch.from_numpy(rows).cuda(),
                                        torch.from_numpy(cols).cuda(), torch.from_numpy(lse).cuda(), ns, 1020)
    torch.cuda.synchronize()
    for h in (0, 11):
        stat = prune.column_mass(cols[0, h], rows[0], bf16_to_f64(q[0, :, h]), bf16_to_f64(kc[0, :, h]),
                                 lse[0, :, h].astype(np.float64), sc, ns)
        assert_keys_close(down(got_key)[0, h], stat.astype(np.float32), f"32K keys h={h}")
        assert np.array_equal(down(got_cols)[0, h], prune.prune_columns(cols[0, h], stat, ns, 1020)), f"32K h={h}"


def test_prune_rejects_bad_arguments(F):
    q = torch.zeros(1, 10, 2, 64, dtype=torch.bfloat16, device="cuda")
    cols = torch.arange(6, dtype=torch.int32, device="cuda").reshape(1, 1, 6).repeat(1, 2, 1)
    lse = torch.zeros(1, 10, 2, dtype=torch.float32, device="cuda")
    with pytest.raises(F.FlashLoopError, match="t_next"):
        F.prune_columns(q, q, None, cols, lse, 2, 5)

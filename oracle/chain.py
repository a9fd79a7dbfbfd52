"""One layer of a looped block end to end (test infrastructure only).

Loop 1 (dense source): base codec of K and V, dense causal attention over the reconstructed base, the
column statistic and the column list.  Sparse loops r = 2..R, in the order the paper describes them
(Section 4, Appendix D): select the active rows from the candidates of the previous loop (Eq. (5)),
quantize and reconstruct their K/V residuals (Eq. (8)), then apply the mass-corrected update to their
attention output (Eq. (7)).

The attention work is O(N^2 d) per head for loop 1, so large workloads can restrict it to some heads
(`heads`) and the per-loop update to some rows (`rows`); token selection and the codec always cover
every head and every row because they are cheap and their results feed all heads.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import attention as att
from . import codec
from . import prune
from . import select
from .numerics import bf16_to_f64


@dataclass
class LoopRecord:
    r: int
    keys: np.ndarray          # float32 [B, n_cand]
    idx: np.ndarray           # int32 [B, k]
    slot: np.ndarray          # int32 [B, N]
    enc_k: dict
    enc_v: dict
    k_new: np.ndarray         # uint16 [B, k, H, d] reconstructed rows of loop r
    v_new: np.ndarray
    o: dict                   # (b, h) -> float64 [N, d] after loop r (valid rows: see `valid`)
    lse: dict                 # (b, h) -> float64 [N]
    mass: dict                # (b, h) -> float64 [N] (nan where not updated)
    cols_next: dict = None    # (b, h) -> int32 list pruned after this loop for a smaller budget, if any
    stat_next: dict = None    # (b, h) -> float64 statistic of the non-sink entries that ranked cols_next


@dataclass
class LayerRecord:
    workload: object
    heads: list
    k_hat1: np.ndarray        # uint16 [B, N, H, d]
    v_hat1: np.ndarray
    enc_k1: dict
    enc_v1: dict
    o1: dict                  # (b, h) -> [N, d]
    lse1: dict                # (b, h) -> [N]
    colscore: dict            # (b, h) -> float64 [N]
    colkey: dict              # (b, h) -> float32 [N]
    cols: dict                # (b, h) -> int32 [c_list]
    loops: list = field(default_factory=list)
    k_hat: np.ndarray = None  # final reconstructions
    v_hat: np.ndarray = None


def _f64(x, b, h):
    return bf16_to_f64(x[b, :, h, :])


def loop1(states, heads=None, cols_only=False):
    """Base codec and the dense source loop for the listed heads (default: all)."""
    w = states.workload
    K1, V1, Q1 = states.k[0], states.v[0], states.q[0]
    enc_k = codec.quantize(K1, None, None, w.base_bits, w.group, codec.AXIS_TOKEN)
    k_hat, _ = codec.reconstruct(None, K1, None, enc_k, w.base_bits, w.group, codec.AXIS_TOKEN)
    enc_v = codec.quantize(V1, None, None, w.base_bits, w.group, codec.AXIS_CHANNEL)
    v_hat, _ = codec.reconstruct(None, V1, None, enc_v, w.base_bits, w.group, codec.AXIS_CHANNEL)
    k_hat, _ = codec.keep_recent(k_hat, None, K1, None, w.tail)
    v_hat, _ = codec.keep_recent(v_hat, None, V1, None, w.tail)
    heads = list(range(w.heads)) if heads is None else list(heads)
    rec = LayerRecord(w, heads, k_hat, v_hat, enc_k, enc_v, {}, {}, {}, {}, {})
    for b in range(w.batch):
        for h in heads:
            o, lse, cs = att.dense_loop(_f64(Q1, b, h), _f64(k_hat, b, h), _f64(v_hat, b, h), w.sm_scale)
            rec.o1[b, h] = o
            rec.lse1[b, h] = lse
            rec.colscore[b, h] = cs
            rec.colkey[b, h] = cs.astype(np.float32)
            rec.cols[b, h] = att.select_columns(rec.colkey[b, h], w.n_sink, w.top_cols)
    return rec


def sparse_loop(states, r, cand, k_hat, v_hat, cols, o, lse, heads, rows=None):
    """One sparse loop r >= 2.  o/lse are dicts (b, h) -> arrays, updated in place.

    rows: None (update every active row) or dict b -> row ids to evaluate (others are left stale).
    Returns (LoopRecord, k_hat_r, v_hat_r).
    """
    w = states.workload
    N = w.seq
    Kr, Kp = states.k[r - 1], states.k[r - 2]
    Vr, Vp = states.v[r - 1], states.v[r - 2]
    Qr, Qp = states.q[r - 1], states.q[r - 2]
    keys = select.token_keys([(Kr, Kp), (Vr, Vp)], cand)
    idx, slot = select.nested_topk(keys, cand, w.k(r), N)
    bits = w.bits_at(r)
    enc_k = codec.quantize(Kr, k_hat, idx, bits, w.group, codec.AXIS_TOKEN)
    k_hat_r, k_new = codec.reconstruct(k_hat, Kr, idx, enc_k, bits, w.group, codec.AXIS_TOKEN)
    enc_v = codec.quantize(Vr, v_hat, idx, bits, w.group, codec.AXIS_CHANNEL)
    v_hat_r, v_new = codec.reconstruct(v_hat, Vr, idx, enc_v, bits, w.group, codec.AXIS_CHANNEL)
    k_hat_r, k_new = codec.keep_recent(k_hat_r, k_new, Kr, idx, w.tail)
    v_hat_r, v_new = codec.keep_recent(v_hat_r, v_new, Vr, idx, w.tail)
    mass = {}
    for b in range(w.batch):
        active = idx[b].astype(np.int64)
        todo = active if rows is None else np.intersect1d(active, np.asarray(rows[b]))
        for h in heads:
            kp, vp = _f64(k_hat, b, h), _f64(v_hat, b, h)
            kc, vc = _f64(k_hat_r, b, h), _f64(v_hat_r, b, h)
            qc, qp = _f64(Qr, b, h), _f64(Qp, b, h)
            mrow = np.full(N, np.nan)
            for i in todo:
                S = att.row_columns(cols[b, h], int(i), w.window)
                o_new, l_new, m = att.correct_row(S, qc[i], qp[i], kp, vp, kc, vc,
                                                  lse[b, h][i], o[b, h][i], w.sm_scale)
                o[b, h][i] = o_new
                lse[b, h][i] = l_new
                mrow[i] = m
            mass[b, h] = mrow
    rec = LoopRecord(r, keys, idx, slot, enc_k, enc_v, k_new, v_new,
                     {key: val.copy() for key, val in o.items()},
                     {key: val.copy() for key, val in lse.items()}, mass)
    return rec, k_hat_r, v_hat_r


def run_layer(states, heads=None, rows=None, cols=None):
    """Loop 1 then sparse loops 2..R.  cols: optional dict (b, h) -> column list to use instead of the
    loop-1 selection (e.g. to evaluate the update alone with all columns).  With a decaying column budget
    (workload.col_decay) the lists are pruned between loops (recorded as LoopRecord.cols_next)."""
    w = states.workload
    rec = loop1(states, heads)
    if cols is not None:
        rec.cols = dict(cols)
    o = {key: val.copy() for key, val in rec.o1.items()}
    lse = {key: val.copy() for key, val in rec.lse1.items()}
    k_hat, v_hat = rec.k_hat1, rec.v_hat1
    cand = None
    cols_r = dict(rec.cols)
    for r in range(2, w.loops + 1):
        lr, k_hat, v_hat = sparse_loop(states, r, cand, k_hat, v_hat, cols_r, o, lse, rec.heads, rows)
        rec.loops.append(lr)
        cand = lr.idx
        if r < w.loops and w.top_cols_at(r + 1) < w.top_cols_at(r):
            # a smaller budget next loop: prune each list by this loop's statistic (Section 4.2), with the
            # reference log-normalisers as the state stores them (fp32)
            assert rows is None, "pruning needs every updated row's log-normaliser"
            lr.cols_next, lr.stat_next = {}, {}
            for b in range(w.batch):
                for h in rec.heads:
                    lse32 = lse[b, h].astype(np.float32).astype(np.float64)
                    stat = prune.column_mass(cols_r[b, h], lr.idx[b], _f64(states.q[r - 1], b, h),
                                             _f64(k_hat, b, h), lse32, w.sm_scale, w.n_sink)
                    lr.stat_next[b, h] = stat
                    lr.cols_next[b, h] = prune.prune_columns(cols_r[b, h], stat, w.n_sink, w.top_cols_at(r + 1))
            cols_r.update(lr.cols_next)
    rec.k_hat, rec.v_hat = k_hat, v_hat
    return rec

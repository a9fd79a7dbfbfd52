"""Attention parts of the per-loop step, for one (batch, head) at a time (test infrastructure only).

* dense_loop      Eq. (2) with a causal mask: softmax(q K^T / sqrt(d)) V for every row, its log-normaliser,
                  and the per-column probability mass accumulated over rows (the statistic the next loop
                  ranks columns by; Section 4.2, Appendix D.2, Eq. (6) with a dense source: all causal
                  keys, cached mass 1).
* select_columns  S = sinks U TopK_t of that statistic (Eq. (6)); ties by lower column index.
* row_columns     S_i = (S U band(i)) restricted to causal columns j <= i, as a set.
* correct_row     Eq. (7) (the mass-corrected form of Eq. (3)): o_i <- o_i - p^(r-1)_S V^(r-1)_S +
                  p^(r)_S V^(r)_S with p^(r)_S = m * softmax over S of the loop-r logits, where the loop-(r-1)
                  probabilities and their mass m are recovered from the cached row log-normaliser.

Readings (where the paper is silent):
* Appendix D.2 is written for one decode position; for a prefill of many rows the column statistic is
  the probability mass a column receives summed over all causal rows, in fp64.
* n_sink leading columns are always kept and a per-row causal band (i - w, i] is always recomputed;
  a column in both is counted once.
* the cached mass m is per (row, head) and is carried as the row's reference log-normaliser
  lse_ref = L - log(m), so that exp(logit - lse_ref) reproduces the cached probabilities next loop.
* an empty S_i, or m == 0, leaves the row unchanged.
* the dense loop attends over the quantized base K_hat^(1), V_hat^(1) (the hats of Eq. (6)).
Everything here is fp64.
"""
from __future__ import annotations

import numpy as np


def dense_loop(q, k, v, sm_scale, want_colscore=True, row_block=512):
    """Causal attention of every row over columns j <= i.

    q, k, v : float64 [N, d].  Returns (o [N, d], lse [N], colscore [N] or None).
    Rows are processed in blocks only to bound memory; each row is computed by the same formula.
    """
    N = q.shape[0]
    o = np.empty_like(q)
    lse = np.empty(N)
    colscore = np.zeros(N) if want_colscore else None
    for i0 in range(0, N, row_block):
        i1 = min(N, i0 + row_block)
        logits = sm_scale * (q[i0:i1] @ k[:i1].T)                  # [rows, i1]
        causal = np.arange(i1)[None, :] <= np.arange(i0, i1)[:, None]
        logits = np.where(causal, logits, -np.inf)
        mx = logits.max(axis=1, keepdims=True)
        l = mx[:, 0] + np.log(np.exp(logits - mx).sum(axis=1))
        p = np.exp(logits - l[:, None])
        o[i0:i1] = p @ v[:i1]
        lse[i0:i1] = l
        if want_colscore:
            colscore[:i1] += p.sum(axis=0)
    return o, lse, colscore


def dense_rows(q, k, v, rows, sm_scale):
    """Causal attention for selected rows only (same definition as dense_loop)."""
    o = np.empty((len(rows), q.shape[1]))
    lse = np.empty(len(rows))
    for n, i in enumerate(rows):
        logits = sm_scale * (k[:i + 1] @ q[i])
        mx = logits.max()
        l = mx + np.log(np.exp(logits - mx).sum())
        o[n] = np.exp(logits - l) @ v[:i + 1]
        lse[n] = l
    return o, lse


def select_columns(colkey, n_sink, t):
    """Column list of one (batch, head): sinks 0..n_sink-1 plus the top-t of the remaining columns by
    (key descending, column ascending), emitted ascending.  colkey: float32 [N]."""
    N = colkey.shape[0]
    ns = min(n_sink, N)
    ids = np.arange(ns, N)
    order = np.lexsort((ids, -colkey[ns:].astype(np.float64)))
    top = ids[order[:t]]
    return np.sort(np.concatenate([np.arange(ns), top])).astype(np.int32)


def row_columns(cols, i, window):
    """S_i: list columns and band columns (i - window, i], restricted to j <= i, as a sorted set."""
    lst = cols[cols <= i].astype(np.int64)
    if window > 0:
        band = np.arange(max(0, i - window + 1), i + 1, dtype=np.int64)
        return np.union1d(lst, band)
    return np.unique(lst)


def subtract_row(S, q_prev, k_prev, v_prev, lse_ref, sm_scale):
    """The subtract half of Eq. (7) for one row: the loop r-1 probabilities of the columns in S, recovered
    from the cached log-normaliser, their value-weighted sum and their mass.  Returns (sub [d], m)."""
    if S.size == 0:
        return np.zeros(v_prev.shape[1]), 0.0
    a = sm_scale * (k_prev[S] @ q_prev)
    pp = np.exp(a - lse_ref)                     # cached loop r-1 probabilities of the columns in S
    return pp @ v_prev[S], pp.sum()              # (their global mass m)


def correct_row(S, q_cur, q_prev, k_prev, v_prev, k_cur, v_cur, lse_ref, o_prev, sm_scale):
    """One row of Eq. (7).  Returns (o_new [d], lse_ref_new, m).

    k_prev/v_prev : loop r-1 reconstructions [N, d];  k_cur/v_cur : loop r reconstructions [N, d]
    """
    if S.size == 0:
        return o_prev.copy(), lse_ref, 0.0
    sub, m = subtract_row(S, q_prev, k_prev, v_prev, lse_ref, sm_scale)
    if m == 0.0:
        return o_prev.copy(), lse_ref, 0.0
    b = sm_scale * (k_cur[S] @ q_cur)
    bmax = b.max()
    L = bmax + np.log(np.exp(b - bmax).sum())
    pc = m * np.exp(b - L)                        # m * softmax over S
    add = pc @ v_cur[S]
    return o_prev - sub + add, L - np.log(m), m

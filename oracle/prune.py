"""Pruning of the column list between sparse loops when the column budget shrinks (test infrastructure
only).

Section 4.2 prunes the selected columns further when a later loop has a smaller budget, ranking them by
the attention statistics of the preceding sparse loop and carrying the kept columns and their mass on.
Appendix D.2, Eq. (6) is the rule for a sparse source: the loop's probabilities over its own columns,
p_j = exp(logit_j - lse_ref) with the cached mass folded into lse_ref, the top c' of them, and
m' = sum over the kept columns.

* column_mass    the statistic of each non-sink list entry j: the probability mass it receives in loop r,
                 summed over the rows updated in loop r that attend to it (i >= j), each row's
                 probabilities recovered from its reference log-normaliser.
* prune_columns  the n_sink leading entries, then the top t' of the other entries by fp32(statistic)
                 descending, ties to the lower column; emitted ascending (a subset of the list).

Readings (where the paper is silent):
* Appendix D.2 is written for one decode row; for a prefill the per-column statistic sums the rows, as the
  dense source statistic of the loop-1 set-up does (attention.dense_loop), over the rows updated in loop r
  (the only rows with loop-r probabilities).
* only the list is pruned; the per-row band (i - w, i] is always recomputed and is not part of the budget
  being pruned.
* the statistic uses the row's stored reference log-normaliser as given (the fp32 value the state keeps);
  the next loop's subtract pass recovers the kept mass m' = sum_{j in S'_i} p_j from the same lse_ref,
  so no other per-row value is carried (attention.correct_row).
Everything is fp64.
"""
from __future__ import annotations

import numpy as np


def column_mass(cols, rows, q, k, lse_ref, sm_scale, n_sink):
    """Statistic of the entries cols[ns:] (ns = min(n_sink, len(cols))) of one (batch, head).

    cols : ascending column list; rows : ascending updated rows; q, k : float64 [N, d] loop-r queries and
    reconstructed keys; lse_ref : float64 [N] (read at rows).  Returns float64 [len(cols) - ns].
    """
    ns = min(n_sink, len(cols))
    js = np.asarray(cols[ns:], dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    if js.size == 0 or rows.size == 0:
        return np.zeros(js.size)
    logits = sm_scale * (q[rows] @ k[js].T)                     # [rows, entries]
    p = np.exp(logits - lse_ref[rows][:, None])
    p = np.where(rows[:, None] >= js[None, :], p, 0.0)          # row i attends list column j iff j <= i
    return p.sum(axis=0)


def prune_columns(cols, stat, n_sink, t_next):
    """Sinks plus the top t_next of the other entries by (fp32(stat) descending, column ascending)."""
    ns = min(n_sink, len(cols))
    js = np.asarray(cols[ns:], dtype=np.int64)
    key = stat.astype(np.float32).astype(np.float64)
    order = np.lexsort((js, -key))
    keep = np.sort(js[order[:t_next]])
    return np.concatenate([np.asarray(cols[:ns], dtype=np.int64), keep]).astype(np.int32)

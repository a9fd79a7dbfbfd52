"""Decode step of one loop for the newest position, one (batch, head) (test infrastructure only).

Appendix D.2, Eqs. (6) and (7) are written for a single decode position:

* a dense source loop attends over every causal column with cached mass 1;
* loop r-1 ranks the columns it attended by their probabilities p^(r-1), keeps the top c^(r) as S,
  and caches their total probability m = sum_{j in S} p^(r-1)_j (Eq. (6));
* loop r recomputes the probabilities over S alone as m * softmax(q^(r) K_S^(r)T / sqrt(d)) and replaces
  the old contribution of S by the new one: o^(r) = o^(r-1) - p_S^(r-1) V_S^(r-1) + p_S^(r) V_S^(r)
  (Eq. (7));
* within loop r the new probabilities prepare the nested selection and mass for loop r+1.

decode_step carries the subtract term p_S^(r-1) V_S^(r-1) from the loop that selected S (it is formed
there, from the same probabilities and values), so a loop needs only its own state.

Readings (where the paper is silent):
* the selection keeps the n_sink leading columns and the `window` most recent ones, as the prefill
  path does (they rank above every other column; if the budget is smaller than their number, the lower
  columns win), then the highest probabilities, ties to the lower column; S is emitted ascending;
* within one row p_j = m * exp(l_j - L) increases with the logit l_j, so the top probabilities are the
  top logits: columns are ranked by the fp32 rounding of their fp64 logit (the GPU ranks the same fp32
  keys, formed before L is known);
* the decode position t = T - 1 is the last cached row and is causal for itself.
Everything is fp64.
"""
from __future__ import annotations

import numpy as np


def decode_step(q, k, v, S, m, sub, o_prev, sm_scale, n_sink, window, c_next):
    """One loop of the decode position.

    q : [d]; k, v : [T, d] this loop's reconstructions of columns 0..T-1; S : int array of the columns
    selected by the previous loop (ascending), or None for a dense source loop (every column, m = 1,
    and then sub and o_prev are ignored); m : cached mass of S; sub : [d] cached subtract term.
    Returns (o [d], S_next int32 [c_next] ascending, m_next, sub_next [d], L) with L the log-normaliser
    of the logits over S.
    """
    T = k.shape[0]
    dense = S is None
    if dense:
        S = np.arange(T)
        m = 1.0
    S = np.asarray(S, dtype=np.int64)
    logits = sm_scale * (k[S] @ q)
    top = logits.max()
    L = top + np.log(np.exp(logits - top).sum())
    p = m * np.exp(logits - L)                        # p_S^(r) = m * softmax over S
    add = p @ v[S]
    o = add if dense else o_prev - sub + add
    # next loop: forced columns first, then the logit (fp32) descending, then column ascending
    key = logits.astype(np.float32).astype(np.float64)
    forced = S < n_sink
    if window > 0:
        forced |= S >= T - window
    key = np.where(forced, np.inf, key)
    order = np.lexsort((S, -key))
    keep = np.sort(order[:c_next])                   # positions in S
    S_next = S[keep].astype(np.int32)
    m_next = p[keep].sum()
    sub_next = p[keep] @ v[S[keep]]
    return o, S_next, m_next, sub_next, L

"""Token scores and nested top-k selection (test infrastructure only).

Follows Section 4.1 and Appendix D.1, Eq. (5): a candidate row's score is the L2 norm of its cross-loop
change divided by the norm of the newer state plus a small epsilon; the active set of loop r is the
top-k_r of the scores over the previous loop's active set, so active sets are nested.

Readings (where the paper is silent):
* the state scored is the K and V rows of all heads together (the step's inputs; Eq. (5) writes the
  hidden state H, which would be the same computation with one pair instead of two);
* squares are summed in fp64 from fp32 differences of the bf16 states; the score is rounded once to an
  fp32 key, and both the oracle and the GPU take the top-k decision on that fp32 key;
* ties are broken by the lower row index; the active set is emitted in ascending row order;
* eps = 1e-6.
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_to_f32


def token_keys(pairs, cand=None, normalize=True, eps=1e-6):
    """fp32 selection keys, one per candidate row.

    pairs : list of (cur, prev) uint16 bf16 arrays, each [B, N, ...] (trailing dims flattened per row)
    cand  : None (all N rows) or int array [B, n_cand] of ascending row ids
    Returns float32 [B, n_cand].
    """
    B, N = pairs[0][0].shape[:2]
    n_cand = N if cand is None else np.asarray(cand).shape[1]
    keys = np.empty((B, n_cand), dtype=np.float32)
    for b in range(B):
        rows = np.arange(N) if cand is None else np.asarray(cand[b], dtype=np.int64)
        num = np.zeros(rows.size, dtype=np.float64)
        den = np.zeros(rows.size, dtype=np.float64)
        for cur, prev in pairs:
            c = bf16_to_f32(cur[b, rows].reshape(rows.size, -1))
            p = bf16_to_f32(prev[b, rows].reshape(rows.size, -1))
            delta = c - p                                   # fp32 difference, round to nearest even
            num += np.sum(delta.astype(np.float64) ** 2, axis=1)
            den += np.sum(c.astype(np.float64) ** 2, axis=1)
        s = np.sqrt(num) / (np.sqrt(den) + eps) if normalize else np.sqrt(num)
        keys[b] = s.astype(np.float32)
    return keys


def nested_topk(keys, cand, k, N):
    """A^(r) = TopK_k over the candidates, by (key descending, row id ascending).

    keys : float32 [B, n_cand];  cand : None (rows 0..N-1) or int [B, n_cand];  k <= n_cand.
    Returns (idx int32 [B, k] ascending, slot int32 [B, N] with slot[idx[p]] = p and -1 elsewhere).
    """
    B, n_cand = keys.shape
    if not 0 <= k <= n_cand:
        raise ValueError("k must lie in [0, n_cand]")
    idx = np.empty((B, k), dtype=np.int32)
    slot = np.full((B, N), -1, dtype=np.int32)
    for b in range(B):
        ids = np.arange(N) if cand is None else np.asarray(cand[b], dtype=np.int64)
        order = np.lexsort((ids, -keys[b].astype(np.float64)))   # primary: key desc; then id asc
        chosen = np.sort(ids[order[:k]])
        idx[b] = chosen
        slot[b, chosen] = np.arange(k, dtype=np.int32)
    return idx, slot

"""Host logic of bench.py: the algorithmic flop and byte counts of one attention launch, checked against
a brute-force construction of every S_i with the oracle's own set definition."""
import numpy as np

import bench
from oracle import attention as att


def test_attention_work_counts_match_brute_force():
    rng = np.random.default_rng(0)
    B, N, H, d, w = 2, 300, 3, 64, 17
    idx = np.stack([np.sort(rng.choice(N, 40, replace=False)) for _ in range(B)]).astype(np.int32)
    slot = np.full((B, N), -1, np.int32)
    for b in range(B):
        slot[b, idx[b]] = np.arange(40)
    cols = np.stack([np.stack([np.sort(np.concatenate([np.arange(4), rng.choice(np.arange(4, N), 30, replace=False)]))
                               for _ in range(H)]) for _ in range(B)]).astype(np.int32)
    nbytes, flops = bench.attn_work(idx, cols, slot, N, H, d, w, B)
    want_flops = 0
    want_bytes = 0
    for b in range(B):
        for h in range(H):
            used = set()
            for i in idx[b]:
                S = att.row_columns(cols[b, h], int(i), w)
                want_flops += 8 * d * S.size
                used |= set(S.tolist())
            n_new = sum(1 for j in used if slot[b, j] >= 0)
            want_bytes += (len(used) + n_new) * d * 4 + len(used) * 4 + cols.shape[2] * 4
        k = idx.shape[1]
        want_bytes += k * H * d * 4 + k * H * d * 8 + k * H * 8 + k * 4
    assert flops == want_flops
    assert nbytes == want_bytes

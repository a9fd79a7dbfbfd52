"""Host logic of bench.py: the algorithmic flop and byte counts of one attention launch (both passes, or
the add pass with stored subtract terms, reading new rows from the compact buffers or from the updated
caches), checked against a brute-force construction of every S_i with the oracle's own set definition."""
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
    for reuse, current in ((False, False), (True, False), (True, True)):
        check(idx, cols, slot, N, H, d, w, B, reuse, current)


def check(idx, cols, slot, N, H, d, w, B, reuse, current):
    nbytes, flops = bench.attn_work(idx, cols, slot, N, H, d, w, B, reuse=reuse, keep_terms=True, current=current)
    want_flops = 0
    want_bytes = 0
    for b in range(B):
        for h in range(H):
            used = set()
            for i in idx[b]:
                S = att.row_columns(cols[b, h], int(i), w)
                want_flops += (4 if reuse else 8) * d * S.size
                used |= set(S.tolist())
            n_new = 0 if current else sum(1 for j in used if slot[b, j] >= 0)
            slots = 0 if current else len(used) * 4
            want_bytes += (len(used) + n_new) * d * 4 + slots + cols.shape[2] * 4
        k = idx.shape[1]
        q_rows = 1 if reuse else 2
        lse_io = 1 if reuse else 2
        want_bytes += q_rows * k * H * d * 2 + k * H * d * 8 + lse_io * k * H * 4 + k * 4
        want_bytes += k * H * d * 4 + k * H * 4                              # terms kept
        if reuse:
            want_bytes += k * H * d * 4 + k * H * 4 + k * 4                  # previous terms read
    assert flops == want_flops
    assert nbytes == want_bytes


def test_prune_work_counts_match_brute_force():
    """fl_prune_columns: one d-long fp64 dot product per (updated row i, non-sink entry j) with i >= j."""
    rng = np.random.default_rng(1)
    B, N, H, d, ns = 2, 400, 3, 64, 4
    rows = np.stack([np.sort(rng.choice(N, 50, replace=False)) for _ in range(B)]).astype(np.int32)
    cols = np.stack([np.stack([np.concatenate([np.arange(ns), np.sort(rng.choice(np.arange(ns, N), 70, replace=False))])
                               for _ in range(H)]) for _ in range(B)]).astype(np.int32)
    nb, nf = bench.prune_work(rows, cols, ns, H, d)
    pairs = sum(1 for b in range(B) for h in range(H) for j in cols[b, h, ns:] for i in rows[b] if i >= j)
    assert nf == 2.0 * d * pairs
    assert nb == B * H * 70 * (2 * d + 4) + B * 50 * H * (2 * d + 4) + B * H * 74 * 8


def test_kv_footprint_matches_the_oracle_codec_outputs():
    # the packed footprint of a small workload equals the bytes of the codes and fp16 metadata the oracle's
    # codec actually produces for the base (all rows) and each sparse loop's active rows
    from oracle import codec
    from workloads import get, make_layer

    w = get("C1")
    st = make_layer(w)
    B, N, H, d = st.k[0].shape
    total = 0
    for axis in (codec.AXIS_TOKEN, codec.AXIS_CHANNEL):
        enc = codec.quantize(st.k[0], None, np.tile(np.arange(N, dtype=np.int32), (B, 1)), w.base_bits,
                             w.group, axis)
        total += enc["codes"].nbytes + enc["scale"].nbytes + enc["zero"].nbytes
    rng = np.random.default_rng(1)
    for r in range(2, w.loops + 1):
        k = w.k(r)
        idx = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
        for axis in (codec.AXIS_TOKEN, codec.AXIS_CHANNEL):
            enc = codec.quantize(st.k[r - 1], st.k[r - 2], idx, w.bits_at(r), w.group, axis)
            total += enc["codes"].nbytes + enc["scale"].nbytes + enc["zero"].nbytes
    fp = bench.kv_footprint(w)
    assert fp["packed_bytes"] == total
    assert fp["bf16_cache_per_loop_MB"] == round(w.loops * 2 * B * N * H * d * 2 / 1e6, 1)

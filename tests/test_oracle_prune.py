"""Pins of the oracle's list pruning (Section 4.2; Appendix D.2, Eq. (6) with a sparse source).

* with every row updated, the full list and the dense log-normalisers (mass 1), the statistic is the dense
  loop's per-column mass (attention.dense_loop, the loop-1 statistic);
* after a sparse loop over S_i (correct_row), the statistic of every entry summed equals the sum of the
  rows' masses m_i (each row's probabilities over S_i add up to its mass);
* pruned lists keep the sinks, are nested and ascending, and match a brute-force ranking (ties to the lower
  column);
* a loop over the pruned list with an unchanged state is the identity: the kept mass recovered from
  lse_ref in the subtract term equals the mass the add term spreads.
"""
import numpy as np

from oracle import attention as att
from oracle import prune
from oracle.numerics import bf16_to_f64, f32_to_bf16


def _rand(rng, *shape, scale=1.0):
    return bf16_to_f64(f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32)))


def test_full_rows_and_list_give_the_dense_statistic():
    rng = np.random.default_rng(0)
    N, d = 300, 32
    q, k, v = _rand(rng, N, d), _rand(rng, N, d), _rand(rng, N, d)
    sc = 1 / np.sqrt(d)
    _, lse, colscore = att.dense_loop(q, k, v, sc)
    cols = np.arange(N, dtype=np.int32)
    stat = prune.column_mass(cols, np.arange(N), q, k, lse, sc, n_sink=4)
    np.testing.assert_allclose(stat, colscore[4:], rtol=1e-11, atol=1e-14)


def test_statistic_sums_to_the_rows_masses():
    rng = np.random.default_rng(1)
    N, d = 400, 32
    sc = 1 / np.sqrt(d)
    q0, k0, v0 = _rand(rng, N, d), _rand(rng, N, d), _rand(rng, N, d)
    _, lse, colscore = att.dense_loop(q0, k0, v0, sc)
    cols = att.select_columns(colscore.astype(np.float32), 4, 60)
    q1, k1, v1 = q0 + _rand(rng, N, d, scale=0.3), k0 + _rand(rng, N, d, scale=0.3), v0 + _rand(rng, N, d)
    rows = np.sort(rng.choice(np.arange(10, N), 80, replace=False))
    lse1, masses = lse.copy(), []
    for i in rows:
        S = att.row_columns(cols, int(i), 0)
        _, lse1[i], m = att.correct_row(S, q1[i], q0[i], k0, v0, k1, v1, lse[i], np.zeros(d), sc)
        masses.append(m)
    stat = prune.column_mass(cols, rows, q1, k1, lse1, sc, n_sink=0)
    assert abs(stat.sum() - np.sum(masses)) < 1e-12 * len(rows)


def test_pruned_lists_are_nested_keep_sinks_and_rank_by_brute_force():
    rng = np.random.default_rng(2)
    cols = np.concatenate([np.arange(3), np.sort(rng.choice(np.arange(3, 500), 90, replace=False))]).astype(np.int32)
    stat = rng.random(90)
    stat[10] = stat[40] = stat[70] = stat[5]                # equal statistics: lower column first
    for t in (0, 1, 30, 90):
        out = prune.prune_columns(cols, stat, 3, t)
        assert out.tolist()[:3] == [0, 1, 2] and len(out) == 3 + t
        assert np.all(np.diff(out) > 0) and set(out.tolist()) <= set(cols.tolist())
        ranked = sorted(range(90), key=lambda e: (-float(np.float32(stat[e])), int(cols[3 + e])))[:t]
        assert out.tolist()[3:] == sorted(int(cols[3 + e]) for e in ranked)


def test_loop_over_the_pruned_list_with_an_unchanged_state_is_the_identity():
    rng = np.random.default_rng(3)
    N, d, w = 500, 32, 16
    sc = 1 / np.sqrt(d)
    q0, k0, v0 = _rand(rng, N, d), _rand(rng, N, d), _rand(rng, N, d)
    o, lse, colscore = att.dense_loop(q0, k0, v0, sc)
    cols = att.select_columns(colscore.astype(np.float32), 4, 120)
    q1, k1, v1 = q0 + _rand(rng, N, d, scale=0.3), k0 + _rand(rng, N, d, scale=0.3), v0 + _rand(rng, N, d, scale=0.3)
    rows = np.sort(rng.choice(np.arange(w, N), 60, replace=False))
    for i in rows:                                           # loop 2 over the full list
        S = att.row_columns(cols, int(i), w)
        o[i], lse[i], _ = att.correct_row(S, q1[i], q0[i], k0, v0, k1, v1, lse[i], o[i], sc)
    stat = prune.column_mass(cols, rows, q1, k1, lse, sc, n_sink=4)
    cols2 = prune.prune_columns(cols, stat, 4, 40)            # budget shrinks for loop 3
    for i in rows:                                           # loop 3 with the same state: no change
        S2 = att.row_columns(cols2, int(i), w)
        o3, lse3, m3 = att.correct_row(S2, q1[i], q1[i], k1, v1, k1, v1, lse[i], o[i], sc)
        np.testing.assert_allclose(o3, o[i], rtol=0, atol=1e-13)
        # the kept mass is the sum of the row's loop-2 probabilities over the pruned set
        assert abs(m3 - np.exp(sc * (k1[S2] @ q1[i]) - lse[i]).sum()) < 1e-14


def _brute_stat(cols, ns, rows, q, k, lse32, sc):
    """The statistic written out entry by entry: for list entry j, the sum over updated rows i >= j of
    exp(sc * q_i . k_j - lse_i) (a scalar loop, no shared helper)."""
    out = []
    for j in cols[ns:]:
        s = 0.0
        for i in rows:
            if i >= j:
                s += float(np.exp(sc * float(np.dot(q[i], k[j])) - lse32[i]))
        out.append(s)
    return np.array(out)


def test_run_layer_prunes_with_loop_r_queries_keys_and_stored_lse():
    """run_layer's pruning branch (Section 4.2) wired by hand: after sparse loop r the statistic uses loop
    r's queries Q^(r), its reconstructed keys K_hat^(r), and lse_ref after loop r as the state stores it
    (fp32); the list is then the sinks plus the top t_(r+1) entries by fp32 statistic, ties to the lower
    column.  The hand-wired chain advances with chain.loop1 / chain.sparse_loop (pinned elsewhere) and
    computes the statistic and ranking by brute force, so a wrong loop's queries or keys, an fp64
    log-normaliser, or a skipped pruning changes the statistic beyond the 1e-12 bound."""
    from oracle import chain
    from workloads import get, make_layer

    w = get("C5").replace(name="prune-wiring", batch=2, seq=160, heads=2, head_dim=32, loops=4,
                          hot_frac=(0.4, 0.3, 0.2), topk_frac=(0.45, 0.35, 0.25), col_budget=48, window=8,
                          col_decay=(48, 36, 24), bits=(4, 4, 2), group=16, delta="normal", hot_scale=0.5)
    st = make_layer(w)
    rec = chain.run_layer(st)
    # hand-wired chain
    ref = chain.loop1(st)
    o = {key: val.copy() for key, val in ref.o1.items()}
    lse = {key: val.copy() for key, val in ref.lse1.items()}
    k_hat, v_hat, cand, cols_r = ref.k_hat1, ref.v_hat1, None, dict(ref.cols)
    pruned = 0
    for r in range(2, w.loops + 1):
        lr, k_hat, v_hat = chain.sparse_loop(st, r, cand, k_hat, v_hat, cols_r, o, lse, ref.heads)
        got = rec.loops[r - 2]
        np.testing.assert_array_equal(got.idx, lr.idx)
        cand = lr.idx
        t_next = w.top_cols_at(r + 1) if r < w.loops else None
        if t_next is None or t_next >= w.top_cols_at(r):
            assert got.cols_next is None
            continue
        for b in range(w.batch):
            for h in ref.heads:
                q = bf16_to_f64(st.q[r - 1][b, :, h, :])
                kk = bf16_to_f64(k_hat[b, :, h, :])
                lse32 = lse[b, h].astype(np.float32).astype(np.float64)
                ns = min(w.n_sink, len(cols_r[b, h]))
                stat = _brute_stat(cols_r[b, h], ns, lr.idx[b], q, kk, lse32, w.sm_scale)
                np.testing.assert_allclose(got.stat_next[b, h], stat, rtol=1e-12, atol=1e-300)
                js = [int(j) for j in cols_r[b, h][ns:]]
                order = sorted(range(len(js)), key=lambda e: (-float(np.float32(stat[e])), js[e]))[:t_next]
                want = [int(j) for j in cols_r[b, h][:ns]] + sorted(js[e] for e in order)
                assert got.cols_next[b, h].tolist() == want
                cols_r[b, h] = np.asarray(want, dtype=np.int32)
                pruned += 1
    assert pruned == 2 * w.batch * w.heads
    # and the final outputs of both chains agree (the pruned lists were used by the loops after)
    for key in o:
        np.testing.assert_allclose(rec.loops[-1].o[key], o[key], rtol=0, atol=1e-12)

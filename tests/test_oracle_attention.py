"""Pins of the oracle's attention parts (Eqs. (2), (3), (6), (7); Sections 3.2, 4.2; Appendix D.2).

* the dense loop equals torch's scaled_dot_product_attention (causal, float64, CPU) and its
  log-normaliser equals scipy's logsumexp of the masked logits;
* each row's probabilities sum to one, so the column statistic sums to N;
* with every row active, every causal column selected and no quantization, the chained mass-corrected
  update reproduces exact dense attention of each loop (the correction subtracts the whole previous
  output and adds the whole new one);
* with unchanged states and a partial column set the update is the identity (checks the mass factor
  and the carried log-normaliser, which cancel only if both are right);
* with only V changing, the update is the closed form sum_S p_j (V^(r)_j - V^(r-1)_j);
* column selection and per-row column sets match brute force.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import attention as att
from oracle import chain
from oracle.numerics import bf16_to_f64, f32_to_bf16
from workloads import get, make_layer


def _sdpa(q, k, v):
    with torch.no_grad():
        out = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None],
            torch.from_numpy(v)[None, None], is_causal=True)
    return out[0, 0].numpy()


def _rand(rng, n, d):
    return bf16_to_f64(f32_to_bf16(rng.standard_normal((n, d)).astype(np.float32)))


def test_dense_loop_matches_sdpa_and_logsumexp():
    rng = np.random.default_rng(0)
    N, d = 300, 64
    q, k, v = (_rand(rng, N, d) for _ in range(3))
    o, lse, cs = att.dense_loop(q, k, v, 1 / np.sqrt(d), row_block=128)
    assert np.allclose(o, _sdpa(q, k, v), rtol=0, atol=1e-12)
    logits = (q @ k.T) / np.sqrt(d)
    logits[np.triu_indices(N, 1)] = -np.inf
    assert np.allclose(lse, logsumexp(logits, axis=1), rtol=0, atol=1e-12)
    assert abs(cs.sum() - N) < 1e-9
    o2, l2 = att.dense_rows(q, k, v, [0, 5, 299], 1 / np.sqrt(d))
    assert np.allclose(o2, o[[0, 5, 299]], atol=1e-12) and np.allclose(l2, lse[[0, 5, 299]], atol=1e-12)


def test_chain_with_all_rows_all_columns_no_quantization_is_exact_attention():
    w = get("C2").replace(seq=200, heads=2, head_dim=32, topk_frac=(1.0, 1.0, 1.0),
                          bits=(16, 16, 16), base_bits=16, group=32)
    st = make_layer(w)
    cols = {(0, h): np.arange(w.seq, dtype=np.int32) for h in range(w.heads)}
    rec = chain.run_layer(st, cols=cols)
    for lr in rec.loops:
        r = lr.r
        for h in range(w.heads):
            q, k, v = (bf16_to_f64(getattr(st, n)[r - 1][0, :, h, :]) for n in "qkv")
            want = _sdpa(q, k, v)
            assert np.max(np.abs(lr.o[0, h] - want)) < 1e-11, (r, h)
            assert np.nanmax(np.abs(lr.mass[0, h] - 1.0)) < 1e-12        # dense source: m = 1
            _, lse, _ = att.dense_loop(q, k, v, w.sm_scale)
            assert np.max(np.abs(lr.lse[0, h] - lse)) < 1e-11


def _one_head_inputs(seed, N=96, d=32):
    rng = np.random.default_rng(seed)
    q, k, v = (_rand(rng, N, d) for _ in range(3))
    o, lse, _ = att.dense_loop(q, k, v, 1 / np.sqrt(d))
    return rng, q, k, v, o, lse


def test_unchanged_states_with_partial_columns_leave_output_unchanged():
    rng, q, k, v, o, lse = _one_head_inputs(1)
    d = q.shape[1]
    cols = np.sort(rng.choice(96, 20, replace=False)).astype(np.int32)
    seen_partial = 0
    for i in range(96):
        S = att.row_columns(cols, i, 5)
        o_new, l_new, m = att.correct_row(S, q[i], q[i], k, v, k, v, lse[i], o[i], 1 / np.sqrt(d))
        assert np.max(np.abs(o_new - o[i])) < 1e-13 and abs(l_new - lse[i]) < 1e-12
        assert 0 < m <= 1 + 1e-12
        seen_partial += m < 1 - 1e-6
    assert seen_partial > 50


def test_value_only_change_is_the_closed_form():
    rng, q, k, v, o, lse = _one_head_inputs(2)
    d = q.shape[1]
    v2 = v + rng.standard_normal(v.shape) * 0.1
    cols = np.array([0, 1, 2, 3, 40, 41, 77], np.int32)
    for i in (10, 45, 80, 95):
        S = att.row_columns(cols, i, 3)
        o_new, l_new, m = att.correct_row(S, q[i], q[i], k, v, k, v2, lse[i], o[i], 1 / np.sqrt(d))
        p = np.exp((k[S] @ q[i]) / np.sqrt(d) - lse[i])
        want = o[i] + p @ (v2[S] - v[S])
        assert np.max(np.abs(o_new - want)) < 1e-13
        assert abs(l_new - lse[i]) < 1e-12


def test_mass_is_monotone_in_the_column_set_and_one_for_all_causal_columns():
    rng, q, k, v, o, lse = _one_head_inputs(3)
    d = q.shape[1]
    sc = 1 / np.sqrt(d)
    i = 90
    small = att.row_columns(np.array([0, 7, 50], np.int32), i, 0)
    big = att.row_columns(np.array([0, 7, 50, 60, 61], np.int32), i, 4)
    _, _, m_small = att.correct_row(small, q[i], q[i], k, v, k, v, lse[i], o[i], sc)
    _, _, m_big = att.correct_row(big, q[i], q[i], k, v, k, v, lse[i], o[i], sc)
    _, _, m_all = att.correct_row(np.arange(i + 1), q[i], q[i], k, v, k, v, lse[i], o[i], sc)
    assert 0 < m_small < m_big < m_all and abs(m_all - 1) < 1e-12
    empty = att.correct_row(np.array([], np.int64), q[i], q[i], k, v, k, v, lse[i], o[i], sc)
    assert np.array_equal(empty[0], o[i]) and empty[1] == lse[i]


def test_select_columns_and_row_sets_match_brute_force():
    rng = np.random.default_rng(4)
    N = 60
    key = rng.integers(0, 9, N).astype(np.float32)          # ties
    for n_sink, t in ((0, 10), (4, 10), (4, 56), (4, 0), (70, 5)):
        got = att.select_columns(key, n_sink, t).tolist()
        ns = min(n_sink, N)
        ranked = sorted(range(ns, N), key=lambda j: (-float(key[j]), j))[:t]
        assert got == sorted(list(range(ns)) + ranked)
    cols = np.array([0, 1, 2, 3, 20, 33, 34, 50], np.int32)
    for i in (0, 2, 21, 33, 40, 59):
        for w in (0, 1, 5, 100):
            want = sorted({j for j in cols.tolist() if j <= i} | {j for j in range(i - w + 1, i + 1) if j >= 0})
            assert att.row_columns(cols, i, w).tolist() == want


def test_tiny_workload_chain_runs_and_keeps_invariants():
    w = get("C1")
    st = make_layer(w)
    rec = chain.run_layer(st)
    lr = rec.loops[0]
    assert lr.idx.shape == (1, w.k(2))
    for h in range(w.heads):
        assert rec.cols[0, h].size == w.c_list
        assert np.array_equal(rec.cols[0, h][:4], np.arange(4))
        m = lr.mass[0, h][lr.idx[0]]
        assert np.all((m > 0) & (m <= 1 + 1e-12))
        untouched = np.setdiff1d(np.arange(w.seq), lr.idx[0])
        assert np.array_equal(lr.o[0, h][untouched], rec.o1[0, h][untouched])

"""Pins of the oracle's decode step (Appendix D.2, Eqs. (6) and (7) for one decode position).

* a dense step equals torch's scaled_dot_product_attention for the last row (float64, CPU) and its
  log-normaliser equals scipy's logsumexp of the logits;
* chaining loops that keep every column (c = T) reproduces, loop after loop, exact attention over each
  loop's new state: the subtract term removes the whole previous output and the mass stays 1;
* with an unchanged state and a partial column set the update is the identity (the cached mass and
  subtract term must both be right for the correction to cancel);
* with only V changing, the update is the closed form sum_S p_j (V^(r)_j - V^(r-1)_j);
* the selection keeps the sinks and the window, then matches a brute-force ranking by probability (ties
  to the lower column); it is nested and its mass is the sum of its probabilities.
"""
import numpy as np
import torch
from scipy.special import logsumexp

from oracle import decode as dec
from oracle.numerics import bf16_to_f64, f32_to_bf16


def _rand(rng, *shape, scale=1.0):
    return bf16_to_f64(f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32)))


def _sdpa_last(q, k, v):
    with torch.no_grad():
        out = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, None, None], torch.from_numpy(k)[None, None],
            torch.from_numpy(v)[None, None])
    return out[0, 0, 0].numpy()


def test_dense_step_matches_sdpa_and_logsumexp():
    rng = np.random.default_rng(0)
    T, d = 500, 64
    q, k, v = _rand(rng, d), _rand(rng, T, d), _rand(rng, T, d)
    sc = 1 / np.sqrt(d)
    o, S, m, sub, L = dec.decode_step(q, k, v, None, None, None, None, sc, 4, 32, 100)
    np.testing.assert_allclose(o, _sdpa_last(q, k, v), rtol=1e-12, atol=1e-13)
    assert abs(L - logsumexp(sc * (k @ q))) < 1e-12
    assert S.shape == (100,) and np.all(np.diff(S) > 0)


def test_keeping_every_column_reproduces_dense_attention_each_loop():
    rng = np.random.default_rng(1)
    T, d = 300, 32
    sc = 1 / np.sqrt(d)
    q, k, v = _rand(rng, d), _rand(rng, T, d), _rand(rng, T, d)
    o, S, m, sub, _ = dec.decode_step(q, k, v, None, None, None, None, sc, 0, 0, T)
    assert np.array_equal(S, np.arange(T)) and abs(m - 1.0) < 1e-12
    for _ in range(3):
        q = q + _rand(rng, d, scale=0.3)
        k = k + _rand(rng, T, d, scale=0.3)
        v = v + _rand(rng, T, d, scale=0.3)
        o, S, m, sub, _ = dec.decode_step(q, k, v, S, m, sub, o, sc, 0, 0, T)
        np.testing.assert_allclose(o, _sdpa_last(q, k, v), rtol=1e-10, atol=1e-12)
        assert abs(m - 1.0) < 1e-12


def test_unchanged_state_with_partial_columns_is_identity():
    rng = np.random.default_rng(2)
    T, d = 400, 64
    sc = 1 / np.sqrt(d)
    q, k, v = _rand(rng, d), _rand(rng, T, d), _rand(rng, T, d)
    o1, S, m, sub, _ = dec.decode_step(q, k, v, None, None, None, None, sc, 4, 16, 60)
    assert m < 1.0
    o2, S2, m2, sub2, _ = dec.decode_step(q, k, v, S, m, sub, o1, sc, 4, 16, 60)
    np.testing.assert_allclose(o2, o1, rtol=0, atol=1e-13)
    assert np.array_equal(S2, S) and abs(m2 - m) < 1e-13


def test_value_only_change_is_the_closed_form():
    rng = np.random.default_rng(3)
    T, d = 256, 32
    sc = 1 / np.sqrt(d)
    q, k, v = _rand(rng, d), _rand(rng, T, d), _rand(rng, T, d)
    o1, S, m, sub, _ = dec.decode_step(q, k, v, None, None, None, None, sc, 2, 8, 40)
    v2 = v + _rand(rng, T, d, scale=0.5)
    o2, _, _, _, _ = dec.decode_step(q, k, v2, S, m, sub, o1, sc, 2, 8, 40)
    logits = sc * (k @ q)
    p = np.exp(logits - logsumexp(logits))          # loop-1 probabilities, unchanged for S
    np.testing.assert_allclose(o2 - o1, p[S] @ (v2[S] - v[S]), rtol=1e-11, atol=1e-13)


def test_selection_forced_columns_ties_and_nesting():
    rng = np.random.default_rng(4)
    T, d = 200, 16
    sc = 1 / np.sqrt(d)
    q, k, v = _rand(rng, d), _rand(rng, T, d), _rand(rng, T, d)
    k[50] = k[120] = k[170] = k[10]                  # four columns with equal probabilities
    n_sink, window, c = 3, 5, 30
    o, S, m, sub, L = dec.decode_step(q, k, v, None, None, None, None, sc, n_sink, window, c)
    p = np.exp(sc * (k @ q) - L)
    forced = set(range(n_sink)) | set(range(T - window, T))
    assert forced <= set(S.tolist())
    rest = [j for j in range(T) if j not in forced]
    ranked = sorted(rest, key=lambda j: (-float(p[j]), j))[:c - len(forced)]   # brute force on the probabilities
    assert S.tolist() == sorted(forced | set(ranked))
    assert abs(m - p[S].sum()) < 1e-14 and m <= 1.0
    np.testing.assert_allclose(sub, p[S] @ v[S], rtol=1e-13)
    # nested: the next selection is a subset of S with a smaller mass
    q2 = q + _rand(rng, d, scale=0.2)
    _, S2, m2, _, _ = dec.decode_step(q2, k, v, S, m, sub, o, sc, n_sink, window, 12)
    assert set(S2.tolist()) <= set(S.tolist()) and len(S2) == 12 and m2 <= m + 1e-15
    assert (set(range(n_sink)) | set(range(T - window, T))) <= set(S2.tolist())
    # a budget below the forced count keeps the lower forced columns
    _, S3, _, _, _ = dec.decode_step(q2, k, v, S, m, sub, o, sc, n_sink, window, 5)
    assert S3.tolist() == [0, 1, 2, T - 5, T - 4]

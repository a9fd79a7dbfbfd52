"""Property tier of the oracle: random small shapes drawn by hypothesis, each checked against what the
definitions fix independently of the code under test (brute force, closed forms, invariants).

* selection (Appendix D.1, Eq. 5): the nested top-k equals a brute-force ranking by (key desc, row asc),
  emitted ascending, with a consistent slot map and nesting in the candidates;
* codec (Section 4.3, Eq. 4; Appendix D.3, Eq. 8): codes stay in range, the dequantized residual is within
  half a step (plus fp32 rounding slack) of the residual, the packed bytes unpack to the codes, and rows
  outside the active set keep their previous reconstruction;
* attention (Appendix D.2, Eqs. 6 and 7): after a dense loop, the subtract half over every causal column is
  the dense output with mass 1, a sparse loop over every causal column equals exact attention over the new
  state (the mass is 1), and over any column set the mass is the sum of the previous loop's probabilities of
  those columns;
* column lists: the sinks are kept, the list is ascending and of the budgeted size, and equals a brute-force
  ranking of the column keys.
"""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import attention as att
from oracle import codec, select
from oracle.numerics import bf16_to_f32, bf16_to_f64, f32_to_bf16

SETTINGS = settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def _bf16(rng, shape, scale=1.0):
    return f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32))


@SETTINGS
@given(seed=st.integers(0, 2**31 - 1), B=st.integers(1, 3), N=st.integers(1, 90), D=st.sampled_from([8, 16, 40]),
       frac=st.floats(0.0, 1.0), nested=st.booleans())
def test_selection_equals_brute_force_ranking(seed, B, N, D, frac, nested):
    rng = np.random.default_rng(seed)
    cur, prev = _bf16(rng, (B, N, D)), _bf16(rng, (B, N, D))
    if N > 3:                                             # a duplicated pair makes an exact tie
        cur[:, N - 1], prev[:, N - 1] = cur[:, 1], prev[:, 1]
    cand = None
    if nested:
        n_c = max(1, N // 2)
        cand = np.stack([np.sort(rng.choice(N, n_c, replace=False)) for _ in range(B)]).astype(np.int32)
    keys = select.token_keys([(cur, prev)], cand)
    n_cand = N if cand is None else cand.shape[1]
    k = int(round(frac * n_cand))
    idx, slot = select.nested_topk(keys, cand, k, N)
    for b in range(B):
        ids = np.arange(N) if cand is None else cand[b]
        ranked = sorted(range(n_cand), key=lambda p: (-float(keys[b, p]), int(ids[p])))[:k]
        want = sorted(int(ids[p]) for p in ranked)
        assert idx[b].tolist() == want
        assert set(want) <= set(ids.tolist())
        for p, i in enumerate(want):
            assert slot[b, i] == p
        assert int(np.sum(slot[b] >= 0)) == k


@SETTINGS
@given(seed=st.integers(0, 2**31 - 1), bits=st.sampled_from([2, 4, 8]), axis=st.sampled_from([0, 1]),
       G=st.sampled_from([8, 16, 32]), N=st.integers(1, 70), H=st.integers(1, 3), scale=st.floats(1e-3, 30.0))
def test_codec_error_bound_range_and_packing(seed, bits, axis, G, N, H, scale):
    rng = np.random.default_rng(seed)
    B, d = 2, 32
    x_ref = _bf16(rng, (B, N, H, d))
    x_cur = f32_to_bf16(bf16_to_f32(x_ref) + (rng.standard_normal((B, N, H, d)) * scale).astype(np.float32))
    k = int(rng.integers(0, N + 1))
    idx = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
    enc = codec.quantize(x_cur, x_ref, idx, bits, G, axis)
    q = enc["q"].astype(np.int64)
    assert q.min(initial=0) >= 0 and q.max(initial=0) <= (1 << bits) - 1
    np.testing.assert_array_equal(codec.unpack(enc["codes"], bits, d), enc["q"])
    dq = codec.dequantize(enc["codes"], enc["scale"], enc["zero"], bits, G, axis, d).astype(np.float64)
    s = codec._expand(enc["scale"], G, axis, k).astype(np.float64)
    z = codec._expand(enc["zero"], G, axis, k).astype(np.float64)
    err = np.abs(enc["delta"].astype(np.float64) - dq)
    bound = s / 2 + 2.0 ** -21 * (np.abs(z) + ((1 << bits) - 1) * s)
    assert np.all(err <= bound)
    x_hat, new_rows = codec.reconstruct(x_ref, x_cur, idx, enc, bits, G, axis)
    for b in range(B):
        rest = np.setdiff1d(np.arange(N), idx[b])
        np.testing.assert_array_equal(x_hat[b, rest], x_ref[b, rest])
        np.testing.assert_array_equal(x_hat[b, idx[b]], new_rows[b])


@SETTINGS
@given(seed=st.integers(0, 2**31 - 1), N=st.integers(2, 60), d=st.sampled_from([4, 8, 16]),
       window=st.integers(0, 12), n_list=st.integers(0, 20))
def test_sparse_loop_after_a_dense_loop(seed, N, d, window, n_list):
    rng = np.random.default_rng(seed)
    sc = 1.0 / np.sqrt(d)
    q0, k0, v0 = (bf16_to_f64(_bf16(rng, (N, d))) for _ in range(3))
    q1 = q0 + bf16_to_f64(_bf16(rng, (N, d), 0.4))
    k1 = k0 + bf16_to_f64(_bf16(rng, (N, d), 0.4))
    v1 = v0 + bf16_to_f64(_bf16(rng, (N, d), 0.4))
    o0, lse0, _ = att.dense_loop(q0, k0, v0, sc)
    # every causal column: the update reproduces exact attention over the new state, with mass 1
    full = np.arange(N, dtype=np.int32)
    want_o, want_lse = att.dense_rows(q1, k1, v1, np.arange(N), sc)
    for i in range(N):
        S = att.row_columns(full, i, 0)
        # the subtract half over every causal column is the dense loop's own output, with mass 1
        sub, m0 = att.subtract_row(S, q0[i], k0, v0, lse0[i], sc)
        np.testing.assert_allclose(sub, o0[i], rtol=0, atol=1e-12)
        assert abs(m0 - 1.0) < 1e-12
        o, lse, m = att.correct_row(S, q1[i], q0[i], k0, v0, k1, v1, lse0[i], o0[i], sc)
        assert abs(m - 1.0) < 1e-12
        np.testing.assert_allclose(o, want_o[i], rtol=0, atol=1e-11)
        assert abs(lse - want_lse[i]) < 1e-11
    # any column set: the mass is the sum of the previous loop's probabilities over S_i
    cols = np.sort(rng.choice(N, min(n_list, N), replace=False)).astype(np.int32)
    for i in range(N):
        S = att.row_columns(cols, i, window)
        _, _, m = att.correct_row(S, q1[i], q0[i], k0, v0, k1, v1, lse0[i], o0[i], sc)
        pp = np.exp(sc * (k0[S] @ q0[i]) - lse0[i]).sum() if S.size else 0.0
        assert abs(m - pp) <= 1e-12 * max(1.0, pp)
        assert m <= 1.0 + 1e-12


@SETTINGS
@given(seed=st.integers(0, 2**31 - 1), N=st.integers(1, 200), n_sink=st.integers(0, 6),
       tfrac=st.floats(0.0, 1.0), levels=st.integers(1, 6))
def test_column_list_equals_brute_force(seed, N, n_sink, tfrac, levels):
    rng = np.random.default_rng(seed)
    key = (rng.integers(0, levels, N) / levels).astype(np.float32)      # few distinct values: many ties
    ns = min(n_sink, N)
    t = int(round(tfrac * (N - ns)))
    cols = att.select_columns(key, n_sink, t)
    assert cols.tolist()[:ns] == list(range(ns))
    assert len(cols) == ns + t and np.all(np.diff(cols) > 0)
    ranked = sorted(range(ns, N), key=lambda j: (-float(key[j]), j))[:t]
    assert cols.tolist()[ns:] == sorted(ranked)

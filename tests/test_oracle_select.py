"""Pins of the oracle's token scoring and nested top-k (Section 4.1, Appendix D.1, Eq. (5)).

Each pin checks the oracle against something other than itself: a brute-force scalar computation on a
tiny input, planted hot rows that must be recovered, constructed exact ties, or a closed form.
"""
import math

import numpy as np
import pytest

from oracle import select
from oracle.numerics import f32_to_bf16
from workloads import get, make_layer


def _bf16(rng, shape, scale=1.0):
    return f32_to_bf16(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def _brute_key(curs, prevs, normalize=True, eps=1e-6):
    """Scalar loop: fp32 differences of the exact bf16 values, exactly rounded fp64 sums (math.fsum)."""
    sq, cc = [], []
    for cur, prev in zip(curs, prevs):
        for c_bits, p_bits in zip(cur.ravel(), prev.ravel()):
            c = np.float32(np.uint32(int(c_bits) << 16).view(np.float32))
            p = np.float32(np.uint32(int(p_bits) << 16).view(np.float32))
            dlt = float(np.float32(c - p))
            sq.append(dlt * dlt)
            cc.append(float(c) * float(c))
    num, den = math.fsum(sq), math.fsum(cc)
    s = math.sqrt(num) / (math.sqrt(den) + eps) if normalize else math.sqrt(num)
    return np.float32(s)


def test_keys_match_scalar_brute_force():
    rng = np.random.default_rng(11)
    B, N, H, d = 2, 12, 2, 8
    kc, kp, vc, vp = (_bf16(rng, (B, N, H, d)) for _ in range(4))
    keys = select.token_keys([(kc, kp), (vc, vp)])
    for b in range(B):
        for i in range(N):
            ref = _brute_key([kc[b, i], vc[b, i]], [kp[b, i], vp[b, i]])
            # the two fp64 sums are both within 1e-15 of exact; fp32 keys agree to one ulp at most
            assert abs(float(keys[b, i]) - float(ref)) <= float(np.spacing(ref))
    raw = select.token_keys([(kc, kp)], normalize=False)
    for i in range(N):
        assert abs(float(raw[0, i]) - float(_brute_key([kc[0, i]], [kp[0, i]], normalize=False))) \
            <= float(np.spacing(raw[0, i]))


def test_topk_matches_sorted_brute_force():
    rng = np.random.default_rng(5)
    B, N = 3, 40
    keys = rng.integers(0, 7, size=(B, N)).astype(np.float32)   # many exact ties
    for k in (0, 1, 7, 23, 40):
        idx, slot = select.nested_topk(keys, None, k, N)
        for b in range(B):
            want = sorted(sorted(range(N), key=lambda i: (-float(keys[b, i]), i))[:k])
            assert idx[b].tolist() == want
            assert [int(slot[b, i]) for i in want] == list(range(k))
            assert sum(1 for v in slot[b] if v >= 0) == k


def test_topk_with_candidates_and_ties_prefers_lower_index():
    N = 30
    cand = np.array([[2, 3, 5, 8, 13, 21, 29]])
    keys = np.array([[1.0, 3.0, 3.0, 2.0, 3.0, 0.5, 3.0]], dtype=np.float32)
    idx, slot = select.nested_topk(keys, cand, 3, N)
    assert idx.tolist() == [[3, 5, 13]]                # ties at 3.0 resolve to rows 3, 5, 13 (not 29)
    assert slot[0, 3] == 0 and slot[0, 5] == 1 and slot[0, 13] == 2 and slot[0, 29] == -1
    idx_all, _ = select.nested_topk(keys, cand, 7, N)
    assert idx_all.tolist() == cand.tolist()            # k = |C| returns C
    with pytest.raises(ValueError):
        select.nested_topk(keys, cand, 8, N)


def test_duplicated_rows_tie_exactly_and_lowest_index_wins():
    rng = np.random.default_rng(9)
    B, N, H, d = 1, 16, 2, 16
    cur = _bf16(rng, (B, N, H, d))
    prev = _bf16(rng, (B, N, H, d))
    cur[0, 9], prev[0, 9] = cur[0, 4], prev[0, 4]       # rows 4 and 9 identical -> identical keys
    keys = select.token_keys([(cur, prev)])
    assert keys[0, 4] == keys[0, 9]
    order = sorted(range(N), key=lambda i: (-float(keys[0, i]), i))
    k = order.index(4) + 1                              # cut right after row 4: row 9 must drop out
    idx, _ = select.nested_topk(keys, None, k, N)
    assert 4 in idx[0] and 9 not in idx[0]


def test_closed_form_unnormalized_score_is_delta_norm():
    rng = np.random.default_rng(3)
    cur = _bf16(rng, (1, 5, 3, 4))
    prev = cur.copy()
    c = np.float32(np.uint32(int(cur[0, 2, 1, 3]) << 16).view(np.float32))
    prev[0, 2, 1, 3] = f32_to_bf16(np.array([c - np.float32(0.75)], np.float32))[0]
    p = np.float32(np.uint32(int(prev[0, 2, 1, 3]) << 16).view(np.float32))
    keys = select.token_keys([(cur, prev)], normalize=False)
    assert keys[0, 0] == 0 and keys[0, 1] == 0 and keys[0, 3] == 0 and keys[0, 4] == 0
    # one changed element: the score is exactly |c - p| (the fp64 square root of a square)
    assert keys[0, 2] == np.float32(abs(float(c) - float(p))) and keys[0, 2] > 0


def test_planted_hot_rows_are_recovered_on_the_tiny_workload():
    w = get("C1")
    st = make_layer(w)
    keys = select.token_keys([(st.k[1], st.k[0]), (st.v[1], st.v[0])])
    idx, _ = select.nested_topk(keys, None, w.k(2), w.seq)
    # hot rows move by N(0, 0.5) per element, cold rows by N(0, 0.01): the top-k is the hot set
    assert idx[0].tolist() == st.hot[0][0].tolist()


def test_nested_selection_over_loops():
    w = get("C2").replace(seq=512, heads=2, head_dim=64)
    st = make_layer(w)
    cand = None
    prev = set(range(w.seq))
    for r in range(2, w.loops + 1):
        keys = select.token_keys([(st.k[r - 1], st.k[r - 2]), (st.v[r - 1], st.v[r - 2])], cand)
        idx, slot = select.nested_topk(keys, cand, w.k(r), w.seq)
        cur = set(idx[0].tolist())
        assert cur <= prev and len(cur) == w.k(r)
        assert np.all(np.diff(idx[0]) > 0)
        prev, cand = cur, idx

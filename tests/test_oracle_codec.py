"""Pins of the oracle's residual codec (Section 4.3, Eq. (4); Appendix D.3, Eq. (8); Appendix E).

Pins: directed fp16 rounding against an exhaustive table of every finite fp16 value; the half-step error
bound; exact grid values re-encoding to their own codes, scale and zero; a scalar brute force of the
grouping and metadata; hand-packed bytes; zero residuals; bits=16 as the identity; inactive rows
untouched.
"""
import bisect

import numpy as np
import pytest

from oracle import codec
from oracle.numerics import bf16_to_f32, bf16_to_f64, f16_down, f16_up, f32_to_bf16
from workloads import get, make_layer

# every finite binary16 value, ascending (as float64)
_ALL16 = np.unique(np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
                   .astype(np.float64))
_ALL16 = _ALL16[np.isfinite(_ALL16)]
_TABLE = _ALL16.tolist()


def _table_down(x):
    i = bisect.bisect_right(_TABLE, x) - 1
    return _TABLE[max(i, 0)]


def _table_up(x):
    i = bisect.bisect_left(_TABLE, x)
    return _TABLE[min(i, len(_TABLE) - 1)]


def test_directed_fp16_rounding_matches_exhaustive_table():
    rng = np.random.default_rng(0)
    xs = np.concatenate([
        rng.standard_normal(4000) * 10.0 ** rng.integers(-9, 5, 4000),      # many binades incl. subnormal
        _ALL16[rng.integers(0, _ALL16.size, 500)],                           # exact fp16 values
        (_ALL16[:-1] + np.diff(_ALL16) / 2)[rng.integers(0, _ALL16.size - 1, 500)],   # exact midpoints
        [0.0, -0.0, 6.0e-8, -6.0e-8, 65504.0, -65504.0, 65519.0, 1e-30, -1e-30],
    ])
    down = f16_down(xs).astype(np.float64)
    up = f16_up(xs).astype(np.float64)
    for x, dn, u in zip(xs.tolist(), down.tolist(), up.tolist()):
        assert dn == _table_down(x), x
        assert u == _table_up(x), x
    # zeros are stored as +0 whatever their sign (a stated reading)
    for z in (f16_down(np.array([0.0, -0.0])), f16_up(np.array([0.0, -0.0]))):
        assert z.view(np.uint16).tolist() == [0, 0]
    # saturation outside the fp16 range (a stated reading)
    assert float(f16_down(np.array([-1e6]))[0]) == -65504.0
    assert float(f16_up(np.array([1e6]))[0]) == 65504.0


def _residuals(rng, shape, scale):
    return (rng.standard_normal(shape) * scale).astype(np.float32)


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("axis", [codec.AXIS_TOKEN, codec.AXIS_CHANNEL])
def test_half_step_error_bound_and_code_range(bits, axis):
    rng = np.random.default_rng(bits * 10 + axis)
    delta = _residuals(rng, (2, 77, 3, 64), 0.3)            # k = 77: a partial last TOKEN group
    enc = codec.encode(delta, bits, 32, axis)
    assert enc["q"].max() <= (1 << bits) - 1
    dq = codec.dequantize(enc["codes"], enc["scale"], enc["zero"], bits, 32, axis, 64)
    s = codec._expand(enc["scale"], 32, axis, 77).astype(np.float64)
    z = codec._expand(enc["zero"], 32, axis, 77).astype(np.float64)
    err = np.abs(delta.astype(np.float64) - dq.astype(np.float64))
    slack = 2.0 ** -22 * (np.abs(delta) + np.abs(z) + np.abs(dq))
    assert np.all(err <= s / 2 + slack)
    # the grid covers the group: z <= min and z + qmax*s >= max
    mn, mx = codec.group_minmax(delta, 32, axis)
    assert np.all(enc["zero"].astype(np.float64) <= mn)
    assert np.all(enc["zero"].astype(np.float64) + ((1 << bits) - 1) * enc["scale"].astype(np.float64) >= mx)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_grid_values_reencode_exactly(bits):
    rng = np.random.default_rng(40 + bits)
    qmax = (1 << bits) - 1
    B, k, H, d, G = 1, 64, 2, 32, 32
    ng = d // G
    z = -rng.integers(0, 1024, (B, k, H, ng)) / 256.0             # multiples of 2^-8: exact fp16
    s = rng.integers(4, 64, (B, k, H, ng)) / 256.0
    q = rng.integers(0, qmax + 1, (B, k, H, d))
    q[..., 0::G] = 0                                              # every group holds its min ...
    q[..., 1::G] = qmax                                           # ... and its max
    zz = np.repeat(z, G, axis=3)
    ss = np.repeat(s, G, axis=3)
    delta = (zz + q * ss).astype(np.float32)                      # exact in fp32
    enc = codec.encode(delta, bits, G, codec.AXIS_CHANNEL)
    assert np.array_equal(enc["q"], q.astype(np.uint8))
    assert np.array_equal(enc["zero"].astype(np.float64), z)
    assert np.array_equal(enc["scale"].astype(np.float64), s)
    dq = codec.dequantize(enc["codes"], enc["scale"], enc["zero"], bits, G, codec.AXIS_CHANNEL, d)
    assert np.array_equal(dq, delta)


def test_zero_residual_gives_zero_codes_and_zero_update():
    x = f32_to_bf16(np.random.default_rng(1).standard_normal((1, 10, 2, 32)).astype(np.float32))
    idx = np.array([[1, 4, 7]])
    for axis in (codec.AXIS_TOKEN, codec.AXIS_CHANNEL):
        enc = codec.quantize(x, x, idx, 4, 32, axis)
        assert not enc["codes"].any() and not enc["scale"].astype(np.float64).any()
        assert not enc["zero"].astype(np.float64).any()
        x_hat, new = codec.reconstruct(x, x, idx, enc, 4, 32, axis)
        assert np.array_equal(x_hat, x)


def _scalar_encode(delta, bits, G, axis):
    """Pure-Python grouping + metadata + codes for a [k, d] slice (one batch, one head)."""
    k, d = delta.shape
    qmax = (1 << bits) - 1
    groups = ([[(p, e) for p in range(g, min(g + G, k))] for g in range(0, k, G) for e in range(d)]
              if axis == codec.AXIS_TOKEN else
              [[(p, e) for e in range(g, g + G)] for p in range(k) for g in range(0, d, G)])
    q = np.zeros((k, d), np.int64)
    meta = []
    for members in groups:
        vals = [float(delta[p, e]) for p, e in members]
        z = _table_down(min(vals))
        s = _table_up((max(vals) - z) / qmax)
        meta.append((z, s))
        for p, e in members:
            if s == 0.0:
                continue
            t = np.float32(np.float32(delta[p, e]) - np.float32(z)) / np.float32(s)
            q[p, e] = min(max(int(np.rint(t)), 0), qmax)
    return q, meta


@pytest.mark.parametrize("axis", [codec.AXIS_TOKEN, codec.AXIS_CHANNEL])
@pytest.mark.parametrize("bits", [2, 4])
def test_encode_matches_scalar_brute_force(axis, bits):
    rng = np.random.default_rng(7 + axis + bits)
    k, d, G = 11, 16, 4
    delta = _residuals(rng, (1, k, 1, d), 0.05)
    enc = codec.encode(delta, bits, G, axis)
    q, meta = _scalar_encode(delta[0, :, 0, :], bits, G, axis)
    assert np.array_equal(enc["q"][0, :, 0, :], q)
    if axis == codec.AXIS_TOKEN:
        got = [(float(enc["zero"][0, g, 0, e]), float(enc["scale"][0, g, 0, e]))
               for g in range(-(-k // G)) for e in range(d)]
    else:
        got = [(float(enc["zero"][0, p, 0, g]), float(enc["scale"][0, p, 0, g]))
               for p in range(k) for g in range(d // G)]
    assert got == meta


def test_packing_by_hand():
    q4 = np.array([[1, 2, 3, 0, 15, 7, 0, 9]], np.uint8)
    assert codec.pack(q4, 4).tolist() == [[0x21, 0x03, 0x7F, 0x90]]
    q2 = np.array([[1, 2, 3, 0, 3, 3, 3, 3]], np.uint8)
    assert codec.pack(q2, 2).tolist() == [[0x39, 0xFF]]
    rng = np.random.default_rng(2)
    for bits in (2, 4, 8):
        q = rng.integers(0, 1 << bits, (3, 5, 64)).astype(np.uint8)
        assert np.array_equal(codec.unpack(codec.pack(q, bits), bits, 64), q)


def test_bits16_is_the_identity_and_inactive_rows_are_untouched():
    w = get("C1")
    st = make_layer(w)
    idx = np.array([[3, 17, 100, 255]])
    x_prev = st.k[0]
    enc = codec.quantize(st.k[1], x_prev, idx, 16, 32, codec.AXIS_TOKEN)
    x_hat, new = codec.reconstruct(x_prev, st.k[1], idx, enc, 16, 32, codec.AXIS_TOKEN)
    assert np.array_equal(x_hat[0, idx[0]], st.k[1][0, idx[0]])
    enc4 = codec.quantize(st.k[1], x_prev, idx, 4, 32, codec.AXIS_TOKEN)
    x_hat4, new4 = codec.reconstruct(x_prev, st.k[1], idx, enc4, 4, 32, codec.AXIS_TOKEN)
    others = np.setdiff1d(np.arange(w.seq), idx[0])
    assert np.array_equal(x_hat4[0, others], x_prev[0, others])
    assert np.array_equal(x_hat4[0, idx[0]], new4[0])


def test_residual_coding_beats_full_state_coding_on_lazy_deltas():
    """Section 3.3 / Fig. 2(c): with small cross-loop deltas the residual codec reconstructs loop r
    better than quantizing the full loop-r state with the same scheme."""
    w = get("C1")
    st = make_layer(w)
    idx = np.arange(w.seq)[None, :]
    for name, axis in (("k", codec.AXIS_TOKEN), ("v", codec.AXIS_CHANNEL)):
        x1, x2 = getattr(st, name)[0], getattr(st, name)[1]
        e1 = codec.quantize(x1, None, None, 4, 32, axis)
        h1, _ = codec.reconstruct(None, x1, None, e1, 4, 32, axis)
        er = codec.quantize(x2, h1, idx, 4, 32, axis)
        hr, _ = codec.reconstruct(h1, x2, idx, er, 4, 32, axis)
        ef = codec.quantize(x2, None, None, 4, 32, axis)
        hf, _ = codec.reconstruct(None, x2, None, ef, 4, 32, axis)
        ref = bf16_to_f32(x2).astype(np.float64)
        err_res = np.linalg.norm(bf16_to_f32(hr) - ref)
        err_full = np.linalg.norm(bf16_to_f32(hf) - ref)
        assert err_res < err_full


def test_recent_tail_keeps_exact_rows_and_only_those():
    """Appendix E's bf16 tail: with tail = N and 4-bit codecs every stored row is exact, so the chain over
    all rows and columns is exact attention in every loop (as without quantization); with a 64-row tail
    the base codes are unchanged, the rows before the tail are the plain reconstructions, the tail rows
    are the exact inputs."""
    from oracle import attention as att
    from oracle import chain
    from workloads import get, make_layer
    w = get("C2").replace(seq=200, heads=2, head_dim=32, topk_frac=(1.0, 1.0, 1.0), bits=(4, 4, 4),
                          base_bits=4, group=32, tail=200)
    st = make_layer(w)
    cols = {(0, h): np.arange(w.seq, dtype=np.int32) for h in range(w.heads)}
    rec = chain.run_layer(st, cols=cols)
    for lr in rec.loops:
        for h in range(w.heads):
            q, k, v = (bf16_to_f64(getattr(st, n)[lr.r - 1][0, :, h, :]) for n in "qkv")
            o, _, _ = att.dense_loop(q, k, v, w.sm_scale, want_colscore=False)
            assert np.max(np.abs(lr.o[0, h] - o)) < 1e-11, (lr.r, h)
    w64 = get("C2").replace(seq=300, heads=2, head_dim=32, group=32, tail=64)
    st = make_layer(w64)
    with_tail = chain.loop1(st)
    without = chain.loop1(make_layer(w64.replace(tail=0)))
    assert np.array_equal(with_tail.enc_k1["codes"], without.enc_k1["codes"])
    assert np.array_equal(with_tail.k_hat1[:, :236], without.k_hat1[:, :236])
    assert np.array_equal(with_tail.k_hat1[:, 236:], st.k[0][:, 236:])
    assert np.array_equal(with_tail.v_hat1[:, 236:], st.v[0][:, 236:])
    assert not np.array_equal(without.k_hat1[:, 236:], st.k[0][:, 236:])

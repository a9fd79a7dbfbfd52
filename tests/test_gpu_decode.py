"""GPU parity of the decode step (fl_decode_step) against the oracle, over chained loops.

Each case runs a dense source loop and then sparse loops on both sides independently (the GPU chain
feeds itself its own selections, masses and subtract terms; the oracle chain its own), with the state
of every loop perturbed on a subset of positions.  Bit-exact: the selected columns of every loop.
Tolerance (max-abs 1e-2, relative Frobenius 2e-3 vs fp64): outputs, log-normalisers, masses and
subtract terms.  Shapes: several 128-position chunks with a ragged tail, ties in the probabilities,
budgets that keep everything, shrink, or stop; and the 32K shape.
"""
import numpy as np
import pytest
import torch

from gpu_util import assert_close, down, say, up, up_bf16
from oracle import decode as dec
from oracle.numerics import bf16_to_f64, f32_to_bf16

pytestmark = pytest.mark.gpu


def _bf16(rng, shape, scale=1.0):
    return f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32))


def _perturb(rng, x, frac, scale):
    """bf16 bits with a random fraction of positions (axis 1) moved by N(0, scale)."""
    B, T = x.shape[:2]
    y = bf16_to_f64(x).astype(np.float32)
    rows = rng.random((B, T)) < frac
    y[rows] += (rng.standard_normal(y[rows].shape) * scale).astype(np.float32)
    return f32_to_bf16(y)


def _run_chain(F, B, T, H, d, budgets, n_sink, window, seed, ties=False, check_heads=None):
    rng = np.random.default_rng(seed)
    q = _bf16(rng, (B, H, d))
    k = _bf16(rng, (B, T, H, d))
    v = _bf16(rng, (B, T, H, d))
    if ties:   # equal keys for a few positions give equal probabilities
        for j in (17, 300, 301, T - 40):
            k[:, j] = k[:, 5]
    sc = 1.0 / np.sqrt(d)
    heads = check_heads or [(b, h) for b in range(B) for h in range(H)]
    # GPU and oracle states
    o_d = torch.zeros(B, H, d, dtype=torch.float32, device="cuda")
    cols_d = mass_d = sub_d = None
    ost = {bh: dict(S=None, m=None, sub=None, o=None) for bh in heads}
    for loop, c_next in enumerate(budgets, start=1):
        if loop > 1:
            q = _perturb(rng, q[:, None], 1.0, 0.3)[:, 0]
            k = _perturb(rng, k, 0.2, 0.3)
            v = _perturb(rng, v, 0.2, 0.3)
        lse_d = torch.empty(B, H, dtype=torch.float32, device="cuda")
        nxt = F.decode_step(up_bf16(q), up_bf16(k), up_bf16(v), cols_d, mass_d, sub_d, o_d, c_next,
                            n_sink=n_sink, window=window, lse=lse_d)
        torch.cuda.synchronize()
        go, glse = down(o_d), down(lse_d)
        want_o, want_l = [], []
        got_o, got_l = [], []
        for (b, h) in heads:
            st = ost[(b, h)]
            o, S, m, sub, L = dec.decode_step(bf16_to_f64(q[b, h]), bf16_to_f64(k[b, :, h]), bf16_to_f64(v[b, :, h]),
                                              st["S"], st["m"], st["sub"], st["o"], sc, n_sink, window, c_next)
            want_o.append(o)
            want_l.append(L)
            got_o.append(go[b, h])
            got_l.append(glse[b, h])
            if c_next > 0:
                assert np.array_equal(down(nxt[0])[b, h], S), f"loop {loop} selection b={b} h={h}"
                assert_close(down(nxt[1])[b, h], m, f"loop {loop} mass b={b} h={h}")
                assert_close(down(nxt[2])[b, h], sub, f"loop {loop} subtract term b={b} h={h}")
            st.update(S=S, m=m, sub=sub, o=o)
        assert_close(np.array(got_o), np.array(want_o), f"loop {loop} output")
        assert_close(np.array(got_l), np.array(want_l), f"loop {loop} log-normaliser")
        cols_d, mass_d, sub_d = nxt
        if c_next == 0:
            break
        say(f"  loop {loop}: {c_next} columns kept")


@pytest.mark.parametrize("d", [64, 128])
def test_decode_chain_small(F, d):
    # T = 700: six chunks, the last ragged; budgets shrink, keep all of S, then stop
    _run_chain(F, B=2, T=700, H=3, d=d, budgets=[180, 120, 120, 37, 0], n_sink=4, window=32, seed=d, ties=True)


def test_decode_edges(F):
    # a single position; forced columns beyond the budget; a window wider than the context
    _run_chain(F, B=1, T=1, H=2, d=64, budgets=[1, 1, 0], n_sink=4, window=8, seed=1)
    _run_chain(F, B=1, T=300, H=2, d=64, budgets=[6, 3, 0], n_sink=4, window=8, seed=2)
    _run_chain(F, B=1, T=90, H=1, d=128, budgets=[90, 90, 20], n_sink=2, window=500, seed=3)


def test_decode_chain_32k(F):
    # the 32K shape: dense loop over 32768 positions, then loops over 2048 columns (sinks 4, window 512)
    _run_chain(F, B=1, T=32768, H=16, d=128, budgets=[2048, 2048, 2048, 1024], n_sink=4, window=512, seed=7,
               check_heads=[(0, h) for h in (0, 5, 15)])


def test_decode_rejects_bad_arguments(F):
    q = torch.zeros(1, 2, 64, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(1, 10, 2, 64, dtype=torch.bfloat16, device="cuda")
    o = torch.zeros(1, 2, 64, dtype=torch.float32, device="cuda")
    with pytest.raises(F.FlashLoopError, match="c_next"):
        F.decode_step(q, kc, kc, None, None, None, o, 11)
    cols = torch.zeros(1, 2, 3, dtype=torch.int32, device="cuda")
    with pytest.raises(F.FlashLoopError, match="mass"):
        F.decode_step(q, kc, kc, cols, None, None, o, 2)

"""GPU parity of every call of the C ABI against the CPU oracle, at sizes the oracle finishes in seconds.

Bit-exact: token keys' top-k indices and slots (keys themselves within one fp32 ulp), residual codes,
fp16 scale/zero bit patterns, reconstructed bf16 rows and caches, column lists.  Tolerance (max-abs
1e-2, relative Frobenius 2e-3 vs fp64): attention outputs and log-normalisers.
Shapes span several tiles with ragged tails (row tiles of 32, column tiles of 32, groups of 32/64).
"""
import numpy as np
import pytest
import torch

from gpu_util import (assert_close, assert_keys_close, down, down_bits16, f16_bits, new_rows, say, up, up_bf16)
from oracle import attention as att
from oracle import chain, codec, select
from oracle.numerics import bf16_to_f64, f32_to_bf16
from workloads import get, make_layer

pytestmark = pytest.mark.gpu


def _bf16(rng, shape, scale=1.0):
    return f32_to_bf16((rng.standard_normal(shape) * scale).astype(np.float32))


# ---------------------------------------------------------------------------------------------------
SELECT_CASES = [("C1", {}), ("C2", dict(seq=3000, heads=4)),
                ("C5", dict(seq=2500, heads=2, batch=3, col_budget=200))]


@pytest.mark.parametrize("name,over", SELECT_CASES)
def test_select_tokens_over_loops(F, name, over):
    w = get(name).replace(**over)
    st = make_layer(w)
    say(f"select {w.name} B={w.batch} N={w.seq} H={w.heads}")
    cand = None
    for r in range(2, w.loops + 1):
        pairs = [(st.k[r - 1], st.k[r - 2]), (st.v[r - 1], st.v[r - 2])]
        want_key = select.token_keys(pairs, cand)
        want_idx, want_slot = select.nested_topk(want_key, cand, w.k(r), w.seq)
        idx, slot, key = F.select_tokens(up_bf16(st.k[r - 1]), up_bf16(st.k[r - 2]), up_bf16(st.v[r - 1]),
                                         up_bf16(st.v[r - 2]), w.k(r),
                                         cand=None if cand is None else up(cand))
        torch.cuda.synchronize()
        assert_keys_close(down(key), want_key, f"loop {r} keys")
        assert np.array_equal(down(idx), want_idx), f"loop {r}: active rows differ"
        assert np.array_equal(down(slot), want_slot), f"loop {r}: slot map differs"
        cand = want_idx


def test_select_tokens_ties_edges_and_one_pair(F):
    rng = np.random.default_rng(21)
    B, N, H, d = 2, 700, 2, 64
    cur, prev = _bf16(rng, (B, N, H, d)), _bf16(rng, (B, N, H, d))
    for dup in (5, 40, 41, 300, 699):            # exact ties with row 3 / row 200
        src = 3 if dup < 200 else 200
        cur[:, dup], prev[:, dup] = cur[:, src], prev[:, src]
    dc, dp = up_bf16(cur), up_bf16(prev)
    for k in (0, 1, 2, 37, 350, 699, 700):
        want_key = select.token_keys([(cur, prev)])
        want_idx, want_slot = select.nested_topk(want_key, None, k, N)
        idx, slot, key = F.select_tokens(dc, dp, None, None, k)
        torch.cuda.synchronize()
        assert np.array_equal(down(idx), want_idx), k
        assert np.array_equal(down(slot), want_slot), k
    # unnormalized scores
    want_key = select.token_keys([(cur, prev)], normalize=False)
    _, _, key = F.select_tokens(dc, dp, None, None, 10, normalize=False)
    assert_keys_close(down(key), want_key, "unnormalized keys")


def test_select_tokens_on_hidden_states(F):
    """Eq. (5) scored on the layer's hidden states instead of K and V: one pair of [B, N, D_model] states
    (D_model = 2048, the 16 x 128 model width), two nested loops (candidates = the previous selection)."""
    rng = np.random.default_rng(22)
    B, N, Dm = 2, 3000, 2048
    h0, h1, h2 = (_bf16(rng, (B, N, Dm)) for _ in range(3))
    idx_prev = None
    for (cur, prev), k in (((h1, h0), 900), ((h2, h1), 300)):
        want_key = select.token_keys([(cur, prev)], idx_prev)
        want_idx, want_slot = select.nested_topk(want_key, idx_prev, k, N)
        cand = None if idx_prev is None else torch.from_numpy(idx_prev).cuda()
        idx, slot, key = F.select_tokens(up_bf16(cur), up_bf16(prev), None, None, k, cand=cand)
        torch.cuda.synchronize()
        assert_keys_close(down(key), want_key, f"hidden-state keys k={k}")
        assert np.array_equal(down(idx), want_idx), k
        assert np.array_equal(down(slot), want_slot), k
        idx_prev = want_idx


# ---------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [2, 4, 8, 16])
@pytest.mark.parametrize("axis", [codec.AXIS_TOKEN, codec.AXIS_CHANNEL])
@pytest.mark.parametrize("d,G", [(64, 32), (128, 64)])
def test_codec_matches_oracle(F, bits, axis, d, G):
    rng = np.random.default_rng(bits * 100 + axis * 10 + d)
    B, N, H, k = 2, 300, 3, 150                    # 150 = 2*64 + 22: a partial last TOKEN group
    ref = _bf16(rng, (B, N, H, d))
    cur = f32_to_bf16(bf16_to_f64(ref).astype(np.float32) + (rng.standard_normal((B, N, H, d)) * 0.05)
                      .astype(np.float32))
    idx = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
    enc = codec.quantize(cur, ref, idx, bits, G, axis)
    x_hat, want_rows = codec.reconstruct(ref, cur, idx, enc, bits, G, axis)
    d_ref = up_bf16(ref)
    codes, scale, zero, rows = F.kv_residual_quant(up_bf16(cur), d_ref, up(idx), bits, G, axis)
    torch.cuda.synchronize()
    assert np.array_equal(down(codes), enc["codes"]), "codes differ"
    if bits != 16:
        assert np.array_equal(down(scale).view(np.uint16), f16_bits(enc["scale"])), "scale differs"
        assert np.array_equal(down(zero).view(np.uint16), f16_bits(enc["zero"])), "zero differs"
    assert np.array_equal(down_bits16(rows), want_rows), "reconstructed rows differ"
    compact = F.kv_residual_dequant(codes, scale, zero, up(idx), bits, G, axis, d_ref, mode=F.DQ_COMPACT)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(compact), want_rows), "COMPACT dequant differs"
    F.kv_residual_dequant(codes, scale, zero, up(idx), bits, G, axis, d_ref, mode=F.DQ_COMMIT)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(d_ref), x_hat), "COMMIT dequant differs"
    # quantize and commit in one pass: same codes and metadata, the cache updated in place
    d_hat = up_bf16(ref)
    codes2, scale2, zero2 = F.kv_residual_quant_commit(up_bf16(cur), d_hat, up(idx), bits, G, axis)
    torch.cuda.synchronize()
    assert np.array_equal(down(codes2), enc["codes"]), "fused commit: codes differ"
    if bits != 16:
        assert np.array_equal(down(scale2).view(np.uint16), f16_bits(enc["scale"])), "fused commit: scale differs"
        assert np.array_equal(down(zero2).view(np.uint16), f16_bits(enc["zero"])), "fused commit: zero differs"
    assert np.array_equal(down_bits16(d_hat), x_hat), "fused commit: cache differs"


def _check_enc(got, enc, bits, what):
    codes, scale, zero = got[:3]
    assert np.array_equal(down(codes), enc["codes"]), f"{what}: codes differ"
    if bits != 16:
        assert np.array_equal(down(scale).view(np.uint16), f16_bits(enc["scale"])), f"{what}: scale differs"
        assert np.array_equal(down(zero).view(np.uint16), f16_bits(enc["zero"])), f"{what}: zero differs"


@pytest.mark.parametrize("bits", [2, 4, 8, 16])
@pytest.mark.parametrize("d,G,k", [(64, 8, 77), (64, 16, 150), (64, 32, 1), (128, 64, 150), (128, 128, 300)])
def test_codec_kv_pair_matches_oracle(F, bits, d, G, k):
    """Keys on the token axis and values on the channel axis in one launch, compact and committed."""
    rng = np.random.default_rng(bits * 1000 + d + G + k)
    B, N, H = 2, 300, 3
    kref, vref = _bf16(rng, (B, N, H, d)), _bf16(rng, (B, N, H, d))
    step = lambda x: f32_to_bf16(bf16_to_f64(x).astype(np.float32)
                                 + (rng.standard_normal((B, N, H, d)) * 0.05).astype(np.float32))
    kcur, vcur = step(kref), step(vref)
    idx = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
    want = {}
    for name, cur, ref, axis in (("k", kcur, kref, codec.AXIS_TOKEN), ("v", vcur, vref, codec.AXIS_CHANNEL)):
        enc = codec.quantize(cur, ref, idx, bits, G, axis)
        want[name] = (enc,) + tuple(codec.reconstruct(ref, cur, idx, enc, bits, G, axis))
    dk, dv = up_bf16(kref), up_bf16(vref)
    ko, vo = F.kv_residual_quant_kv(up_bf16(kcur), dk, up_bf16(vcur), dv, up(idx), bits, G)
    torch.cuda.synchronize()
    for name, got in (("k", ko), ("v", vo)):
        enc, _, rows = want[name]
        _check_enc(got, enc, bits, f"pair {name}")
        assert np.array_equal(down_bits16(got[3]), rows), f"pair {name}: reconstructed rows differ"
    assert np.array_equal(down_bits16(dk), kref) and np.array_equal(down_bits16(dv), vref), "COMPACT wrote refs"
    ko, vo = F.kv_residual_quant_kv(up_bf16(kcur), dk, up_bf16(vcur), dv, up(idx), bits, G, rows=False)
    torch.cuda.synchronize()
    assert ko[3] is None and vo[3] is None
    _check_enc(ko, want["k"][0], bits, "pair k (no rows)")
    _check_enc(vo, want["v"][0], bits, "pair v (no rows)")
    # the pair reconstruction from those codes: compact rows, then committed in place
    kr_, vr_ = F.kv_residual_dequant_kv(ko[:3], vo[:3], up(idx), bits, G, dk, dv)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(kr_), want["k"][2]), "pair dequant: key rows differ"
    assert np.array_equal(down_bits16(vr_), want["v"][2]), "pair dequant: value rows differ"
    dk2, dv2 = up_bf16(kref), up_bf16(vref)
    F.kv_residual_dequant_kv(ko[:3], vo[:3], up(idx), bits, G, dk2, dv2, mode=F.DQ_COMMIT)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(dk2), want["k"][1]), "pair dequant commit: key cache differs"
    assert np.array_equal(down_bits16(dv2), want["v"][1]), "pair dequant commit: value cache differs"
    ko, vo = F.kv_residual_quant_kv(up_bf16(kcur), dk, up_bf16(vcur), dv, up(idx), bits, G, mode=F.DQ_COMMIT)
    torch.cuda.synchronize()
    _check_enc(ko, want["k"][0], bits, "pair commit k")
    _check_enc(vo, want["v"][0], bits, "pair commit v")
    assert np.array_equal(down_bits16(dk), want["k"][1]), "pair commit: key cache differs"
    assert np.array_equal(down_bits16(dv), want["v"][1]), "pair commit: value cache differs"


def test_keep_recent_matches_oracle(F):
    """fl_kv_keep_recent against codec.keep_recent: tails longer and shorter than the active set, rows with
    no active tail row, every row (idx = NULL), the caches and the compact rows, tail = 0."""
    rng = np.random.default_rng(31)
    B, N, H, d = 2, 500, 3, 64
    x = _bf16(rng, (B, N, H, d))
    for k, tail in ((40, 64), (200, 16), (30, 0), (N, 70)):
        idx = None if k == N else np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B)]).astype(np.int32)
        if idx is not None:
            idx[0, -3:] = [N - 3, N - 2, N - 1]                # batch 0 ends in the tail
            idx[1] = np.sort(rng.choice(N - 100, k, replace=False))   # batch 1 has no tail row
        cache = _bf16(rng, (B, N, H, d))
        rows = _bf16(rng, (B, k, H, d))
        want_c, want_r = codec.keep_recent(cache, rows, x, idx, tail)
        dc, dr = up_bf16(cache), up_bf16(rows)
        F.kv_keep_recent(up_bf16(x), None if idx is None else torch.from_numpy(idx).cuda(), tail, cache=dc, rows=dr)
        torch.cuda.synchronize()
        assert np.array_equal(down_bits16(dc), want_c), (k, tail)
        assert np.array_equal(down_bits16(dr), want_r), (k, tail)


def test_codec_kv_pair_empty_selection(F):
    rng = np.random.default_rng(9)
    B, N, H, d = 1, 40, 2, 64
    kref, vref = _bf16(rng, (B, N, H, d)), _bf16(rng, (B, N, H, d))
    dk, dv = up_bf16(kref), up_bf16(vref)
    idx = torch.empty(B, 0, dtype=torch.int32, device="cuda")
    ko, vo = F.kv_residual_quant_kv(up_bf16(kref), dk, up_bf16(vref), dv, idx, 4, 32, mode=F.DQ_COMMIT)
    torch.cuda.synchronize()
    assert ko[0].numel() == 0 and vo[0].numel() == 0
    assert np.array_equal(down_bits16(dk), kref) and np.array_equal(down_bits16(dv), vref)


@pytest.mark.parametrize("axis", [codec.AXIS_TOKEN, codec.AXIS_CHANNEL])
def test_base_codec_all_rows(F, axis):
    rng = np.random.default_rng(5 + axis)
    B, N, H, d, G = 1, 333, 2, 128, 64
    x = _bf16(rng, (B, N, H, d))
    enc = codec.quantize(x, None, None, 4, G, axis)
    x_hat, _ = codec.reconstruct(None, x, None, enc, 4, G, axis)
    out = torch.empty(B, N, H, d, dtype=torch.bfloat16, device="cuda")
    codes, scale, zero, _ = F.kv_residual_quant(up_bf16(x), None, None, 4, G, axis, rows=out)
    torch.cuda.synchronize()
    assert np.array_equal(down(codes), enc["codes"])
    assert np.array_equal(down(scale).view(np.uint16), f16_bits(enc["scale"]))
    assert np.array_equal(down(zero).view(np.uint16), f16_bits(enc["zero"]))
    assert np.array_equal(down_bits16(out), x_hat)


# ---------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("d", [64, 128])
def test_dense_loop_and_column_selection(F, d):
    rng = np.random.default_rng(d)
    B, N, H = 2, 333, 2
    q, k, v = (_bf16(rng, (B, N, H, d)) for _ in range(3))
    o, lse = F.dense_attn(up_bf16(q), up_bf16(k), up_bf16(v))
    col_key = F.column_scores(up_bf16(q), up_bf16(k))
    cols = F.select_columns(col_key, 4, 60)
    torch.cuda.synchronize()
    go, gl, gk, gc = down(o), down(lse), down(col_key), down(cols)
    sc = 1 / np.sqrt(d)
    want_o = np.empty((B, N, H, d))
    want_l = np.empty((B, N, H))
    for b in range(B):
        for h in range(H):
            oo, ll, cs = att.dense_loop(bf16_to_f64(q[b, :, h]), bf16_to_f64(k[b, :, h]),
                                        bf16_to_f64(v[b, :, h]), sc)
            want_o[b, :, h], want_l[b, :, h] = oo, ll
            assert_keys_close(gk[b, h], cs.astype(np.float32), f"column keys b={b} h={h}")
            assert np.array_equal(gc[b, h], att.select_columns(cs.astype(np.float32), 4, 60))
    assert_close(go, want_o, f"dense o d={d}")
    assert_close(gl, want_l, f"dense lse d={d}")


# ---------------------------------------------------------------------------------------------------
CHAIN_CASES = [
    ("C1", {}),
    ("C2", dict(seq=1024, heads=3, col_budget=128)),
    ("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300)),
    ("C5", dict(seq=1200, heads=2, batch=2, col_budget=200)),
    ("C3", dict(seq=1500, heads=2, col_budget=160)),
    # a decaying column budget: lists pruned after loops 3 and 4, loops 4 and 5 recompute their subtract pass
    ("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300, loops=5, hot_frac=(0.1, 0.08, 0.06, 0.05),
                topk_frac=(0.1, 0.08, 0.06, 0.05), bits=(4, 2, 2, 2),
                col_decay=(4 + 128 + 300, 4 + 128 + 300, 4 + 128 + 150, 4 + 128 + 60))),
    ("C5", dict(seq=1200, heads=2, batch=2, col_budget=200, col_decay=(200, 200, 160, 120, 80, 60, 40))),
    # the most recent 64 positions stored exactly in bf16 (Appendix E), with a band and with a batch
    ("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300, tail=64)),
    ("C5", dict(seq=1200, heads=2, batch=2, col_budget=200, tail=64)),
]


def _dict_to_array(dct, B, H):
    return np.stack([np.stack([dct[b, h] for h in range(H)], axis=1) for b in range(B)])


@pytest.mark.parametrize("name,over", CHAIN_CASES)
def test_chain_matches_oracle(F, name, over):
    """GPU state end to end (setup, then every sparse loop) against the oracle's chain."""
    from paper_2609_29812_amd import driver
    w = get(name).replace(**over)
    st = make_layer(w)
    say(f"chain {w.name} B={w.batch} N={w.seq} H={w.heads} d={w.head_dim} R={w.loops} w={w.window}")
    rec = chain.run_layer(st)
    B, H = w.batch, w.heads
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                      w.window, tail=w.tail)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(gs.k_hat), rec.k_hat1), "base K reconstruction differs"
    assert np.array_equal(down_bits16(gs.v_hat), rec.v_hat1), "base V reconstruction differs"
    assert np.array_equal(down(gs.base["codes_k"]), rec.enc_k1["codes"])
    assert np.array_equal(down(gs.base["codes_v"]), rec.enc_v1["codes"])
    gk = down(gs.base["col_key"])
    for b in range(B):
        for h in range(H):
            assert_keys_close(gk[b, h], rec.colkey[b, h], f"column keys b={b} h={h}")
    want_cols = np.stack([np.stack([rec.cols[b, h] for h in range(H)]) for b in range(B)])
    assert np.array_equal(down(gs.cols), want_cols), "column lists differ"
    assert_close(down(gs.o), _dict_to_array(rec.o1, B, H), "loop 1 o")
    assert_close(down(gs.lse), _dict_to_array(rec.lse1, B, H), "loop 1 lse")
    for lr in rec.loops:
        r = lr.r
        out = driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                                 dev["v"][r - 1], dev["v"][r - 2], w.k(r), w.bits_at(r), keep=True)
        torch.cuda.synchronize()
        say(f" loop {r}: k={w.k(r)} bits={w.bits_at(r)}")
        assert_keys_close(down(out["key"]), lr.keys, f"loop {r} keys")
        assert np.array_equal(down(out["idx"]), lr.idx), f"loop {r} active rows"
        assert np.array_equal(down(out["slot"]), lr.slot), f"loop {r} slot"
        assert np.array_equal(down(out["codes_k"]), lr.enc_k["codes"]), f"loop {r} K codes"
        assert np.array_equal(down(out["codes_v"]), lr.enc_v["codes"]), f"loop {r} V codes"
        if w.bits_at(r) != 16:
            assert np.array_equal(down(out["scale_k"]).view(np.uint16), f16_bits(lr.enc_k["scale"]))
            assert np.array_equal(down(out["zero_k"]).view(np.uint16), f16_bits(lr.enc_k["zero"]))
            assert np.array_equal(down(out["scale_v"]).view(np.uint16), f16_bits(lr.enc_v["scale"]))
            assert np.array_equal(down(out["zero_v"]).view(np.uint16), f16_bits(lr.enc_v["zero"]))
        assert np.array_equal(new_rows(out, "k_new", gs.k_hat), lr.k_new), f"loop {r} new K rows"
        assert np.array_equal(new_rows(out, "v_new", gs.v_hat), lr.v_new), f"loop {r} new V rows"
        assert_close(down(gs.o), _dict_to_array(lr.o, B, H), f"loop {r} o (chained)")
        assert_close(down(gs.lse), _dict_to_array(lr.lse, B, H), f"loop {r} lse (chained)")
        if lr.cols_next is not None:
            driver.prune_list(gs, dev["q"][r - 1], w.top_cols_at(r + 1), w.n_sink)
            want = np.stack([np.stack([lr.cols_next[b, h] for h in range(H)]) for b in range(B)])
            assert np.array_equal(down(gs.cols), want), f"lists pruned after loop {r} differ"
            say(f" pruned after loop {r} to {want.shape[2]} entries")
    assert np.array_equal(down_bits16(gs.k_hat), rec.k_hat), "final K cache differs"
    assert np.array_equal(down_bits16(gs.v_hat), rec.v_hat), "final V cache differs"
    assert torch.equal(gs.v16.view(torch.int16), gs.v_hat.float().half().view(torch.int16)), "fp16 value copy"


@pytest.mark.parametrize("name,over", [("C4", dict(seq=1100, heads=2, window=100, col_budget=4 + 100 + 150)),
                                       ("C2", dict(seq=900, heads=2, head_dim=64, col_budget=100))])
def test_sparse_attn_stepwise_from_oracle_state(F, name, over):
    """One call of fl_loop_sparse_attn fed exactly the oracle's loop r-1 state."""
    w = get(name).replace(**over)
    st = make_layer(w)
    rec = chain.run_layer(st)
    B, H = w.batch, w.heads
    o_prev, l_prev = _dict_to_array(rec.o1, B, H), _dict_to_array(rec.lse1, B, H)
    k_hat, v_hat = rec.k_hat1, rec.v_hat1
    cols = up(np.stack([np.stack([rec.cols[b, h] for h in range(H)]) for b in range(B)]))
    for lr in rec.loops:
        r = lr.r
        o = up(o_prev.astype(np.float32))
        lse = up(l_prev.astype(np.float32))
        F.loop_sparse_attn(up_bf16(st.q[r - 1]), up_bf16(st.q[r - 2]), up_bf16(k_hat), up_bf16(v_hat),
                           up_bf16(lr.k_new), up_bf16(lr.v_new), up(lr.slot), up(lr.idx), cols, w.window,
                           lse, o)
        torch.cuda.synchronize()
        want_o, want_l = _dict_to_array(lr.o, B, H), _dict_to_array(lr.lse, B, H)
        rows = lr.idx[0]
        assert_close(down(o)[:, rows], want_o[:, rows], f"loop {r} o (step-wise, active rows)")
        assert_close(down(lse)[:, rows], want_l[:, rows], f"loop {r} lse (step-wise, active rows)")
        others = np.setdiff1d(np.arange(w.seq), rows)
        assert np.array_equal(down(o)[:, others], o_prev.astype(np.float32)[:, others])
        o_prev, l_prev = want_o, want_l
        k_hat = codec.reconstruct(k_hat, st.k[r - 1], lr.idx, lr.enc_k, w.bits_at(r), w.group, codec.AXIS_TOKEN)[0]
        v_hat = codec.reconstruct(v_hat, st.v[r - 1], lr.idx, lr.enc_v, w.bits_at(r), w.group, codec.AXIS_CHANNEL)[0]


@pytest.mark.parametrize("name,over", [("C4", dict(seq=1100, heads=2, window=100, col_budget=4 + 100 + 150)),
                                       # two batch elements; the band alone (an empty list); d = 64; fewer rows
                                       # than one segment
                                       ("C4", dict(seq=1500, heads=2, batch=2, window=128, col_budget=4 + 128 + 200)),
                                       ("C4", dict(seq=1500, heads=2, window=128, n_sink=0, col_budget=128)),
                                       ("C4", dict(seq=1300, heads=2, head_dim=64, window=96, col_budget=4 + 96 + 120)),
                                       ("C4", dict(seq=600, heads=2, window=64, col_budget=4 + 64 + 50)),
                                       # the 64-row kernel: no band (d = 128 with a ragged row tile, d = 64,
                                       # two batch elements over seven sparse loops), and a band with a list
                                       # longer than the segment kernel keeps
                                       ("C2", dict(seq=900, heads=2, col_budget=100)),
                                       ("C1", dict()),
                                       ("C5", dict(seq=600, heads=2, batch=2)),
                                       ("C4", dict(seq=2600, heads=1, window=64, col_budget=4 + 64 + 2100)),
                                       # enough rows for the one-team kernels (ceil(k / 128) * B * H = 384)
                                       ("C5", dict(seq=1600, heads=16, batch=2, loops=2, hot_frac=(0.9,),
                                                   topk_frac=(0.9,), bits=(4,), col_budget=100)),
                                       ("C5", dict(seq=1600, heads=16, head_dim=64, batch=2, loops=2,
                                                   hot_frac=(0.9,), topk_frac=(0.9,), bits=(2,), col_budget=60)),
                                       # d = 64 with 57-row segments: a group of 25 rows, so one of the
                                       # epilogue's four-row instructions holds a single existing row
                                       ("C5", dict(seq=1500, heads=2, head_dim=64, batch=1, loops=2,
                                                   hot_frac=(0.3,), topk_frac=(0.3,), bits=(4,), col_budget=124,
                                                   group=32))])
def test_subtract_pass_then_add_pass_from_oracle_state(F, name, over):
    """fl_loop_subtract_terms on the oracle's loop r-1 state: every row's subtract term and mass against the
    oracle's subtract half of Eq. 7; then the new rows committed and the add pass run with those terms
    (fl_loop_sparse_attn_terms), against the oracle's loop r outputs."""
    w = get(name).replace(**over)
    st = make_layer(w)
    rec = chain.run_layer(st)
    B, H, d, N = w.batch, w.heads, w.head_dim, w.seq
    sc = 1.0 / np.sqrt(d)
    say(f"subtract pass {w.name} B={B} N={N} H={H} d={d} window={w.window}")
    o_prev, l_prev = _dict_to_array(rec.o1, B, H), _dict_to_array(rec.lse1, B, H)
    k_hat, v_hat = rec.k_hat1, rec.v_hat1
    cols_np = np.stack([np.stack([rec.cols[b, h] for h in range(H)]) for b in range(B)])
    cols = up(cols_np)
    assert F.subtract_terms_supported(rec.loops[0].idx.shape[1], cols_np.shape[2], w.window, N, d)
    for lr in rec.loops:
        say(f" loop {lr.r}: k={lr.idx.shape[1]} subtract pass "
            f"{F.attn_kernel_name(F.PASS_SUBTRACT, lr.idx.shape[1], cols_np.shape[2], w.window, B, N, H, d)}, add pass "
            f"{F.attn_kernel_name(F.PASS_ADD, lr.idx.shape[1], cols_np.shape[2], w.window, B, N, H, d)}")
    for lr in rec.loops:
        r = lr.r
        k = lr.idx.shape[1]
        l32 = l_prev.astype(np.float32)
        qp = up_bf16(st.q[r - 2])
        kc, vc = up_bf16(k_hat), up_bf16(v_hat)
        term, mass = F.subtract_terms(qp, kc, vc, up(lr.idx), cols, w.window, up(l32))
        torch.cuda.synchronize()
        want_t = np.zeros((B, k, H, d))
        want_m = np.zeros((B, k, H))
        for b in range(B):
            for h in range(H):
                kp, vp = bf16_to_f64(k_hat[b, :, h]), bf16_to_f64(v_hat[b, :, h])
                for p, i in enumerate(lr.idx[b]):
                    S = att.row_columns(cols_np[b, h], int(i), w.window)
                    want_t[b, p, h], want_m[b, p, h] = att.subtract_row(
                        S, bf16_to_f64(st.q[r - 2][b, i, h]), kp, vp, float(l32[b, i, h]), sc)
        assert_close(down(term), want_t, f"loop {r} subtract terms")
        assert_close(down(mass), want_m, f"loop {r} masses")
        # commit the new rows, then the add pass alone with these terms (slot_prev: this loop's slot map)
        o = up(o_prev.astype(np.float32))
        lse = up(l32)
        F.kv_residual_quant_kv(up_bf16(st.k[r - 1]), kc, up_bf16(st.v[r - 1]), vc, up(lr.idx), w.bits_at(r),
                               w.group, mode=F.DQ_COMMIT)
        F.loop_sparse_attn(up_bf16(st.q[r - 1]), None, kc, vc, None, None, up(lr.slot), up(lr.idx), cols,
                           w.window, lse, o, term_prev=term, mass_prev=mass, slot_prev=up(lr.slot))
        torch.cuda.synchronize()
        k_hat = codec.reconstruct(k_hat, st.k[r - 1], lr.idx, lr.enc_k, w.bits_at(r), w.group, codec.AXIS_TOKEN)[0]
        v_hat = codec.reconstruct(v_hat, st.v[r - 1], lr.idx, lr.enc_v, w.bits_at(r), w.group, codec.AXIS_CHANNEL)[0]
        assert np.array_equal(down_bits16(kc), k_hat) and np.array_equal(down_bits16(vc), v_hat), \
            f"loop {r} committed caches"
        want_o, want_l = _dict_to_array(lr.o, B, H), _dict_to_array(lr.lse, B, H)
        for b in range(B):
            rows = lr.idx[b]
            assert_close(down(o)[b][rows], want_o[b][rows], f"loop {r} o (subtract pass, then add pass), b={b}")
            assert_close(down(lse)[b][rows], want_l[b][rows], f"loop {r} lse (subtract pass, then add pass), b={b}")
            others = np.setdiff1d(np.arange(N), rows)
            assert np.array_equal(down(o)[b][others], o_prev.astype(np.float32)[b][others])
        o_prev, l_prev = want_o, want_l


def test_subtract_pass_coverage_and_arguments(F):
    """The query covers lists of at most 3072 entries (the segment kernel with a band and at most 2048, the
    64-row kernel otherwise); beyond that the call returns FL_E_UNSUPPORTED without a launch; k = 0 is a
    no-op."""
    from paper_2609_29812_amd.flashloop import FlashLoopError
    assert F.subtract_terms_supported(100, 512, 64, 4096, 128)
    assert F.subtract_terms_supported(100, 2048, 1, 4096, 64)
    assert F.subtract_terms_supported(100, 512, 0, 4096, 128)           # no band
    assert F.subtract_terms_supported(100, 3072, 64, 4096, 128)         # beyond the segment kernel's list
    assert not F.subtract_terms_supported(100, 3073, 64, 4096, 128)     # list beyond the LDS copy
    assert not F.subtract_terms_supported(100, 3073, 0, 4096, 128)
    assert not F.subtract_terms_supported(100, 512, 64, 4096, 96)       # head dim
    B, N, H, d = 1, 256, 2, 64
    q = torch.zeros(B, N, H, d, dtype=torch.bfloat16, device="cuda")
    rows = torch.arange(0, N, 4, dtype=torch.int32, device="cuda").view(1, -1)
    cols = torch.arange(0, 32, dtype=torch.int32, device="cuda").view(1, 1, -1).repeat(1, H, 1).contiguous()
    lse = torch.zeros(B, N, H, dtype=torch.float32, device="cuda")
    N4 = 4096
    q4 = torch.zeros(B, N4, H, d, dtype=torch.bfloat16, device="cuda")
    rows4 = torch.arange(0, N4, 64, dtype=torch.int32, device="cuda").view(1, -1)
    long_cols = torch.arange(0, 3100, dtype=torch.int32, device="cuda").view(1, 1, -1).repeat(1, H, 1).contiguous()
    lse4 = torch.zeros(B, N4, H, dtype=torch.float32, device="cuda")
    with pytest.raises(FlashLoopError, match="above 3072"):
        F.subtract_terms(q4, q4, q4, rows4, long_cols, 0, lse4)
    empty = torch.zeros(1, 0, dtype=torch.int32, device="cuda")
    t, m = F.subtract_terms(q, q, q, empty, cols, 16, lse)
    assert t.shape == (1, 0, H, d) and m.shape == (1, 0, H)


@pytest.mark.parametrize("name,over", [("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300)),
                                       ("C5", dict(seq=1200, heads=2, batch=2, col_budget=200)),
                                       ("C2", dict(seq=900, heads=2, head_dim=64, col_budget=100)),
                                       # lists at the LDS copy's capacity (3072 entries) and beyond it (the
                                       # record-table kernel), with and without a band
                                       ("C5", dict(seq=4000, heads=2, col_budget=3072)),
                                       ("C5", dict(seq=4500, heads=2, col_budget=3300)),
                                       ("C4", dict(seq=5000, heads=2, window=256, col_budget=4 + 256 + 3200)),
                                       # the band alone (an empty list), and fewer rows than one 64-row tile
                                       ("C4", dict(seq=1500, heads=2, window=128, n_sink=0, col_budget=128)),
                                       ("C4", dict(seq=600, heads=2, window=64, col_budget=4 + 64 + 50))])
def test_reused_subtract_terms_match_recomputed_ones(F, name, over):
    """Loops >= 3 with the previous loop's add terms as subtract terms against the same loops with the
    subtract pass recomputed: equal up to fp32 rounding (Eq. 7 with fixed S and nested rows)."""
    from paper_2609_29812_amd import driver
    w = get(name).replace(**over)
    st = make_layer(w)
    say(f"reuse {w.name} B={w.batch} N={w.seq} H={w.heads} d={w.head_dim} R={w.loops}")
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    runs = []
    for reuse in (False, True):
        gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                          w.window)
        gs.reuse = reuse
        outs = []
        for r in range(2, w.loops + 1):
            driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                               dev["v"][r - 1], dev["v"][r - 2], w.k(r), w.bits_at(r))
            torch.cuda.synchronize()
            outs.append((down(gs.o), down(gs.lse), down(gs.cand)))
        runs.append(outs)
    for r, (full, reu) in enumerate(zip(*runs), start=2):
        assert np.array_equal(full[2], reu[2]), f"loop {r} active rows"
        assert_close(reu[0], full[0], f"loop {r} o: reused vs recomputed subtract terms")
        assert_close(reu[1], full[1], f"loop {r} lse: reused vs recomputed subtract terms")


def test_reuse_leaves_rows_without_a_previous_term_unchanged(F):
    from paper_2609_29812_amd import driver
    w = get("C2").replace(seq=600, heads=2, col_budget=80)
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                      w.window)
    driver.sparse_step(gs, dev["q"][1], dev["q"][0], dev["k"][1], dev["k"][0], dev["v"][1], dev["v"][0],
                       w.k(2), w.bits_at(2))
    torch.cuda.synchronize()
    dropped = int(down(gs.cand)[0, 3])
    gs.slot_prev[0, dropped] = -1
    o_before = down(gs.o)[0, dropped].copy()
    driver.sparse_step(gs, dev["q"][2], dev["q"][1], dev["k"][2], dev["k"][1], dev["v"][2], dev["v"][1],
                       w.k(3), w.bits_at(3))
    torch.cuda.synchronize()
    assert dropped in down(gs.cand)[0]
    assert np.array_equal(down(gs.o)[0, dropped], o_before)
    assert not down(gs.mass)[0, list(down(gs.cand)[0]).index(dropped)].any()


@pytest.mark.parametrize("n,kind", [(40004, "equal"), (40004, "few_values"), (40004, "random"),
                                    (32772, "random"), (1700, "few_values"), (5000, "one_bin")])
def test_topk_threshold_search_matches_oracle(F, n, kind):
    """The shared top-k kernel (through fl_select_columns) on large, tied and single-bin key sets: above
    32K keys a histogram bin can exceed the LDS buffer (register fallback); ties go to lower indices."""
    rng = np.random.default_rng(n)
    keys = {"equal": np.full(n, 0.25, np.float32),
            "few_values": rng.choice(np.float32([0.0, 1e-3, 0.5, 0.5000001, 3.0]), n).astype(np.float32),
            "random": rng.random(n, dtype=np.float32) ** 3,
            "one_bin": (1.0 + rng.integers(0, 64, n) * 2.0 ** -20).astype(np.float32)}[kind]
    say(f"top-k n={n} kind={kind}")
    for t in (1, 777, (n - 4) // 2, n - 4):
        got = down(F.select_columns(up(keys[None, None, :]), 4, t))[0, 0]
        want = att.select_columns(keys, 4, t)
        assert np.array_equal(got, want), f"n={n} kind={kind} t={t}"


def test_all_rows_all_columns_no_quantization_is_dense_attention(F):
    """The special case that reduces the chain to exact dense attention of each loop, on the GPU."""
    from paper_2609_29812_amd import driver
    w = get("C2").replace(seq=500, heads=2, head_dim=128, topk_frac=(1.0, 1.0, 1.0), bits=(16, 16, 16),
                          col_budget=500, n_sink=500)
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], 16, w.group, w.seq, 0, 0)
    for r in range(2, w.loops + 1):
        driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                           dev["v"][r - 1], dev["v"][r - 2], w.seq, 16)
        o, lse = F.dense_attn(dev["q"][r - 1], dev["k"][r - 1], dev["v"][r - 1])
        torch.cuda.synchronize()
        assert_close(down(gs.o), down(o), f"loop {r}: corrected vs dense (GPU)")
        for h in range(w.heads):
            want, _, _ = att.dense_loop(*(bf16_to_f64(getattr(st, n)[r - 1][0, :, h]) for n in "qkv"),
                                        w.sm_scale, want_colscore=False)
            assert_close(down(gs.o)[0, :, h], want, f"loop {r} h={h}: corrected vs oracle dense")


def test_results_are_deterministic(F):
    from paper_2609_29812_amd import driver
    w = get("C4").replace(seq=1500, heads=2, window=64, col_budget=4 + 64 + 200)
    st = make_layer(w)
    outs = []
    for _ in range(2):
        dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
        gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink,
                          w.top_cols, w.window)
        for r in range(2, w.loops + 1):
            driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                               dev["v"][r - 1], dev["v"][r - 2], w.k(r), w.bits_at(r))
        torch.cuda.synchronize()
        outs.append([down(gs.o), down(gs.lse), down_bits16(gs.k_hat), down(gs.cols), down(gs.base["col_key"])])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


def test_ragged_batch_budgets_on_single_element_views(F):
    """A token budget per batch element (Appendix D.1, Eq. 5 with its own k_b^(r) per element): every entry
    point takes one k for the whole batch, so a ragged batch runs the per-loop step once per element on
    B = 1 views of the batched tensors (batch is the leading dimension, so each view is contiguous) and
    must match the oracle's chain run on that element alone, with that element's budgets."""
    from paper_2609_29812_amd import driver
    from workloads.gen import LoopStates
    w = get("C5").replace(batch=3, seq=1500, heads=2, head_dim=64, loops=4, hot_frac=(0.3, 0.2, 0.1),
                          topk_frac=(0.3, 0.2, 0.1), bits=(4, 4, 2), col_budget=4 + 120, group=32)
    budgets = [(0.3, 0.2, 0.1), (0.15, 0.15, 0.05), (0.4, 0.1, 0.02)]
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    for b, fr in enumerate(budgets):
        wb = w.replace(name=f"ragged-b{b}", batch=1, topk_frac=fr)
        sb = LoopStates(wb, 0, [a[b:b + 1] for a in st.q], [a[b:b + 1] for a in st.k], [a[b:b + 1] for a in st.v],
                        [[hot[b]] for hot in st.hot])
        rec = chain.run_layer(sb)
        view = {n: [t[b:b + 1] for t in dev[n]] for n in "qkv"}
        say(f"ragged element {b}: k per loop {[wb.k(r) for r in range(2, wb.loops + 1)]}")
        gs = driver.setup(view["q"][0], view["k"][0], view["v"][0], wb.base_bits, wb.group, wb.n_sink,
                          wb.top_cols, wb.window)
        for lr in rec.loops:
            r = lr.r
            out = driver.sparse_step(gs, view["q"][r - 1], view["q"][r - 2], view["k"][r - 1], view["k"][r - 2],
                                     view["v"][r - 1], view["v"][r - 2], wb.k(r), wb.bits_at(r), keep=True)
            torch.cuda.synchronize()
            assert np.array_equal(down(out["idx"]), lr.idx), f"element {b} loop {r}: active rows"
            assert np.array_equal(down(out["codes_k"]), lr.enc_k["codes"]), f"element {b} loop {r}: K codes"
            assert np.array_equal(down(out["codes_v"]), lr.enc_v["codes"]), f"element {b} loop {r}: V codes"
            assert_close(down(gs.o), _dict_to_array(lr.o, 1, wb.heads), f"element {b} loop {r} o")
            assert_close(down(gs.lse), _dict_to_array(lr.lse, 1, wb.heads), f"element {b} loop {r} lse")
        assert np.array_equal(down_bits16(gs.k_hat), rec.k_hat), f"element {b}: final K cache"
        assert np.array_equal(down_bits16(gs.v_hat), rec.v_hat), f"element {b}: final V cache"
    # the views never wrote outside their element: the batched input tensors are untouched
    for n in "qkv":
        for r in range(w.loops):
            assert np.array_equal(down_bits16(dev[n][r]), getattr(st, n)[r]), f"input {n}{r + 1} was modified"

"""Parity at the workloads' full sizes, in the launch configuration the benchmark times (the driver's
chain: dense set-up, then every sparse loop with the add terms reused from loop 3 on).

Selection keys, active rows, slot maps, residual codes and metadata, the reconstructed rows and the
final caches are compared for every head and row.  The attention state (o, lse_ref) is compared for
every updated row of a few sampled heads, which the oracle computes one row at a time (its loop-1 set-up
is O(N^2 d) per head, so it evaluates only those heads).  The oracle and the GPU advance loop by loop.
"""
import time

import numpy as np
import pytest
import torch

from gpu_util import assert_close, assert_keys_close, down, down_bits16, f16_bits, new_rows, say, up_bf16
from oracle import chain
from workloads import get, make_layer

pytestmark = pytest.mark.gpu

# (workload, layer, sampled heads (None = all))
CASES = [
    ("C4", 0, [0, 9]),            # 32K long prefill, window 512, int2 residuals
    ("C2", 0, None),              # 4K, every head
    ("C3", 7, [0, 15]),           # 8K, one layer of the 48-layer stack
    ("C5", 0, [3]),               # B = 4, 16K, 8 loops (int4 residuals, then int2 from loop 4)
]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,layer,heads", CASES)
def test_full_size_chain_matches_oracle(F, name, layer, heads):
    from paper_2609_29812_amd import driver
    w = get(name)
    t0 = time.time()
    say(f"full size {w.name} layer {layer}: B={w.batch} N={w.seq} H={w.heads} d={w.head_dim} loops 2-{w.loops}")
    st = make_layer(w, layer)
    B, H = w.batch, w.heads
    heads = list(range(H)) if heads is None else heads
    say(f" inputs generated ({time.time() - t0:.0f}s); oracle loop 1 for heads {heads}")
    rec = chain.loop1(st, heads)
    say(f" oracle loop 1 done ({time.time() - t0:.0f}s)")

    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                      w.window)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(gs.k_hat), rec.k_hat1) and np.array_equal(down_bits16(gs.v_hat), rec.v_hat1)
    cols = down(gs.cols)
    for b in range(B):
        for h in heads:
            assert np.array_equal(cols[b, h], rec.cols[b, h]), f"column list b={b} h={h}"
    o = {key: val.copy() for key, val in rec.o1.items()}
    lse = {key: val.copy() for key, val in rec.lse1.items()}
    k_hat, v_hat, cand = rec.k_hat1, rec.v_hat1, None
    for r in range(2, w.loops + 1):
        lr, k_hat, v_hat = chain.sparse_loop(st, r, cand, k_hat, v_hat, rec.cols, o, lse, heads)
        cand = lr.idx
        out = driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                                 dev["v"][r - 1], dev["v"][r - 2], w.k(r), w.bits_at(r), keep=True)
        torch.cuda.synchronize()
        say(f" loop {r}: k={w.k(r)} bits={w.bits_at(r)} ({time.time() - t0:.0f}s)")
        assert_keys_close(down(out["key"]), lr.keys, f"loop {r} keys")
        assert np.array_equal(down(out["idx"]), lr.idx), f"loop {r} active rows"
        assert np.array_equal(down(out["slot"]), lr.slot), f"loop {r} slot map"
        assert np.array_equal(down(out["codes_k"]), lr.enc_k["codes"]), f"loop {r} K codes"
        assert np.array_equal(down(out["codes_v"]), lr.enc_v["codes"]), f"loop {r} V codes"
        if w.bits_at(r) != 16:
            assert np.array_equal(down(out["scale_k"]).view(np.uint16), f16_bits(lr.enc_k["scale"]))
            assert np.array_equal(down(out["zero_k"]).view(np.uint16), f16_bits(lr.enc_k["zero"]))
            assert np.array_equal(down(out["scale_v"]).view(np.uint16), f16_bits(lr.enc_v["scale"]))
            assert np.array_equal(down(out["zero_v"]).view(np.uint16), f16_bits(lr.enc_v["zero"]))
        assert np.array_equal(new_rows(out, "k_new", gs.k_hat), lr.k_new), f"loop {r} new K rows"
        assert np.array_equal(new_rows(out, "v_new", gs.v_hat), lr.v_new), f"loop {r} new V rows"
        go, gl = down(gs.o), down(gs.lse)
        for b in range(B):
            rows = lr.idx[b]
            for h in heads:
                assert_close(go[b, rows, h], lr.o[b, h][rows], f"loop {r} o b={b} h={h} ({rows.size} rows)")
                assert_close(gl[b, rows, h], lr.lse[b, h][rows], f"loop {r} lse b={b} h={h}")
    assert np.array_equal(down_bits16(gs.k_hat), k_hat), "final K cache"
    assert np.array_equal(down_bits16(gs.v_hat), v_hat), "final V cache"
    assert torch.equal(gs.v16.view(torch.int16), gs.v_hat.float().half().view(torch.int16)), "fp16 value copy"

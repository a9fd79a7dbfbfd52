"""The packed streams as the state of record (Section 4.3, Eq. 4 and Eq. 8; Appendix G).

The layer keeps bf16 caches for the attention to read, but they are derived data: the base codes and
metadata of loop 1 and, for every sparse loop, the residual codes and metadata of its active rows rebuild
them bit for bit.  The rebuild starts from zero caches, applies the base reconstruction to every row, then
each loop's residual to that loop's rows in loop order (the same bf16 rounding the quantizers applied when
they committed the rows), and must equal the caches the step left, and the fp16 value copy must equal the
rebuilt values converted to fp16.  Shapes: a band (the 32K structure at a small size) and a batch without a
band over seven sparse loops."""
import numpy as np
import pytest
import torch

from gpu_util import down_bits16, say, up_bf16
from workloads import get, make_layer

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,over", [("C4", dict(seq=2000, heads=2, window=128, col_budget=4 + 128 + 300)),
                                       ("C5", dict(seq=1200, heads=2, batch=2, col_budget=200))])
def test_packed_streams_rebuild_the_caches(F, name, over):
    from paper_2609_29812_amd import driver
    w = get(name).replace(**over)
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    say(f"packed rebuild {w.name} B={w.batch} N={w.seq} H={w.heads} R={w.loops} window={w.window}")
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols,
                      w.window)
    loops = []
    for r in range(2, w.loops + 1):
        out = driver.sparse_step(gs, dev["q"][r - 1], dev["q"][r - 2], dev["k"][r - 1], dev["k"][r - 2],
                                 dev["v"][r - 1], dev["v"][r - 2], w.k(r), w.bits_at(r), keep=True)
        loops.append((out, w.bits_at(r)))
    torch.cuda.synchronize()
    kh, vh = torch.zeros_like(gs.k_hat), torch.zeros_like(gs.v_hat)
    base = gs.base
    F.kv_residual_dequant(base["codes_k"], base["scale_k"], base["zero_k"], None, w.base_bits, w.group,
                          F.AXIS_TOKEN, kh, mode=F.DQ_COMMIT)
    F.kv_residual_dequant(base["codes_v"], base["scale_v"], base["zero_v"], None, w.base_bits, w.group,
                          F.AXIS_CHANNEL, vh, mode=F.DQ_COMMIT)
    for out, bits in loops:
        F.kv_residual_dequant_kv((out["codes_k"], out["scale_k"], out["zero_k"]),
                                 (out["codes_v"], out["scale_v"], out["zero_v"]), out["idx"], bits, w.group,
                                 kh, vh, mode=F.DQ_COMMIT)
    torch.cuda.synchronize()
    assert np.array_equal(down_bits16(kh), down_bits16(gs.k_hat)), "keys rebuilt from the packed streams"
    assert np.array_equal(down_bits16(vh), down_bits16(gs.v_hat)), "values rebuilt from the packed streams"
    assert torch.equal(gs.v16.view(torch.int16), vh.float().half().view(torch.int16)), "fp16 value copy"
    # the loops changed the caches: the rebuild is not the base reconstruction alone
    kb = torch.zeros_like(kh)
    F.kv_residual_dequant(base["codes_k"], base["scale_k"], base["zero_k"], None, w.base_bits, w.group,
                          F.AXIS_TOKEN, kb, mode=F.DQ_COMMIT)
    assert not torch.equal(kb, kh)

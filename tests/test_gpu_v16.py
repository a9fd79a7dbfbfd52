"""The fp16 copy of the value cache (fl_kv_f16_rows, fl_kv_residual_quant_kv_v16) and the attention calls that
read it (fl_loop_sparse_attn_terms_v16, fl_loop_subtract_terms_v16).

The copy holds fp16(bf16 value), rounded to nearest even; it is checked bit for bit against torch's own
conversion of the same values, including the ends of the fp16 range (subnormals, the largest finite value,
overflow to infinity).  The attention calls with the copy load value tiles as they are instead of converting
them in LDS, with the same rounding, so their outputs must equal those of the calls without the copy bit
for bit: checked on shapes with a band (the two-team segment kernels) and without one (the one-team and
two-team kernels)."""
import numpy as np
import pytest
import torch

from gpu_util import say, up_bf16
from workloads import get, make_layer

pytestmark = pytest.mark.gpu


def _f16_of(x_bf16):
    return x_bf16.float().half()


def test_f16_rows_all_and_selected(F):
    g = torch.Generator(device="cuda").manual_seed(5)
    B, N, H, d = 2, 300, 3, 64
    x = (torch.randn(B, N, H, d, device="cuda", generator=g) * 3).to(torch.bfloat16)
    # values at the ends of the fp16 range: subnormals, tiny values that round to 0, the largest finite
    # value, values that overflow, signed zeros
    special = torch.tensor([2.0 ** -14, 2.0 ** -20, 2.0 ** -24, 2.0 ** -26, 65504.0, 65536.0, -70000.0, -0.0,
                            1.0 + 2.0 ** -7, 3.0e-8], device="cuda").to(torch.bfloat16)
    x[0, 7, 1, :special.numel()] = special
    say("f16 rows: every row, then rows idx")
    y = F.kv_f16_rows(x)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), _f16_of(x).view(torch.int16))
    idx = torch.stack([torch.tensor([0, 7, 8, 150, 299], device="cuda"),
                       torch.tensor([1, 2, 3, 4, 298], device="cuda")]).to(torch.int32)
    z = torch.full_like(y, 7.0)
    F.kv_f16_rows(x, idx, out=z)
    torch.cuda.synchronize()
    want = torch.full_like(y, 7.0)
    for b in range(B):
        want[b, idx[b].long()] = _f16_of(x[b, idx[b].long()])
    assert torch.equal(z.view(torch.int16), want.view(torch.int16))
    F.kv_f16_rows(x, idx[:, :0].contiguous(), out=z)          # k = 0: nothing changes
    torch.cuda.synchronize()
    assert torch.equal(z.view(torch.int16), want.view(torch.int16))


@pytest.mark.parametrize("bits", [2, 4, 16])
def test_quant_kv_v16_matches_commit(F, bits):
    g = torch.Generator(device="cuda").manual_seed(bits)
    B, N, H, d, k, G = 2, 700, 2, 128, 200, 64
    kc, vc = (torch.randn(B, N, H, d, device="cuda", generator=g).to(torch.bfloat16) for _ in range(2))
    kr, vr = (torch.randn(B, N, H, d, device="cuda", generator=g).to(torch.bfloat16) for _ in range(2))
    idx = torch.stack([torch.sort(torch.randperm(N, device="cuda", generator=g)[:k]).values for _ in range(B)])
    idx = idx.to(torch.int32)
    say(f"quantize and commit with the fp16 value copy: bits {bits}")
    ka, va = kr.clone(), vr.clone()
    outa = F.kv_residual_quant_kv(kc, ka, vc, va, idx, bits, G, mode=F.DQ_COMMIT)
    kb, vb = kr.clone(), vr.clone()
    v16 = F.kv_f16_rows(vr)
    before = v16.clone()
    outb = F.kv_residual_quant_kv(kc, kb, vc, vb, idx, bits, G, mode=F.DQ_COMMIT, v_f16=v16)
    torch.cuda.synchronize()
    for ta, tb in zip([t for p in outa for t in p[:3] if t is not None], [t for p in outb for t in p[:3] if t is not None]):
        assert torch.equal(ta.view(torch.uint8), tb.view(torch.uint8))
    assert torch.equal(ka.view(torch.int16), kb.view(torch.int16))
    assert torch.equal(va.view(torch.int16), vb.view(torch.int16))
    want = before.clone()
    for b in range(B):
        want[b, idx[b].long()] = _f16_of(vb[b, idx[b].long()])
    assert torch.equal(v16.view(torch.int16), want.view(torch.int16)), "fp16 copy of the committed rows"
    assert torch.equal(v16.view(torch.int16), _f16_of(vb).view(torch.int16))


@pytest.mark.parametrize("name,over", [
    ("C4", dict(seq=3000, heads=4, window=256, col_budget=4 + 256 + 400)),           # band: two teams
    ("C2", dict(seq=2000, heads=8, col_budget=160)),                                # no band, few rows: two teams
    ("C5", dict(seq=1600, heads=16, batch=2, loops=2, hot_frac=(0.9,), topk_frac=(0.9,), bits=(4,),
                col_budget=100)),                                                   # no band, one team
    ("C5", dict(seq=1600, heads=16, head_dim=64, batch=2, loops=2, hot_frac=(0.9,), topk_frac=(0.9,),
                bits=(2,), col_budget=60))])
def test_attention_with_value_copy_is_bitwise_the_same(F, name, over):
    from paper_2609_29812_amd import driver
    w = get(name).replace(**over)
    st = make_layer(w)
    dev = {n: [up_bf16(a) for a in getattr(st, n)] for n in "qkv"}
    B, N, H, d = dev["k"][0].shape
    gs = driver.setup(dev["q"][0], dev["k"][0], dev["v"][0], w.base_bits, w.group, w.n_sink, w.top_cols, w.window,
                      v16=False)
    idx, slot, _ = F.select_tokens(dev["k"][1], dev["k"][0], dev["v"][1], dev["v"][0], w.k(2))
    k = idx.shape[1]
    c = gs.cols.shape[2]
    say(f"{w.name}: k={k} subtract pass {F.attn_kernel_name(F.PASS_SUBTRACT, k, c, w.window, B, N, H, d)}, "
        f"add pass {F.attn_kernel_name(F.PASS_ADD, k, c, w.window, B, N, H, d)}")
    v16 = F.kv_f16_rows(gs.v_hat)
    # subtract pass over the loop-1 state, with and without the copy
    sub_a = F.subtract_terms(dev["q"][0], gs.k_hat, gs.v_hat, idx, gs.cols, w.window, gs.lse)
    sub_b = F.subtract_terms(dev["q"][0], gs.k_hat, gs.v_hat, idx, gs.cols, w.window, gs.lse, v16=v16)
    torch.cuda.synchronize()
    for a, b in zip(sub_a, sub_b):
        assert torch.equal(a, b), "subtract pass with the value copy"
    # commit (with the copy), then the add pass with and without it
    F.kv_residual_quant_kv(dev["k"][1], gs.k_hat, dev["v"][1], gs.v_hat, idx, w.bits_at(2), w.group,
                           mode=F.DQ_COMMIT, v_f16=v16)
    outs = []
    for use in (False, True):
        o, lse = gs.o.clone(), gs.lse.clone()
        term = torch.empty(B, k, H, d, dtype=torch.float32, device="cuda")
        mass = torch.empty(B, k, H, dtype=torch.float32, device="cuda")
        F.loop_sparse_attn(dev["q"][1], None, gs.k_hat, gs.v_hat, None, None, slot, idx, gs.cols, w.window, lse, o,
                           term_prev=sub_a[0], mass_prev=sub_a[1], slot_prev=slot, term_out=term, mass_out=mass,
                           v16=v16 if use else None)
        outs.append((o, lse, term, mass))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b), "add pass with the value copy"
    assert not torch.equal(outs[0][0], gs.o), "the update changed nothing"

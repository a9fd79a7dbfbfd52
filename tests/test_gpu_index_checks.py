"""The optional index-list checks (fl_set_index_checks): with the checks on, a call given an unsorted or
out-of-range index list returns FL_E_RANGE and launches nothing; with them off (the default), valid lists
behave as before.  Every list here is a valid device buffer, so no kernel ever reads out of bounds: the bad
lists are rejected on the host before any launch."""
import numpy as np
import pytest
import torch

from gpu_util import say, up, up_bf16
from oracle.numerics import f32_to_bf16

pytestmark = pytest.mark.gpu


def _bf16(rng, shape):
    return up_bf16(f32_to_bf16(rng.standard_normal(shape).astype(np.float32)))


def test_unsorted_and_out_of_range_lists_are_rejected(F):
    rng = np.random.default_rng(5)
    B, N, H, d = 1, 300, 2, 64
    x, y = _bf16(rng, (B, N, H, d)), _bf16(rng, (B, N, H, d))
    good = up(np.array([[3, 10, 50, 120]], dtype=np.int32))
    unsorted = up(np.array([[3, 50, 10, 120]], dtype=np.int32))
    beyond = up(np.array([[3, 10, 50, N]], dtype=np.int32))
    F.set_index_checks(True)
    try:
        say("index checks on: select candidates, codec rows, attention rows and columns")
        F.select_tokens(x, y, None, None, 2, cand=good)                       # valid: accepted
        with pytest.raises(F.FlashLoopError, match="not strictly ascending"):
            F.select_tokens(x, y, None, None, 2, cand=unsorted)
        with pytest.raises(F.FlashLoopError, match="outside"):
            F.kv_residual_quant(x, y, beyond, 4, 32, F.AXIS_TOKEN)
        slot = torch.full((B, N), -1, dtype=torch.int32, device="cuda")
        cols = up(np.tile(np.array([0, 1, 2, 7, 9, 9], dtype=np.int32), (B, H, 1)))   # a repeated entry
        o = torch.zeros(B, N, H, d, dtype=torch.float32, device="cuda")
        lse = torch.zeros(B, N, H, dtype=torch.float32, device="cuda")
        with pytest.raises(F.FlashLoopError, match="cols.*not strictly ascending"):
            F.loop_sparse_attn(x, y, x, y, x[:, :4].contiguous(), y[:, :4].contiguous(), slot, good, cols, 8,
                               lse, o)
        torch.cuda.synchronize()
        assert float(o.abs().max()) == 0.0, "a rejected call wrote its output"
    finally:
        F.set_index_checks(False)
    F.select_tokens(x, y, None, None, 2, cand=good)                           # checks off again
    torch.cuda.synchronize()


def test_values_beyond_fp16_are_rejected_when_checking(F):
    # the attention's products with V run in fp16: with the checks on, a V cache holding |v| > 65504 is
    # rejected before any attention launch, and one within range is accepted
    rng = np.random.default_rng(6)
    B, N, H, d = 1, 200, 2, 64
    q, k = _bf16(rng, (B, N, H, d)), _bf16(rng, (B, N, H, d))
    v_ok = _bf16(rng, (B, N, H, d))
    big = rng.standard_normal((B, N, H, d)).astype(np.float32)
    big[0, 17, 1, 5] = 1.0e5
    v_big = up_bf16(f32_to_bf16(big))
    o = torch.zeros(B, N, H, d, dtype=torch.float32, device="cuda")
    lse = torch.zeros(B, N, H, dtype=torch.float32, device="cuda")
    F.set_index_checks(True)
    try:
        say("range check on: dense loop over a V cache with one value of 1e5, then one within range")
        with pytest.raises(F.FlashLoopError, match="65504"):
            F.dense_attn(q, k, v_big, o=o, lse=lse)
        torch.cuda.synchronize()
        assert float(o.abs().max()) == 0.0, "a rejected call wrote its output"
        F.dense_attn(q, k, v_ok, o=o, lse=lse)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(o).all())
    finally:
        F.set_index_checks(False)

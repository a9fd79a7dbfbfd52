"""The decode step without a workspace (fl_decode_step_noalloc) against the decode step with one
(fl_decode_step), through the C ABI: the same kernels on the same inputs, so every output must be
bitwise the same.  Two calls in a row on the library's scratch array (a dense loop at the larger shape, then
a sparse loop at a smaller one, and back), each compared with a fresh workspace call, so a stale region
left by the first call would show in the second."""
import numpy as np
import pytest
import torch

from gpu_util import say, up_bf16
from oracle.numerics import f32_to_bf16

pytestmark = pytest.mark.gpu


def _bf16(rng, shape):
    return up_bf16(f32_to_bf16(rng.standard_normal(shape).astype(np.float32)))


def _pair(F, q, k, v, cols, mass, sub, c_next, n_sink, window, seed_o):
    """Run both entry points from the same starting output; return both result tuples."""
    B, T, H, d = k.shape
    res = []
    for fn in ("ws", "noalloc"):
        o = seed_o.clone()
        lse = torch.empty(B, H, dtype=torch.float32, device="cuda")
        outs = None
        if c_next > 0:
            outs = (torch.full((B, H, c_next), -7, dtype=torch.int32, device="cuda"),
                    torch.full((B, H), float("nan"), dtype=torch.float32, device="cuda"),
                    torch.full((B, H, d), float("nan"), dtype=torch.float32, device="cuda"))
        if fn == "ws":
            ws = F.decode_ws(k, cols, c_next)
            ws.fill_(0xA5)                       # a workspace with garbage in it, as the scratch may hold
            r = F.decode_step(q, k, v, cols, mass, sub, o, c_next, n_sink=n_sink, window=window, lse=lse,
                              out=outs, ws=ws)
        else:
            r = F.decode_step_noalloc(q, k, v, cols, mass, sub, o, c_next, out=outs, n_sink=n_sink,
                                      window=window, lse=lse)
        torch.cuda.synchronize()
        res.append((o.cpu(), lse.cpu()) + tuple(None if t is None else t.cpu() for t in r))
    return res


def _same(a, b, what):
    for x, y, name in zip(a, b, ("o", "lse", "cols_next", "mass_next", "sub_next")):
        if x is None:
            assert y is None
            continue
        assert torch.equal(x.view(-1).view(torch.int32) if x.dtype == torch.float32 else x,
                           y.view(-1).view(torch.int32) if y.dtype == torch.float32 else y), f"{what}: {name} differs"


@pytest.mark.parametrize("d", [64, 128])
def test_noalloc_matches_the_workspace_call_on_two_calls_in_a_row(F, d):
    rng = np.random.default_rng(11 + d)
    # call 1: a dense loop at B=2, T=3000, H=4, selecting 700 columns
    B, T, H = 2, 3000, 4
    say(f"noalloc d={d}: dense B={B} T={T} H={H}")
    q, k, v = _bf16(rng, (B, H, d)), _bf16(rng, (B, T, H, d)), _bf16(rng, (B, T, H, d))
    o0 = torch.zeros(B, H, d, dtype=torch.float32, device="cuda")
    ws_res, na_res = _pair(F, q, k, v, None, None, None, 700, 4, 64, o0)
    _same(ws_res, na_res, "dense")
    # call 2: a smaller sparse loop (B=1, T=900, H=2) over 300 of its columns, selecting 100
    B2, T2, H2 = 1, 900, 2
    say(f"noalloc d={d}: sparse B={B2} T={T2} H={H2}")
    q2, k2, v2 = _bf16(rng, (B2, H2, d)), _bf16(rng, (B2, T2, H2, d)), _bf16(rng, (B2, T2, H2, d))
    cols = torch.from_numpy(np.stack([np.stack([np.sort(rng.choice(T2, 300, replace=False)) for _ in range(H2)])
                                      for _ in range(B2)]).astype(np.int32)).cuda()
    mass = torch.from_numpy(rng.uniform(0.5, 1.0, (B2, H2)).astype(np.float32)).cuda()
    sub = torch.from_numpy((rng.standard_normal((B2, H2, d)) * 0.1).astype(np.float32)).cuda()
    o2 = torch.from_numpy((rng.standard_normal((B2, H2, d)) * 0.1).astype(np.float32)).cuda()
    ws_res, na_res = _pair(F, q2, k2, v2, cols, mass, sub, 100, 4, 16, o2)
    _same(ws_res, na_res, "sparse")
    # call 3: the larger dense call again, after the smaller one
    say(f"noalloc d={d}: dense again")
    ws_res, na_res = _pair(F, q, k, v, None, None, None, 0, 4, 64, o0)
    _same(ws_res, na_res, "dense, no selection")


def test_noalloc_rejects_a_step_beyond_its_scratch(F):
    B, T, H, d = 1, 65536, 40, 64
    assert F.load().fl_decode_step_ws(B, T, H, d, 0, 16) > 32 << 20
    k = torch.empty(B, T, H, d, dtype=torch.bfloat16, device="cuda")
    q = torch.empty(B, H, d, dtype=torch.bfloat16, device="cuda")
    o = torch.zeros(B, H, d, dtype=torch.float32, device="cuda")
    with pytest.raises(F.FlashLoopError, match="scratch"):
        F.decode_step_noalloc(q, k, k, None, None, None, o, 16)

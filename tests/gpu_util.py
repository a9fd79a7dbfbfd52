"""Host<->device helpers and the float tolerance used by the GPU parity tests.

Tolerance (attention outputs, log-normalisers): max-abs error <= 1e-2 and relative Frobenius error
<= 2e-3 against the fp64 oracle.  Integer and bit-pattern results (indices, slots, codes, fp16
metadata, reconstructed bf16 K/V) must be identical.
"""
import sys

import numpy as np
import torch

MAX_ABS = 1e-2
REL_FRO = 2e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def up_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def up(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def down_bits16(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def down(t):
    return t.cpu().numpy()


def f16_bits(a):
    return np.ascontiguousarray(a).astype(np.float16).view(np.uint16)


def assert_close(got, want, what, max_abs=MAX_ABS, rel_fro=REL_FRO):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    err = got - want
    mab = float(np.max(np.abs(err))) if err.size else 0.0
    den = float(np.linalg.norm(want))
    rf = float(np.linalg.norm(err)) / den if den > 0 else float(np.linalg.norm(err))
    say(f"  {what}: max_abs={mab:.3e} rel_fro={rf:.3e}")
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert mab <= max_abs, f"{what}: max abs error {mab:.3e} > {max_abs}"
    assert rf <= rel_fro, f"{what}: relative Frobenius error {rf:.3e} > {rel_fro}"
    return mab, rf


def assert_keys_close(got, want, what):
    """fp32 selection keys: identical up to one ulp (two fp64 summation orders)."""
    got = np.asarray(got, np.float32)
    want = np.asarray(want, np.float32)
    diff = np.abs(got.astype(np.float64) - want.astype(np.float64))
    ulp = np.spacing(np.abs(want)).astype(np.float64)
    n_off = int(np.sum(diff > 0))
    say(f"  {what}: {n_off} of {want.size} keys differ (<= 1 ulp allowed)")
    assert np.all(diff <= ulp), f"{what}: key differs by more than one ulp"


def new_rows(out, name, cache):
    """The loop's reconstructed rows X_hat^(r)[idx] as [B, k, H, d] bf16 bits: the compact rows the quantizer
    wrote, or (a loop that committed straight into the caches) the cache rows at idx."""
    if out[name] is not None:
        return down_bits16(out[name])
    idx = down(out["idx"])
    c = down_bits16(cache)
    return np.stack([c[b, idx[b]] for b in range(idx.shape[0])])

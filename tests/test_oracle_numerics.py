"""Pins of the oracle's rounding helpers against a library routine (torch's CPU bfloat16 cast).

f32_to_bf16 defines the round-to-nearest-even reconstruction of Appendix D.3, Eq. (8) (the bf16 state
X_hat = bf16(fp32(X_hat) + z + q s)), on which every bit-exact cache and the next loop's codes depend.
torch's CPU `.to(torch.bfloat16)` rounds fp32 to nearest with ties to even, so the two must agree bit for
bit on every finite input: random values over every binade, exact halfway cases with an even and an odd
retained bit, values just off the halfway point, subnormals, signed zeros and the largest finite values
(whose ties round up to infinity).  A truncating or ties-away rounding fails the halfway cases.
"""
import numpy as np
import torch

from oracle.numerics import bf16_to_f32, f32_to_bf16


def _torch_bf16_bits(u32: np.ndarray) -> np.ndarray:
    x = torch.from_numpy(u32.view(np.float32).copy())
    return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _check(u32: np.ndarray):
    u32 = np.ascontiguousarray(u32, dtype=np.uint32)
    got = f32_to_bf16(u32.view(np.float32))
    want = _torch_bf16_bits(u32)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (f"{bad.size} mismatches, first input 0x{int(u32[bad[0]]):08x}: "
                           f"oracle 0x{int(got[bad[0]]):04x}, torch 0x{int(want[bad[0]]):04x}")


def test_random_values_over_every_binade():
    rng = np.random.default_rng(0)
    n = 400_000
    sign = rng.integers(0, 2, n, dtype=np.uint32) << np.uint32(31)
    expo = rng.integers(0, 255, n, dtype=np.uint32) << np.uint32(23)      # 0 .. 254: finite only
    mant = rng.integers(0, 1 << 23, n, dtype=np.uint32)
    _check(sign | expo | mant)


def test_halfway_cases_round_to_even():
    rng = np.random.default_rng(1)
    hi = rng.integers(0, 0x7F80, 50_000, dtype=np.uint32)                # finite upper halves
    hi = np.concatenate([hi, hi ^ np.uint32(1)])                         # both parities of the kept bit
    sign = rng.integers(0, 2, hi.size, dtype=np.uint32) << np.uint32(31)
    base = sign | (hi << np.uint32(16))
    cases = [base | np.uint32(0x8000),                                   # exact ties
             base | np.uint32(0x7FFF), base | np.uint32(0x8001),        # just below / above a tie
             base, base | np.uint32(0x0001), base | np.uint32(0xFFFF)]
    _check(np.concatenate(cases))
    # the tie rule itself, spelled out on two values: 1 + 2^-8 (kept bit even) stays at 1, 1 + 3 * 2^-8
    # (kept bit odd) goes up to 1 + 2^-6
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3.0 * 2.0 ** -8], dtype=np.float32)
    np.testing.assert_array_equal(bf16_to_f32(f32_to_bf16(x)), np.array([1.0, 1.0 + 2.0 ** -6], dtype=np.float32))


def test_subnormals_zeros_and_the_largest_finite_values():
    sub = np.arange(0, 1 << 23, 997, dtype=np.uint32)                    # subnormals and +0
    top = np.arange(0x7F7F0000, 0x7F800000, 3, dtype=np.uint32)          # up to the largest finite fp32
    vals = np.concatenate([sub, top, np.array([0x7F7F7FFF, 0x7F7F8000, 0x7F7FFFFF, 0x00008000,
                                               0x00018000], dtype=np.uint32)])
    _check(np.concatenate([vals, vals | np.uint32(0x80000000)]))
    # ties above the largest finite bf16 round to infinity, as IEEE rounding to nearest does
    assert f32_to_bf16(np.array([0x7F7F8000], dtype=np.uint32).view(np.float32))[0] == 0x7F80


def test_bf16_to_f32_is_exact_on_every_finite_pattern():
    pats = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = (pats & 0x7F80) != 0x7F80
    pats = pats[finite]
    want = torch.from_numpy(pats.view(np.int16).copy()).view(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(bf16_to_f32(pats).view(np.uint32), want.view(np.uint32))
    # and the cast back is the identity
    np.testing.assert_array_equal(f32_to_bf16(bf16_to_f32(pats)), pats)

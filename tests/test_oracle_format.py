"""Pins for the oracle's number formats: bf16 decode and binary64 -> bf16
round-to-nearest-even, checked against torch's own conversions and against a
brute-force nearest search in exact rational arithmetic."""
from fractions import Fraction

import numpy as np
import torch

import oracle


def _bf16_bits_from_torch(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_decode_matches_torch():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_round_fp32_exact_inputs_matches_torch_rne():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(200000).astype(np.float32)
    # plant exact ties: lower 16 bits = 0x8000, both parities of the kept bit
    u = x.view(np.uint32).copy()
    u[:1000] = (u[:1000] & 0xFFFF0000) | 0x8000
    u[1000:2000] = (u[1000:2000] & 0xFFFE0000) | 0x00018000
    x = u.view(np.float32)
    ours = oracle.f64_to_bf16(x.astype(np.float64))
    assert np.array_equal(ours, _bf16_bits_from_torch(x))


def _nearest_bf16_bruteforce(v: float) -> int:
    """Nearest bf16 to v among all finite bf16 values near it, ties to even,
    in exact rational arithmetic."""
    t = np.array([v], dtype=np.float32)  # a nearby fp32 to locate the neighbourhood
    base = int(t.view(np.uint32)[0] >> 16)
    best = None
    fv = Fraction(v)
    for cand in range(max(0, (base & 0x7FFF) - 2), min(0x7F7F, (base & 0x7FFF) + 3) + 1):
        bits = (base & 0x8000) | cand
        c = Fraction(float(oracle.bf16_to_f64(np.array([bits], dtype=np.uint16))[0]))
        dist = abs(fv - c)
        key = (dist, cand & 1)  # on a tie, the even mantissa wins
        if best is None or key < best[0]:
            best = (key, bits)
    return best[1]


def test_round_binary64_bruteforce():
    rng = np.random.default_rng(2)
    vals = list(rng.standard_normal(3000) * np.exp(rng.uniform(-30, 30, 3000)))
    # binary64 values just off a bf16 halfway point: a route through fp32 would
    # round them to the tie first and then to even, which is wrong
    for m in range(1, 200):
        lo = 1.0 + (2 * m) / 256.0          # an even-mantissa bf16 value in [1, 2)
        half = lo + 1.0 / 256.0             # the exact midpoint to the next value
        vals += [half, half + 2.0 ** -40, half - 2.0 ** -40, -half - 2.0 ** -40]
    ours = oracle.f64_to_bf16(np.array(vals))
    for v, o in zip(vals, ours):
        assert int(o) == _nearest_bf16_bruteforce(float(v)), v


def test_round_specials():
    big = float(np.finfo(np.float32).max)
    vals = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 2.0 ** 128, big,
                     3.3895313892515355e38,   # largest finite bf16
                     2.0 ** -133, 2.0 ** -134, 2.0 ** -134 * 1.5, 2.0 ** -126])
    out = oracle.f64_to_bf16(vals)
    assert out[0] == 0x0000 and out[1] == 0x8000
    assert out[2] == 0x7F80 and out[3] == 0xFF80
    assert (out[4] & 0x7F80) == 0x7F80 and (out[4] & 0x007F) != 0
    assert out[5] == 0x7F80 and out[6] == 0x7F80   # fp32 max rounds up to inf in bf16
    assert out[7] == 0x7F7F
    assert out[8] == 0x0001                         # smallest bf16 subnormal
    assert out[9] == 0x0000                         # half of it: tie to even (zero)
    assert out[10] == 0x0001                        # above the tie
    assert out[11] == 0x0080                        # smallest normal

"""Pins of the oracle's rounding primitives against library casts and exact arithmetic."""
from fractions import Fraction

import numpy as np
import torch

from oracle.numerics import bf16_round, fp16_round


def _structured_f32():
    """Bit patterns around bf16 ties, carries into the exponent, subnormals, signs."""
    his = np.array([0x0000, 0x0001, 0x007F, 0x0080, 0x3F80, 0x3FFF, 0x4049, 0x7F7E, 0x7F00,
                    0x8001, 0xBF80, 0xC2F6, 0x3C23, 0x0100], dtype=np.uint32)
    los = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x7FFE, 0xC000, 0x4000],
                   dtype=np.uint32)
    bits = (his[:, None] << 16 | los[None, :]).ravel()
    return bits.view(np.float32)


def test_bf16_matches_torch_cast_structured_and_random():
    rng = np.random.default_rng(1)
    rnd = rng.integers(0, 2**32, size=2_000_000, dtype=np.uint64).astype(np.uint32)
    # keep finite values only (no NaN / Inf inputs)
    rnd = rnd[((rnd >> 23) & 0xFF) != 0xFF]
    x = np.concatenate([_structured_f32(), rnd.view(np.float32)])
    x = x[np.isfinite(x) & (np.abs(x) < 3.3e38)]
    ours = bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def _nearest_bf16_exact(v: float) -> float:
    """Nearest bf16 to the float64 v by exact rational comparison, ties to even."""
    if v == 0.0:
        return 0.0
    f = Fraction(v)
    sign = -1 if f < 0 else 1
    a = abs(f)
    e = 0
    while a >= 2:
        a /= 2
        e += 1
    while a < 1:
        a *= 2
        e -= 1
    # a in [1, 2): bf16 keeps 7 fraction bits
    scaled = a * 128
    lo = int(scaled)
    hi = lo + 1
    dlo, dhi = scaled - lo, hi - scaled
    m = lo if (dlo < dhi or (dlo == dhi and lo % 2 == 0)) else hi
    return float(sign * Fraction(m, 128) * Fraction(2) ** e)


def test_bf16_from_float64_is_direct_rounding():
    rng = np.random.default_rng(2)
    vals = list(rng.normal(0, 3, 3000)) + list(rng.normal(0, 1e-3, 500))
    # float64 values just off a bf16 tie, where rounding through float32 would round twice
    for base in (1.0, 1.5, 3.0, -2.0, 0.0078125):
        tie = base * (1 + 2.0 ** -8)            # exact midpoint between two bf16 values
        vals += [tie, tie + abs(base) * 2.0 ** -40, tie - abs(base) * 2.0 ** -40]
    x = np.array(vals, dtype=np.float64)
    got = bf16_round(x).astype(np.float64)
    want = np.array([_nearest_bf16_exact(float(v)) for v in x])
    assert np.array_equal(got, want)


def test_fp16_matches_torch_half_and_exact():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.normal(0, 1, 100000), rng.normal(0, 1e-5, 10000),
                        rng.uniform(-60000, 60000, 10000)]).astype(np.float32)
    ours = fp16_round(x)
    ref = torch.from_numpy(x).to(torch.float16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)
    # ties: 1 + 2^-11 is halfway between 1 and 1 + 2^-10 -> even (1.0)
    assert fp16_round(np.float32(1 + 2 ** -11)) == 1.0
    assert fp16_round(np.float32(1 + 3 * 2 ** -11)) == np.float32(1 + 2 ** -9)

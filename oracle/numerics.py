"""Rounding primitives of the oracle -- test infrastructure only.

The paper names FP16 as the unquantised format (Sec. 3.2); the build stores
activations and weights as bf16 and scales as fp16.  Both roundings are
round-to-nearest, ties-to-even.  Pinned against torch's CPU bfloat16 cast and
numpy's float16 cast (library routines) in tests/test_oracle_numerics.py.
"""
import numpy as np


def bf16_round(x) -> np.ndarray:
    """Round to the nearest bf16 value (ties to even); returns float32.

    float32 input: integer rounding of the bit pattern.  float64 input is
    rounded directly (not via float32, which could round twice): scale the
    value so that its 8 significant bits sit left of the binary point, rint,
    scale back; every step but rint is exact."""
    a = np.asarray(x)
    if a.dtype == np.float64:
        m, e = np.frexp(a)                       # a = m * 2^e, 0.5 <= |m| < 1
        r = np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)
        return r.astype(np.float32)
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns (uint16) of bf16-valued float32 data."""
    a = np.ascontiguousarray(bf16_round(x), dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def fp16_round(x) -> np.ndarray:
    """Round a float32 value to the nearest fp16 (ties to even); returns float32."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)


def rint_even(x) -> np.ndarray:
    """Round to the nearest integer, ties to even (IEEE roundTiesToEven)."""
    return np.rint(x)

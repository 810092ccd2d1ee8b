"""Seeded synthetic inputs shared by the oracle and the tests/bench of the HIP path.

This module draws numbers and nothing else: no quantisation, normalisation or
any other arithmetic of the fingerprint layer lives here.  The fingerprint's
Generator (paper, Sec. 5.1) reads a real checkpoint; no checkpoint is available,
so weights, gains and prompt hidden states are synthesised from a seed by a
counter-based generator that any implementation can reproduce bit for bit.

Generator (SplitMix64 of Steele, Lea & Flood, OOPSLA 2014, as a hash):
    key   = mix64(mix64(seed) + G*(((layer+1) << 8) | tensor))
    word c = mix64(key + G*(c+1)),  element i uses words 3i, 3i+1, 3i+2
    S = sum of their twelve unsigned 16-bit lanes (Irwin-Hall of 12 uniforms)
    z = float32(S - 393210) * 2^-16          (exact; mean 0, variance 1 - 2^-32)
    value = bf16_rne(float32(mean + float32(sigma * z)))

Conventions: weights use mean 0, sigma 0.02; norm gains mean 1, sigma 0.02;
prompt hidden states use layer -1, tensor 15, mean 0, sigma 1.  Elements are
numbered row-major over the tensor's shape.

The C build (``_fpgen.so``, compiled by ``build()``) is used when present; the
numpy implementation below is the same algorithm and is kept for small sizes
and as the cross-check.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1

# tensor ids used throughout (the C ABI uses the same numbering)
T_ATTN_NORM, T_Q, T_K, T_V, T_O, T_MLP_NORM, T_GATE, T_UP, T_DOWN = range(9)
T_INPUT = 15
# the blocks outside the hidden layers (layer id -1): token embedding [vocab, hidden],
# final norm gain [hidden], LM head [vocab, hidden]
T_EMBED, T_FINAL_NORM, T_LM_HEAD = 16, 17, 18

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "_fpgen.so")
_lib = None


def build_c(verbose: bool = False) -> str:
    """Compile fpgen.c into _fpgen.so with gcc (OpenMP, no FP contraction)."""
    import subprocess
    src = os.path.join(_HERE, "fpgen.c")
    tmp = _SO + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared", src, "-o", tmp]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(tmp, _SO)
    global _lib
    _lib = None
    return _SO


def _load():
    global _lib
    if _lib is None and os.path.exists(_SO):
        lib = ctypes.CDLL(_SO)
        lib.fpgen_mix64.restype = ctypes.c_uint64
        lib.fpgen_mix64.argtypes = [ctypes.c_uint64]
        lib.fpgen_key.restype = ctypes.c_uint64
        lib.fpgen_key.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32]
        lib.fpgen_z.restype = None
        lib.fpgen_z.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                ctypes.c_int64, ctypes.c_void_p]
        lib.fpgen_bf16.restype = None
        lib.fpgen_bf16.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                   ctypes.c_int64, ctypes.c_float, ctypes.c_float, ctypes.c_void_p]
        _lib = lib
    return _lib


def have_c() -> bool:
    return _load() is not None


# ----------------------------------------------------------------- numpy path
def mix64_np(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=True)
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= np.uint64(0xBF58476D1CE4E5B9)
        z ^= z >> np.uint64(27)
        z *= np.uint64(0x94D049BB133111EB)
        z ^= z >> np.uint64(31)
    return z


def mix64(z: int) -> int:
    z &= MASK64
    z ^= z >> 30
    z = (z * 0xBF58476D1CE4E5B9) & MASK64
    z ^= z >> 27
    z = (z * 0x94D049BB133111EB) & MASK64
    z ^= z >> 31
    return z


def key(seed: int, layer: int, tensor: int) -> int:
    ident = (((layer + 1) << 8) | tensor) & MASK64
    return mix64((mix64(seed) + GAMMA * ident) & MASK64)


def z_np(seed: int, layer: int, tensor: int, start: int, n: int) -> np.ndarray:
    k = np.uint64(key(seed, layer, tensor))
    i = np.arange(start, start + n, dtype=np.uint64)
    s = np.zeros(n, dtype=np.int64)
    with np.errstate(over="ignore"):
        for c in range(3):
            w = mix64_np(k + np.uint64(GAMMA) * (np.uint64(3) * i + np.uint64(c + 1)))
            for sh in (0, 16, 32, 48):
                s += ((w >> np.uint64(sh)) & np.uint64(0xFFFF)).astype(np.int64)
    return (s - 393210).astype(np.float32) * np.float32(1.0 / 65536.0)


def _bf16_rne_bits_np(f: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_np(seed, layer, tensor, start, n, mean, sigma) -> np.ndarray:
    z = z_np(seed, layer, tensor, start, n)
    v = np.float32(mean) + np.float32(sigma) * z          # two separately rounded fp32 ops
    return _bf16_rne_bits_np(v.astype(np.float32))


# ------------------------------------------------------------- public helpers
def z_scores(seed: int, layer: int, tensor: int, n: int, start: int = 0) -> np.ndarray:
    lib = _load()
    if lib is None:
        return z_np(seed, layer, tensor, start, n)
    out = np.empty(n, dtype=np.float32)
    lib.fpgen_z(seed & MASK64, layer, tensor, start, n, out.ctypes.data)
    return out


def bf16_bits(seed: int, layer: int, tensor: int, n: int, mean: float, sigma: float,
              start: int = 0) -> np.ndarray:
    """uint16 bf16 bit patterns of elements [start, start+n) of one stream."""
    lib = _load()
    if lib is None:
        return bf16_bits_np(seed, layer, tensor, start, n, mean, sigma)
    out = np.empty(n, dtype=np.uint16)
    lib.fpgen_bf16(seed & MASK64, layer, tensor, start, n, float(mean), float(sigma), out.ctypes.data)
    return out


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to exactly equal float32 values."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def weight(seed: int, layer: int, tensor: int, shape) -> np.ndarray:
    """Synthetic weight ~N(0, 0.02), bf16-valued float32 array of ``shape`` ([N, K] row-major)."""
    n = int(np.prod(shape))
    return bits_to_f32(bf16_bits(seed, layer, tensor, n, 0.0, 0.02)).reshape(shape)


def gain(seed: int, layer: int, tensor: int, n: int) -> np.ndarray:
    """Synthetic norm gain 1 + N(0, 0.02), bf16-valued float32 array [n]."""
    return bits_to_f32(bf16_bits(seed, layer, tensor, n, 1.0, 0.02))


def prompt(seed: int, B: int, P: int, H: int, b_start: int = 0, b_count: int | None = None) -> np.ndarray:
    """Prompt hidden states ~N(0,1) [b_count, P, H] (rows b_start.. of the [B, P, H] stream)."""
    if b_count is None:
        b_count = B - b_start
    n = b_count * P * H
    bits = bf16_bits(seed, -1, T_INPUT, n, 0.0, 1.0, start=b_start * P * H)
    return bits_to_f32(bits).reshape(b_count, P, H)


T_TOKENS = 19


def token_ids(seed: int, n: int, vocab: int, start: int = 0) -> np.ndarray:
    """Synthetic prompt token ids, uniform over [0, vocab): element i is the top 32 bits of
    word mix64(key(seed, -1, 19) + G*(i+1)), times vocab, over 2^32 (int32 [n])."""
    k = np.uint64(key(seed, -1, T_TOKENS))
    i = np.arange(start, start + n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        w = mix64_np(k + np.uint64(GAMMA) * (i + np.uint64(1)))
    hi = (w >> np.uint64(32)).astype(np.uint64)
    return ((hi * np.uint64(vocab)) >> np.uint64(32)).astype(np.int32)

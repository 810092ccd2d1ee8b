"""Weight and KV-cache quantisers of the oracle -- test infrastructure only.

The paper's compression menu (Sec. 3.2, Table A.1): INT8 and INT4 weight-only
quantisation (memory -50% / -75%) and an INT8 KV cache.  It gives no formulas;
the readings below are the ones the build fixes:

* int8 weights, symmetric per output channel (row n of W[N, K]):
      s_n  = fp16(absmax_k |W[n,k]| / 127)          (fp32 division, then RNE)
      code = clamp(rint(W / float(s_n)), -127, 127)  (IEEE fp32 division)
  absmax = 0 gives s = 0 and all-zero codes.  Dequantised weight = code * s
  (exact in fp32).
* int4 weights, asymmetric per group of 128 consecutive k in a row:
      lo = min(0, min w), hi = max(0, max w)
      s  = fp16((hi - lo) / 15); s = 1 if hi == lo
      z  = clamp(rint(-lo / s), 0, 15)            (integer zero point, stored fp16)
      q  = clamp(rint(w / s) + z, 0, 15)          (rint before adding z)
  Dequantised weight = (q - z) * s.
* int4 packing: nibble j of int32 word [n, w] holds the code at k = 8w + j in
  bits 4j..4j+3; codes [N, K/8] int32, scales and zeros [N, K/128] fp16.
* int8 KV: per (sequence, position, kv head), separately for K (after the
  rotary embedding) and V, the int8 rule above over the head_dim elements.

* 2:4 semi-structured sparsity (the pruning of Sec. 3.3, Table A.1: 2 of every 4
  weights zero), scored by magnitude: in each group of 4 consecutive k of a row the
  2 weights of largest |w| are kept, the lower k first among equal magnitudes, and
  the other 2 set to zero.  The kept weights stay bf16.  Compressed form: the kept
  values of each group in k order, [N, K/2], and their positions in the group
  (0..3, first < second), [N, K/2].

Pins (tests/test_oracle_quant.py): brute-force nearest-code search over every
code, the |w - w_hat| <= s/2 bound, exact grids, pack/unpack round trips, and
exact ties (w / s = k + 1/2 with power-of-two scales): int8 codes and int8 KV
codes go to the even neighbour, int4 rounds to the even integer before the odd
zero point is added, and a tie in -lo / s gives the even zero point.
"""
import numpy as np

from .numerics import fp16_round, rint_even

F32 = np.float32


def quant_int8_rows(w: np.ndarray):
    """Symmetric int8 over the last axis.  Returns (codes int8, scales fp16-valued float32)."""
    w = np.asarray(w, dtype=F32)
    absmax = np.max(np.abs(w), axis=-1, keepdims=True)
    s = fp16_round(absmax / F32(127.0))
    safe = np.where(s == 0, F32(1.0), s)
    codes = np.clip(rint_even(w / safe), -127, 127)
    codes = np.where(s == 0, 0.0, codes).astype(np.int8)
    return codes, s[..., 0].astype(F32)


def quant_int8_channel(w: np.ndarray):
    """int8 per-output-channel weight quantisation of W[N, K]."""
    return quant_int8_rows(w)


def dequant_int8_channel(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    return codes.astype(F32) * scales.astype(F32)[..., None]


def quant_int4_g128(w: np.ndarray, group: int = 128):
    """int4 asymmetric group-128 quantisation of W[N, K].

    Returns (codes uint8 [N, K] in 0..15, scales [N, K/128], zeros [N, K/128]),
    scales fp16-valued float32, zeros integer-valued float32."""
    w = np.asarray(w, dtype=F32)
    N, K = w.shape
    assert K % group == 0
    g = w.reshape(N, K // group, group)
    lo = np.minimum(F32(0.0), g.min(axis=-1))
    hi = np.maximum(F32(0.0), g.max(axis=-1))
    s = fp16_round((hi - lo) / F32(15.0))
    s = np.where(hi == lo, F32(1.0), s).astype(F32)
    z = np.clip(rint_even(-lo / s), 0, 15).astype(F32)
    q = np.clip(rint_even(g / s[..., None]) + z[..., None], 0, 15).astype(np.uint8)
    return q.reshape(N, K), s, z


def dequant_int4_g128(q: np.ndarray, s: np.ndarray, z: np.ndarray, group: int = 128) -> np.ndarray:
    N, K = q.shape
    g = q.reshape(N, K // group, group).astype(F32)
    return ((g - z[..., None]) * s[..., None]).reshape(N, K).astype(F32)


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Pack codes [N, K] (0..15) into int32 words [N, K/8]; nibble j <-> k = 8w + j."""
    N, K = q.shape
    assert K % 8 == 0
    q = q.astype(np.uint32).reshape(N, K // 8, 8)
    word = np.zeros((N, K // 8), dtype=np.uint32)
    for j in range(8):
        word |= (q[..., j] & 0xF) << np.uint32(4 * j)
    return word.view(np.int32)


def unpack_int4(words: np.ndarray) -> np.ndarray:
    """Inverse of pack_int4: int32 words [N, K/8] -> codes uint8 [N, K]."""
    w = np.ascontiguousarray(words).view(np.uint32)
    N, W = w.shape
    out = np.empty((N, W, 8), dtype=np.uint8)
    for j in range(8):
        out[..., j] = (w >> np.uint32(4 * j)) & 0xF
    return out.reshape(N, W * 8)


def quant_kv_int8(x: np.ndarray):
    """int8 KV quantisation over the last (head_dim) axis of fp32 K or V.

    Returns (codes int8, scales fp16-valued float32 with the last axis removed)."""
    return quant_int8_rows(np.asarray(x, dtype=F32))


def prune_2of4(w: np.ndarray) -> np.ndarray:
    """Magnitude 2:4 mask of W[N, K] (K a multiple of 4): True for the two weights of
    largest |w| in each group of 4 consecutive k, the lower k first among equal |w|."""
    w = np.asarray(w, dtype=F32)
    N, K = w.shape
    assert K % 4 == 0
    g = np.abs(w).reshape(N, K // 4, 4)
    # rank by (-|w|, k): a stable sort on -|w| keeps the lower k first among ties
    order = np.argsort(-g, axis=-1, kind="stable")
    mask = np.zeros_like(g, dtype=bool)
    np.put_along_axis(mask, order[..., :2], True, axis=-1)
    return mask.reshape(N, K)


def compress_2of4(w: np.ndarray, mask: np.ndarray):
    """(values [N, K/2], positions [N, K/2]) of the kept weights, in k order per group."""
    N, K = w.shape
    pos = np.nonzero(mask.reshape(N, K // 4, 4))[2].reshape(N, K // 4, 2)
    vals = np.take_along_axis(np.asarray(w, dtype=F32).reshape(N, K // 4, 4), pos, axis=-1)
    return vals.reshape(N, K // 2), pos.reshape(N, K // 2).astype(np.uint8)


def decompress_2of4(vals: np.ndarray, pos: np.ndarray) -> np.ndarray:
    N, K2 = vals.shape
    out = np.zeros((N, K2 // 2, 4), dtype=F32)
    np.put_along_axis(out, pos.reshape(N, K2 // 2, 2).astype(np.int64), vals.reshape(N, K2 // 2, 2), axis=-1)
    return out.reshape(N, 2 * K2)

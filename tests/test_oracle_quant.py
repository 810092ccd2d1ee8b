"""Pins of the oracle's quantisers: brute-force nearest code, error bounds, exact grids,
int4 pack/unpack round trips."""
import os

import numpy as np

from oracle.quant import (quant_int8_channel, dequant_int8_channel, quant_int4_g128,
                          dequant_int4_g128, pack_int4, unpack_int4, quant_kv_int8)
from oracle.numerics import bf16_round

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _bf16_weights(rng, shape, sigma=0.02):
    return bf16_round(rng.normal(0, sigma, shape).astype(np.float32))


def test_int8_codes_are_brute_force_nearest():
    rng = np.random.default_rng(0)
    w = _bf16_weights(rng, (64, 256))
    codes, s = quant_int8_channel(w)
    cand = np.arange(-127, 128, dtype=np.float64)
    for n in range(w.shape[0]):
        err = np.abs(w[n].astype(np.float64)[:, None] - cand[None, :] * float(s[n]))
        best = err.min(axis=1)
        mine = np.abs(w[n].astype(np.float64) - codes[n].astype(np.float64) * float(s[n]))
        assert np.array_equal(mine, best)
    # the absmax element lands on +-127 and the scale is absmax/127 to fp16 precision
    am = np.abs(w).max(axis=1)
    assert np.all(np.abs(codes).max(axis=1) == 127)
    assert np.all(np.abs(s.astype(np.float64) * 127 / am - 1) <= 2.0 ** -11)


def test_int8_error_bound_and_grid():
    rng = np.random.default_rng(1)
    w = _bf16_weights(rng, (32, 512))
    c, s = quant_int8_channel(w)
    deq = dequant_int8_channel(c, s)
    assert np.all(np.abs(w - deq) <= s[:, None] / 2)
    # exact multiples k*s quantise to k
    s0 = np.float32(0.0078125)
    k = np.arange(-127, 128).astype(np.float32)
    grid = (k * s0)[None, :]
    cg, sg = quant_int8_channel(grid)
    assert sg[0] == np.float32(127 * s0 / 127) and np.array_equal(cg[0], k.astype(np.int8))
    # all-zero row
    cz, sz = quant_int8_channel(np.zeros((1, 16), np.float32))
    assert sz[0] == 0 and not cz.any()


def test_int4_codes_are_brute_force_nearest_and_bounded():
    rng = np.random.default_rng(2)
    w = _bf16_weights(rng, (16, 512))
    q, s, z = quant_int4_g128(w)
    assert q.max() <= 15 and z.min() >= 0 and z.max() <= 15
    deq = dequant_int4_g128(q, s, z)
    sfull = np.repeat(s, 128, axis=1)
    zfull = np.repeat(z, 128, axis=1)
    err = np.abs(w.astype(np.float64) - deq.astype(np.float64))
    assert np.all(err <= sfull / 2 + 15 * 2.0 ** -11 * sfull)
    # brute force: no other code in 0..15 reconstructs strictly closer
    cand = np.arange(16, dtype=np.float64)
    allerr = np.abs(w.astype(np.float64)[..., None]
                    - (cand[None, None, :] - zfull[..., None]) * sfull[..., None])
    assert np.all(err <= allerr.min(axis=-1) + 1e-12 * sfull)
    # the range of every group contains 0 and z reproduces 0 exactly
    assert np.all((0 - z) * s == -(z * s))


def test_int4_exact_grid_and_zero_group():
    s0 = np.float32(0.00390625)
    zt = 5
    k = np.tile(np.arange(16, dtype=np.float32), 8)         # 128 values, codes 0..15
    w = ((k - zt) * s0)[None, :]
    q, s, z = quant_int4_g128(w)
    assert s[0, 0] == s0 and z[0, 0] == zt and np.array_equal(q[0], k.astype(np.uint8))
    assert np.array_equal(dequant_int4_g128(q, s, z), w)
    q0, s1, z0 = quant_int4_g128(np.zeros((2, 128), np.float32))
    assert np.all(s1 == 1.0) and np.all(z0 == 0) and not q0.any()
    # an all-positive group: lo = 0 -> z = 0
    q2, s2, z2 = quant_int4_g128(np.abs(_bf16_weights(np.random.default_rng(9), (1, 128))))
    assert z2[0, 0] == 0 and q2.max() == 15


def test_int4_pack_golden_and_round_trips():
    with open(os.path.join(GOLD, "int4_nibble_order.txt")) as f:
        lines = [l for l in f if not l.startswith("#")]
    codes = np.array([int(t) for t in lines[0].split(":")[1].split()], dtype=np.uint8)[None, :]
    words = [int(t, 16) for t in lines[1].split(":")[1].split()]
    packed = pack_int4(codes)
    assert [int(v) for v in packed.view(np.uint32)[0]] == words
    assert np.array_equal(unpack_int4(packed), codes)
    # every value in every nibble position
    allc = np.array([[(v + j) % 16 for j in range(8)] for v in range(16)], dtype=np.uint8)
    assert np.array_equal(unpack_int4(pack_int4(allc)), allc)
    rng = np.random.default_rng(4)
    wd = rng.integers(0, 2**32, size=(1000, 1250), dtype=np.uint64).astype(np.uint32)
    edge = np.array([[0, 0xFFFFFFFF, 0xAAAAAAAA, 0x55555555, 0x80000000, 0x00000001]], np.uint32)
    for arr in (wd, edge):
        assert np.array_equal(pack_int4(unpack_int4(arr.view(np.int32))).view(np.uint32), arr)


def test_kv_int8_per_head_bound():
    rng = np.random.default_rng(5)
    k = rng.normal(0, 1.3, (2, 3, 7, 128)).astype(np.float32)
    c, s = quant_kv_int8(k)
    assert c.shape == k.shape and s.shape == k.shape[:-1]
    assert np.all(np.abs(k - c.astype(np.float32) * s[..., None]) <= s[..., None] / 2)
    assert np.all(np.abs(c).max(axis=-1) == 127)


def test_int8_exact_ties_round_to_even():
    """w / s landing exactly on k + 1/2 goes to the even neighbour (round half to even),
    for both signs.  s = 2^-7 is exact in fp16, and the row's absmax 127 s makes
    fp16(absmax / 127) = s exactly, so every w / s below is an exact fp32 quotient."""
    s0 = np.float32(2.0 ** -7)
    half = np.arange(-126, 126, dtype=np.float64) + 0.5          # -125.5 .. 125.5
    w = np.concatenate([[127.0], half]) * float(s0)
    c, s = quant_int8_channel(w.astype(np.float32)[None, :])
    assert s[0] == s0
    want = 2.0 * np.round(half / 2.0)                               # the even neighbour
    assert np.all(np.abs(want - half) == 0.5) and np.all(want % 2 == 0)
    assert np.array_equal(c[0, 1:].astype(np.float64), want)
    # e.g. 0.5 -> 0, 1.5 -> 2, 2.5 -> 2, -0.5 -> 0, -1.5 -> -2, -2.5 -> -2
    idx = {v: i for i, v in enumerate(half)}
    assert [int(c[0, 1 + idx[v]]) for v in (0.5, 1.5, 2.5, -0.5, -1.5, -2.5)] == [0, 2, 2, 0, -2, -2]


def test_int4_ties_round_before_the_zero_point_is_added():
    """One 128-input group with lo = -5 s and hi = 10 s for s = 2^-6: the scale is
    fp16((hi - lo) / 15) = s exactly and the zero point z = 5 is odd.  Inputs at
    w / s = m + 1/2 round to the even m first and then add z; rounding after adding z
    (an odd offset) would pick the other neighbour every time."""
    s0 = np.float32(2.0 ** -6)
    ties = np.array([-4.5, -3.5, -2.5, -1.5, -0.5, 0.5, 1.5, 2.5, 3.5, 4.5, 5.5, 6.5, 7.5, 8.5, 9.5])
    vals = np.concatenate([[-5.0, 10.0], ties, np.zeros(128 - 2 - len(ties))])
    w = (vals * float(s0)).astype(np.float32)[None, :]
    q, s, z = quant_int4_g128(w)
    assert s[0, 0] == s0 and z[0, 0] == 5
    want = 2.0 * np.round(ties / 2.0) + 5                             # rint first, then + z
    assert np.array_equal(q[0, 2:2 + len(ties)].astype(np.float64), want)
    assert np.all(q[0, 2:2 + len(ties)] != np.round(ties + 5))       # the other order differs
    # a tie in the zero point itself: lo = -2.5 s, hi = 12.5 s -> s exact, z = rint(2.5) = 2
    vals2 = np.concatenate([[-2.5, 12.5, 1.5, -1.5], np.zeros(124)])
    q2, s2, z2 = quant_int4_g128((vals2 * float(s0)).astype(np.float32)[None, :])
    assert s2[0, 0] == s0 and z2[0, 0] == 2
    assert [int(v) for v in q2[0, :4]] == [0, 14, 4, 0]               # -2->0, 12->14, 2->4, -2->0


def test_kv_int8_ties_and_fp32_input():
    """The KV quantiser is the int8 row rule over head_dim: an exact tie goes to the even
    code, and the scale comes from the fp32 values as given (no prior bf16 rounding:
    1 + 2^-10 is not a bf16 value and must survive into the quotient)."""
    s0 = np.float32(2.0 ** -7)
    row = np.zeros(16, np.float64)
    row[0], row[1], row[2] = 127.0, 2.5, -3.5
    c, s = quant_kv_int8((row * float(s0)).astype(np.float32)[None, None, :])
    assert s[0, 0] == s0 and int(c[0, 0, 1]) == 2 and int(c[0, 0, 2]) == -4
    # 100.5 + 2^-3: above the tie in fp32, exactly the tie once rounded to bf16 (ulp 0.5 at 100)
    v = np.float32((100.5 + 2.0 ** -3) * float(s0))
    row2 = np.array([127.0 * float(s0), v] + [0.0] * 14, np.float32)
    c2, _ = quant_kv_int8(row2[None, None, :])
    assert int(c2[0, 0, 1]) == 101


def test_2of4_mask_keeps_the_two_largest_magnitudes_brute_force():
    """Every group of 4 keeps exactly 2; the kept pair has the largest sum of |w| among the
    6 possible pairs, and among pairs with the same kept magnitudes the lower positions
    win (the k order tie rule)."""
    import itertools
    from oracle.quant import prune_2of4
    rng = np.random.default_rng(11)
    w = _bf16_weights(rng, (40, 64))
    w[0, :8] = [0.5, -0.5, 0.5, 0.25, 0, 0, 0, 0]      # ties in magnitude and all-zero group
    w[1, :4] = [-1.0, 1.0, 1.0, -1.0]
    m = prune_2of4(w)
    assert m.shape == w.shape and np.all(m.reshape(40, 16, 4).sum(-1) == 2)
    pairs = list(itertools.combinations(range(4), 2))
    for n in range(w.shape[0]):
        for g in range(16):
            grp = np.abs(w[n, 4 * g:4 * g + 4]).astype(np.float64)
            # the best pair: sort positions by (-|w|, k) and take the first two
            want = tuple(sorted(sorted(range(4), key=lambda k: (-grp[k], k))[:2]))
            assert want in pairs
            got = tuple(np.nonzero(m[n, 4 * g:4 * g + 4])[0])
            assert got == want, (n, g, grp, got)
            kept = grp[list(got)].sum()
            assert all(kept >= grp[list(p)].sum() for p in pairs)
    assert tuple(np.nonzero(m[0, :4])[0]) == (0, 1) and tuple(np.nonzero(m[0, 4:8])[0]) == (0, 1)
    assert tuple(np.nonzero(m[1, :4])[0]) == (0, 1)


def test_2of4_compress_round_trip_and_bytes():
    from oracle.quant import prune_2of4, compress_2of4, decompress_2of4
    rng = np.random.default_rng(12)
    w = _bf16_weights(rng, (32, 256))
    m = prune_2of4(w)
    dense = np.where(m, w, 0).astype(np.float32)
    v, p = compress_2of4(dense, m)
    assert v.shape == (32, 128) and p.shape == (32, 128)
    assert np.all(p.reshape(32, 64, 2)[..., 0] < p.reshape(32, 64, 2)[..., 1]) and p.max() <= 3
    assert np.array_equal(decompress_2of4(v, p), dense)
    # half the bf16 values plus 2 bits per kept value: 9/16 of the dense bf16 bytes
    assert (v.size * 2 + p.size * 2 / 8) / (w.size * 2) == 9 / 16

"""Pins of the seeded input generator (SplitMix64 + Irwin-Hall-12)."""
import os

import numpy as np
import pytest

import fpgen

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _golden_words():
    with open(os.path.join(GOLD, "splitmix64_seed0.txt")) as f:
        return [int(l, 16) for l in f if l.strip() and not l.startswith("#")]


def test_mix64_published_sequence():
    want = _golden_words()
    got = [fpgen.mix64((fpgen.GAMMA * k) & fpgen.MASK64) for k in range(1, 6)]
    assert got == want
    got_np = fpgen.mix64_np(np.array([(fpgen.GAMMA * k) & fpgen.MASK64 for k in range(1, 6)],
                                     dtype=np.uint64))
    assert [int(v) for v in got_np] == want


def test_c_build_matches_numpy_and_python_ints():
    assert fpgen.have_c(), "gcc build of fpgen failed"
    lib = fpgen._load()
    for z in (0, 1, fpgen.GAMMA, 2**64 - 1, 0x0123456789ABCDEF):
        assert lib.fpgen_mix64(z) == fpgen.mix64(z)
    for (seed, layer, tensor) in [(0, 0, 1), (0, -1, 15), (7, 3, 8), (2**63 + 5, 1, 0)]:
        assert lib.fpgen_key(seed & fpgen.MASK64, layer, tensor) == fpgen.key(seed, layer, tensor)
        for mean, sigma in [(0.0, 0.02), (1.0, 0.02), (0.0, 1.0)]:
            a = fpgen.bf16_bits(seed, layer, tensor, 5000, mean, sigma, start=123)
            b = fpgen.bf16_bits_np(seed, layer, tensor, 123, 5000, mean, sigma)
            assert np.array_equal(a, b)
        assert np.array_equal(fpgen.z_scores(seed, layer, tensor, 777, start=9),
                              fpgen.z_np(seed, layer, tensor, 9, 777))


def test_z_element_by_python_integers():
    """Element i of a stream summed from its three words with plain Python ints."""
    seed, layer, tensor = 0, 2, 6
    k = fpgen.key(seed, layer, tensor)
    z = fpgen.z_scores(seed, layer, tensor, 40)
    for i in (0, 1, 17, 39):
        s = 0
        for c in range(3):
            w = fpgen.mix64(k + fpgen.GAMMA * (3 * i + c + 1))
            s += sum((w >> sh) & 0xFFFF for sh in (0, 16, 32, 48))
        assert z[i] == np.float32(s - 393210) / np.float32(65536)


def test_irwin_hall_moments_and_support():
    z = fpgen.z_scores(0, 0, 1, 1_000_000).astype(np.float64)
    n = z.size
    assert abs(z.mean()) < 5 / np.sqrt(n)
    # var of the sample variance of a distribution with kurtosis 3 - 1.2/12 ... use 5 sigma
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / n)
    assert np.abs(z).max() <= 6.0
    # exact lattice: z * 2^16 is an integer
    assert np.all(np.floor(z * 65536) == z * 65536)


def test_value_conventions():
    w = fpgen.weight(0, 0, 1, (64, 128))
    assert w.dtype == np.float32 and w.shape == (64, 128)
    assert abs(w.std() - 0.02) < 0.002
    g = fpgen.gain(0, 0, 0, 4096)
    assert abs(g.mean() - 1.0) < 0.002
    # weight value is bf16(0.02f * z)
    z = fpgen.z_scores(0, 0, 1, 64 * 128)
    prod = (np.float32(0.02) * z).astype(np.float32)
    u = prod.view(np.uint32).astype(np.uint64)
    ref = (((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16).astype(np.uint32).view(np.float32)
    assert np.array_equal(w.ravel(), ref)


def test_prompt_rows_are_stream_slices():
    full = fpgen.prompt(0, 4, 8, 32)
    part = fpgen.prompt(0, 4, 8, 32, b_start=2, b_count=1)
    assert np.array_equal(full[2:3], part)

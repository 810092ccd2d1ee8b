"""Pins of the oracle's blocks outside the hidden layers (embedding gather, final RMSNorm,
LM head, greedy argmax) and of a token-level dummy request."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

import fpgen
from fpgen.workloads import Shape
from oracle.layer import Fingerprint, argmax_first
from oracle.numerics import bf16_round

SH = Shape(2, 128, 4, 2, 32, 256, 2, 12, 24, vocab=512)


def test_embedding_is_a_row_gather():
    fp = Fingerprint(SH, "int4", "int8")
    ids = fpgen.token_ids(1, 40, SH.vocab).reshape(2, 20)
    got = fp.embed(ids)
    ref = Fnn.embedding(torch.from_numpy(ids.astype(np.int64)), torch.from_numpy(fp.embed_table)).numpy()
    assert np.array_equal(got, ref)
    # the table is the generator's bf16 stream (seed, layer -1, tensor 16), as are the
    # final gain and the LM head (16-bit under every weight format)
    assert np.array_equal(fp.embed_table, fpgen.weight(0, -1, 16, (SH.vocab, SH.hidden)))
    assert np.array_equal(fp.lm_head, fpgen.weight(0, -1, 18, (SH.vocab, SH.hidden)))
    assert np.array_equal(fp.final_norm, fpgen.gain(0, -1, 17, SH.hidden))
    with pytest.raises(AssertionError):
        fp.embed(np.array([SH.vocab]))


def test_head_matches_torch_linear_over_rms_norm():
    fp = Fingerprint(SH, "bf16", "bf16")
    y = bf16_round(np.random.default_rng(0).normal(0, 1.5, (3, SH.hidden)).astype(np.float32))
    logits, ids = fp.head(y)
    yt = torch.from_numpy(y.astype(np.float64))
    yn = Fnn.rms_norm(yt, (SH.hidden,), weight=torch.from_numpy(fp.final_norm.astype(np.float64)), eps=1e-5)
    yn = torch.from_numpy(bf16_round(yn.numpy()).astype(np.float64))
    ref = Fnn.linear(yn, torch.from_numpy(fp.lm_head.astype(np.float64))).numpy()
    assert np.allclose(logits, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(ids, np.argmax(ref, axis=-1))


def test_argmax_takes_the_lowest_index_among_equal_maxima():
    rng = np.random.default_rng(3)
    x = rng.normal(size=(50, 97))
    for row, got in zip(x, argmax_first(x)):
        best, idx = -np.inf, -1
        for j, v in enumerate(row):
            if v > best:
                best, idx = v, j
        assert got == idx
    t = np.array([[1.0, 3.0, 2.0, 3.0], [5.0, 5.0, 5.0, 5.0], [-1.0, -2.0, -1.0, -3.0]])
    assert list(argmax_first(t)) == [1, 0, 0]


@pytest.mark.parametrize("wq,kvq", [("bf16", "bf16"), ("int4", "int8")])
def test_generate_equals_full_recompute(wq, kvq):
    """Tokens of a KV-cached request equal what a prefill over the prompt and the
    generated tokens yields at every position (the KV cache only avoids recompute)."""
    fp = Fingerprint(SH, wq, kvq)
    ids = fpgen.token_ids(2, 2 * 8, SH.vocab).reshape(2, 8)
    toks, logits = fp.generate(ids, 6)
    assert toks.shape == (7, 2) and logits.shape == (7, 2, SH.vocab)
    full = np.concatenate([ids, toks[:-1].T], axis=1)            # prompt + tokens 0..5
    y = fp.prefill(fp.embed(full))
    for i in range(7):
        lg, tk = fp.head(y[:, 8 - 1 + i, :])
        assert np.allclose(lg, logits[i], rtol=1e-9, atol=1e-9), i
        assert np.array_equal(tk, toks[i]), i
    # a teacher equal to the generated tokens reproduces the free run
    toks2, logits2 = fp.generate(ids, 6, teacher=toks[:-1])
    assert np.array_equal(toks2, toks) and np.array_equal(logits2, logits)

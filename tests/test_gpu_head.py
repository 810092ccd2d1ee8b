"""Parity of the fingerprint's blocks outside the hidden layers (embedding gather, final
RMSNorm, LM head, greedy argmax) and of a token-level dummy request (fp_generate) with
the oracle.  Bars: bit-exact head weights and embedding rows; logits within 2e-2
normwise; every greedy decision is the argmax of the GPU's own fp32 logits (lowest id
on ties) and, given the logits error e, within 2e from the oracle's best logit (the
decision the oracle would accept).  Requests are teacher-forced on the oracle's tokens."""
import dataclasses

import numpy as np
import pytest

import fpgen
from fpgen.workloads import Shape, LLAMA2_VOCAB
from oracle.layer import Fingerprint as OracleFingerprint
from oracle.numerics import bf16_round
from tests.gpu_harness import TOL, log, rel_inf, bf16_to_np, np_to_bf16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2501_13111_amd as P
    P.load()
    yield


def _check_decisions(gpu_logits, gpu_ids, orc_logits, what):
    """gpu_ids is the argmax of the GPU's own logits, and a decision the oracle accepts."""
    gl = np.asarray(gpu_logits, np.float64)
    ol = np.asarray(orc_logits, np.float64)
    assert np.array_equal(gpu_ids, np.argmax(np.asarray(gpu_logits, np.float32), axis=-1)), what
    e = np.abs(gl - ol).max()
    for b, i in enumerate(gpu_ids):
        assert ol[b, i] >= ol[b].max() - 2 * e - 1e-12, (what, b, i, ol[b, i], ol[b].max(), e)


def test_head_weights_and_embedding_rows_bit_exact():
    import torch
    from paper_2501_13111_amd import Fingerprint
    s = Shape(1, 256, 4, 4, 64, 384, 3, 16, 24, vocab=1024)
    orc = OracleFingerprint(s, "int4", "int8", seed=13)
    with Fingerprint(s, "int4", "int8", seed=13) as fp:
        for name, ref in (("embed", orc.embed_table), ("lm_head", orc.lm_head), ("final_norm", orc.final_norm)):
            got, _, _ = fp.export_weight(-1, name)
            want = (np.ascontiguousarray(ref, np.float32).view(np.uint32) >> 16).astype(np.uint16)
            assert np.array_equal(got, want), name
        ids = np.concatenate([fpgen.token_ids(13, 40, s.vocab), [-1, s.vocab, 2**31 - 1, 0]]).astype(np.int32)
        t = torch.from_numpy(ids).cuda()
        x = torch.empty(len(ids) * s.hidden, dtype=torch.bfloat16, device="cuda")
        fp.embed(t, x)
        g = bf16_to_np(x).reshape(len(ids), s.hidden)
        assert np.array_equal(g[:40], orc.embed(ids[:40]))
        assert not g[40:43].any()                                  # out of range -> zeros
        assert np.array_equal(g[43], orc.embed_table[0])


@pytest.mark.parametrize("B,T", [(1, 1), (1, 5), (4, 1), (5, 3), (33, 2)])
def test_head_logits_and_argmax(B, T):
    import torch
    from paper_2501_13111_amd import Fingerprint
    s = Shape(1, 512, 4, 4, 128, 640, 40, 8, 16, vocab=2048 + 16)    # a ragged last logit block
    orc = OracleFingerprint(s, "bf16", "bf16", seed=14)
    y = bf16_round(np.random.default_rng(B * 10 + T).normal(0, 1.3, (B, T, s.hidden)).astype(np.float32))
    with Fingerprint(s, "int8", "bf16", seed=14) as fp:
        ids = torch.empty(B, dtype=torch.int32, device="cuda")
        lg = torch.empty(B * s.vocab, dtype=torch.float32, device="cuda")
        fp.head(np_to_bf16(y.reshape(-1)), B, T, ids, lg)
        torch.cuda.synchronize()
        gl = lg.cpu().numpy().reshape(B, s.vocab)
        gi = ids.cpu().numpy()
    ol, oi = orc.head(y[:, T - 1, :])
    err = rel_inf(gl, ol)
    log(f"head B={B} T={T}: logits err {err:.2e}, ids agree {np.mean(gi == oi):.3f}")
    assert err <= TOL
    _check_decisions(gl, gi, ol, f"B={B} T={T}")


CASES = [
    ("tiny-bf16", Shape(2, 256, 4, 4, 64, 688, 1, 32, 48, vocab=1024), "bf16", "bf16", 1, 32, 8),
    ("batch-int4-int8kv", Shape(2, 512, 8, 2, 64, 768, 3, 24, 32, vocab=2048), "int4", "int8", 3, 24, 6),
    ("7b-layer-vocab32000", Shape(1, 4096, 32, 32, 128, 11008, 2, 64, 70, vocab=LLAMA2_VOCAB),
     "bf16", "bf16", 2, 64, 4),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_generate_teacher_forced(case):
    import torch
    from paper_2501_13111_amd import Fingerprint
    name, s, wq, kvq, B, P, n = case
    log(f"generate {name}: B={B} P={P} n_out={n}")
    prompt = fpgen.token_ids(15, B * P, s.vocab).reshape(B, P)
    orc = OracleFingerprint(s, wq, kvq, seed=15)
    otoks, ologits = orc.generate(prompt, n)
    outs = {}
    for graph in (True, False):
        with Fingerprint(s, wq, kvq, seed=15) as fp:
            fp.set_decode_graph(graph)
            pid = torch.from_numpy(prompt.astype(np.int32)).cuda()
            force = torch.from_numpy(otoks[:-1].astype(np.int32).copy()).cuda()
            out = torch.empty((n + 1) * B, dtype=torch.int32, device="cuda")
            lg = torch.empty((n + 1) * B * s.vocab, dtype=torch.float32, device="cuda")
            for rep in range(2):                       # a second request on the same handle
                fp.generate(pid.view(B, P), n, out, lg, force_ids=force)
                torch.cuda.synchronize()
                outs[(graph, rep)] = (out.cpu().numpy().reshape(n + 1, B), lg.cpu().numpy().reshape(n + 1, B, -1))
            assert fp.position() == (P + n, B)
    gt, gl = outs[(True, 0)]
    for k, (t2, l2) in outs.items():                   # graph replay, eager and repeats agree bit for bit
        assert np.array_equal(t2, gt) and np.array_equal(l2.view(np.uint32), gl.view(np.uint32)), k
    errs = [rel_inf(gl[i], ologits[i]) for i in range(n + 1)]
    log(f"{name}: logits err per step {[f'{e:.2e}' for e in errs]}, token agreement {np.mean(gt == otoks):.3f}")
    assert max(errs) <= TOL
    for i in range(n + 1):
        _check_decisions(gl[i], gt[i], ologits[i], f"{name} step {i}")


def test_generate_free_running_tokens_are_valid_decisions():
    """Without teacher forcing the GPU feeds back its own tokens; each step's decision is
    checked against the oracle run on the GPU's own token history."""
    import torch
    from paper_2501_13111_amd import Fingerprint
    s = Shape(2, 512, 8, 2, 64, 768, 2, 16, 28, vocab=1024)
    B, P, n = 2, 16, 10
    prompt = fpgen.token_ids(16, B * P, s.vocab).reshape(B, P)
    with Fingerprint(s, "int8", "int8", seed=16) as fp:
        pid = torch.from_numpy(prompt.astype(np.int32)).cuda()
        out = torch.empty((n + 1) * B, dtype=torch.int32, device="cuda")
        lg = torch.empty((n + 1) * B * s.vocab, dtype=torch.float32, device="cuda")
        ms = fp.generate(pid.view(B, P), n, out, lg, timed=True)
        gt = out.cpu().numpy().reshape(n + 1, B)
        gl = lg.cpu().numpy().reshape(n + 1, B, -1)
    assert ms is not None and ms > 0
    orc = OracleFingerprint(s, "int8", "int8", seed=16)
    _, ologits = orc.generate(prompt, n, teacher=gt[:-1])
    for i in range(n + 1):
        assert rel_inf(gl[i], ologits[i]) <= TOL
        _check_decisions(gl[i], gt[i], ologits[i], f"step {i}")

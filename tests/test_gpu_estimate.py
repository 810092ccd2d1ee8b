"""The paper's fingerprint-based estimators on MI355X measurements (Sec. 5.2, Sec. 5.3).

L2: fingerprints of the Llama-2-7B shape (bf16, with embedding, final norm and LM head
over a 32000-token vocabulary) with 1 and 2 hidden layers, each timed on dummy requests
of two output lengths at batch 1; Eq. 1 per fingerprint, then Eq. 2 and Eq. 3, give the
per-layer and other-block TTFT and TPOT.  The library's solver must equal the oracle's on
the same measurements, and the predictions must hold for requests not used in the fit:
another output length, and 4 hidden layers.

M2: the device memory (hipMemGetInfo) a fingerprint holds with 1 and 2 hidden layers,
extrapolated linearly, must give the 4-layer fingerprint's footprint, and the observed
footprints must match the bytes the handle reports (weights W, KV cache and workspace A).
"""
import dataclasses
import statistics

import numpy as np
import pytest

import fpgen
from fpgen.workloads import Shape, LLAMA2_VOCAB
from oracle import estimate as E
from tests.gpu_harness import log

pytestmark = pytest.mark.gpu

SHAPE = Shape(1, 4096, 32, 32, 128, 11008, 1, 512, 612, vocab=LLAMA2_VOCAB)
P = 512
FIT_LAYERS, FIT_LEN = (1, 2), (16, 64)
HELD_OUT = [(1, 100), (2, 100), (4, 16), (4, 100)]
PRED_TOL = 0.10          # relative error of a held-out prediction


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2501_13111_amd as P_
    P_.load()
    yield


def _latencies(n_layers, lengths, reps=5):
    """Median request latency (ms) of a fingerprint with n_layers hidden layers at each length."""
    import torch
    from paper_2501_13111_amd import Fingerprint
    s = dataclasses.replace(SHAPE, n_layers=n_layers)
    pid = torch.from_numpy(fpgen.token_ids(0, P, s.vocab).reshape(1, P)).cuda()
    out = {}
    with Fingerprint(s, "bf16", "bf16", seed=0) as fp:
        bufs = {n: torch.empty(n + 1, dtype=torch.int32, device="cuda") for n in lengths}
        for n in lengths:                     # capture each length's decode graph once
            fp.generate(pid, n, bufs[n])
        torch.cuda.synchronize()
        for n in lengths:
            out[n] = statistics.median(fp.generate(pid, n, bufs[n], timed=True) for _ in range(reps))
    return out


def test_l2_latency_estimator_predicts_held_out_requests():
    from paper_2501_13111_amd import binding
    meas = {}
    for L in sorted({l for l, _ in HELD_OUT} | set(FIT_LAYERS)):
        lens = sorted({n for l, n in HELD_OUT if l == L} | (set(FIT_LEN) if L in FIT_LAYERS else set()))
        for n, ms in _latencies(L, lens).items():
            meas[(L, n)] = ms
            log(f"measured: {L} layer(s), output length {n}: {ms:.4f} ms")
    lat = [[meas[(L, n)] for n in FIT_LEN] for L in FIT_LAYERS]
    model = binding.fit_latency_l2(FIT_LAYERS, FIT_LEN, lat)
    ref = E.fit_l2(FIT_LAYERS, FIT_LEN, lat)
    for k in ref:
        assert abs(model[k] - ref[k]) <= 1e-9 * (1 + abs(ref[k])), k
    log("fit (ms): " + ", ".join(f"{k} {v:.4f}" for k, v in model.items()))
    for L, n in HELD_OUT:
        _, _, pred = binding.predict_latency(model, L, n)
        err = abs(pred - meas[(L, n)]) / meas[(L, n)]
        log(f"held out: {L} layer(s), length {n}: predicted {pred:.4f} ms, measured {meas[(L, n)]:.4f} ms, "
            f"error {100 * err:.2f}%")
        assert err <= PRED_TOL, (L, n, pred, meas[(L, n)])
    assert model["tpot_layer"] > 0 and model["ttft_layer"] > 0 and model["tpot_other"] > 0


def test_m2_memory_extrapolation_in_layers():
    import torch
    from paper_2501_13111_amd import Fingerprint, binding
    with Fingerprint(dataclasses.replace(SHAPE, n_layers=1, vocab=0), "bf16", "bf16"):
        pass                                  # loads every code object before measuring
    torch.cuda.synchronize()
    used, planned = {}, {}
    for L in (1, 2, 4):
        s = dataclasses.replace(SHAPE, n_layers=L)
        u0 = binding.device_memory()[0]
        fp = Fingerprint(s, "int4", "int8", seed=0)
        torch.cuda.synchronize()
        used[L] = binding.device_memory()[0] - u0
        planned[L] = sum(fp.memory_bytes())
        w, kv, ws = fp.memory_bytes()
        fp.close()
        torch.cuda.synchronize()
        log(f"M2: {L} layer(s): observed {used[L] / 2**20:.1f} MiB, held by the handle "
            f"{planned[L] / 2**20:.1f} MiB (W {w / 2**20:.1f}, KV {kv / 2**20:.1f}, workspace {ws / 2**20:.1f})")
        assert abs(used[L] - planned[L]) <= 0.02 * planned[L] + (64 << 20)
    ext = binding.extrapolate_layers((1, 2), (used[1], used[2]), 4)
    assert ext == pytest.approx(E.extrapolate_layers((1, 2), (used[1], used[2]), 4), rel=1e-12)
    err = abs(ext - used[4]) / used[4]
    log(f"M2: 4 layers extrapolated from 1 and 2: {ext / 2**20:.1f} MiB, observed {used[4] / 2**20:.1f} MiB, "
        f"error {100 * err:.2f}%")
    assert err <= 0.02

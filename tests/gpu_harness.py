"""Shared driver of the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them.

Decode parity is teacher-forced: at every step both sides consume the oracle's
previous output, so the comparison measures one step's error rather than the
feedback loop's amplification of ulp-level differences.  Free-running drift is
measured separately and reported only.
"""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import fpgen
from oracle.layer import Fingerprint as OracleFingerprint
from oracle.numerics import bf16_round

TOL = 2e-2          # max normwise relative error, ||g - r||_inf / ||r||_inf


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def rel_inf(g: np.ndarray, r: np.ndarray) -> float:
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))


def rel_2(g, r) -> float:
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))


def bf16_to_np(t) -> np.ndarray:
    """bf16 CUDA/CPU tensor -> float32 numpy (exact)."""
    import torch
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def np_to_bf16(a: np.ndarray, device="cuda"):
    import torch
    bits = (np.ascontiguousarray(bf16_round(a), np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)


@dataclasses.dataclass
class ParityResult:
    prefill_err: float              # end to end (all layers chained on each side)
    decode_errs: list
    prefill_err2: float = 0.0
    decode_errs2: list = dataclasses.field(default_factory=list)
    layer_errs: list = dataclasses.field(default_factory=list)   # prefill, layer-wise teacher-forced
    chained_ref: np.ndarray = None  # the oracle's chained prefill output of the compared rows


def run_parity(shape, wq, kvq, B, P, S, rows=None, seed=0, graph=True, acc=np.float64,
               oracle=None, fp=None, layerwise=False):
    """Prefill + S teacher-forced decode steps on the GPU and the oracle; compares
    sequences ``rows`` (all by default).  With ``layerwise`` the GPU also dumps every
    layer's prefill output and the oracle runs each layer on the GPU's own input of
    that layer (``layer_errs``); decode then continues from that oracle cache.
    Returns ParityResult."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal

    rows = list(range(B)) if rows is None else list(rows)
    H = shape.hidden
    own_fp = fp is None
    if own_fp:
        fp = Fingerprint(shape, wq, kvq, seed)
    fp.set_decode_graph(graph)
    x = torch.empty(B * P * H, dtype=torch.bfloat16, device="cuda")
    fill_normal(x, seed, -1, fpgen.T_INPUT, 0.0, 1.0)
    y = torch.empty_like(x)
    dump = None
    if layerwise:
        dump = torch.empty(shape.n_layers, B, P, H, dtype=torch.bfloat16, device="cuda")
        fp.set_debug_layer_dump(dump)
    fp.prefill(x, y, B, P)
    torch.cuda.synchronize()
    if layerwise:
        fp.set_debug_layer_dump(None)

    orc = oracle or OracleFingerprint(shape, wq, kvq, seed, acc=acc)
    xo = np.concatenate([fpgen.prompt(seed, B, P, H, b_start=r, b_count=1) for r in rows])
    yo = orc.prefill(xo)
    yg = bf16_to_np(y).reshape(B, P, H)
    res = ParityResult(rel_inf(yg[rows], yo), [], rel_2(yg[rows], yo), [])
    res.chained_ref = yo
    if layerwise:
        ridx = torch.tensor(rows, device="cuda")
        gl = [bf16_to_np(dump[l].index_select(0, ridx)).reshape(len(rows), P, H) for l in range(shape.n_layers)]
        del dump
        assert np.array_equal(gl[-1], yg[rows])
        ys = orc.prefill_layers([xo] + gl[:-1])
        res.layer_errs = [rel_inf(g, r) for g, r in zip(gl, ys)]
        yo = ys[-1]

    ins = [torch.empty(B, H, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    outs = [torch.empty(B, H, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    ins[0].copy_(y.view(B, P, H)[:, -1, :])
    ins[0][rows] = np_to_bf16(yo[:, -1, :])
    prev_o = yo[:, -1, :]
    for s in range(S):
        cur_in, out = ins[s % 2], outs[s % 2]
        fp.decode_step(cur_in, out)
        yo_s = orc.decode(prev_o)
        torch.cuda.synchronize()
        g = bf16_to_np(out).reshape(B, H)
        res.decode_errs.append(rel_inf(g[rows], yo_s))
        res.decode_errs2.append(rel_2(g[rows], yo_s))
        nxt = ins[(s + 1) % 2]
        nxt.copy_(out)
        nxt[rows] = np_to_bf16(yo_s)
        prev_o = yo_s
    if own_fp:
        fp.close()
    return res

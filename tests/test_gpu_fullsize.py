"""Parity at the workloads' full sizes, in the launch configuration the benchmark times
(the whole batch, prefill over the full prompt, every decode step replayed as a graph).

The oracle computes sampled sequences one by one (sequences are independent): the
first and / or last of the batch.  Teacher forcing as everywhere: each prefill layer
is compared given the GPU's own input of that layer, each decode step given the same
input on both sides, over all decode steps, so the last step reads a cache filled to
its maximum length.  Bars: bf16 outputs within 2e-2 normwise per compared tensor; the
chained prefill (every layer fed the previous layer's output on each side) within
max(2e-2, 1.5 x the drift of an fp32-accumulating oracle from the fp64 oracle on the
same sequence), since rounding differences of any fp32 implementation grow with depth
over these random weights; int8 KV codes within one code of the oracle's, at most 1e-3
of them differing, and bit-exact when the oracle quantises the GPU's own fp32 K / V;
weight codes, scales and zeros bit-exact on sampled rows of every matrix.

Each test logs a line starting with PARITY and a JSON record of its figures."""
import dataclasses
import json

import numpy as np
import pytest

import fpgen
from fpgen.workloads import CONFIGS
from oracle.layer import Fingerprint as OracleFingerprint, TENSOR_ID, weight_shapes
from oracle.quant import quant_kv_int8, quant_int8_channel, quant_int4_g128, pack_int4, prune_2of4
from tests.gpu_harness import TOL, log, run_parity, rel_inf

pytestmark = pytest.mark.gpu

# sampled sequences per workload: the oracle's cost grows with each one
FULL = [("llama2-7b-bf16", None), ("llama2-7b-int8", (0, 15)), ("llama2-13b-int4", (31,)),
        ("llama2-70b-tp8-int4", (0, 63)), ("llama2-7b-sp24", (0, 15))]
CHAIN_DRIFT_FACTOR = 1.5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2501_13111_amd as P
    P.load()
    yield


def _record(kind, name, **kw):
    log("PARITY " + json.dumps(dict(kind=kind, workload=name, **kw)))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,rows", FULL, ids=[f[0] for f in FULL])
def test_full_size_sampled_sequences(name, rows):
    from paper_2501_13111_amd import Fingerprint
    c = CONFIGS[name]
    s = c["shape"]
    assert c["P"] + c["S"] == s.max_seq
    rows = list(range(c["B"])) if rows is None else list(rows)
    log(f"full size {name}: B={c['B']} P={c['P']} S={c['S']} rows={rows}")
    orc = OracleFingerprint(s, c["wq"], c["kvq"], 0)
    fp = Fingerprint(s, c["wq"], c["kvq"], 0)
    res = run_parity(s, c["wq"], c["kvq"], c["B"], c["P"], c["S"], rows=rows, graph=True, layerwise=True,
                     oracle=orc, fp=fp)
    kv = None
    if c["kvq"] == "int8":
        # end-to-end codes: the oracle's layer l stored K / V from the GPU's own input of layer l
        kv = []
        for l in range(s.n_layers):
            k, v, _, _ = fp.export_kv(l)
            oc = orc.kv_codes[l]
            for mine, ref in ((k[rows], oc["k"]), (v[rows], oc["v"])):
                d = np.abs(mine[:, :, :c["P"]].astype(np.int32) - ref[:, :, :c["P"]].astype(np.int32))
                kv.append((int(d.max()), float((d > 0).mean())))
    fp.close()
    # the chained prefill against the fp32-accumulating oracle's own drift on the first row
    orc32 = OracleFingerprint(dataclasses.replace(s, max_batch=1), c["wq"], c["kvq"], 0, acc=np.float32)
    y32 = orc32.prefill(fpgen.prompt(0, c["B"], c["P"], s.hidden, b_start=rows[0], b_count=1))
    drift = rel_inf(y32, res.chained_ref[:1])
    bound = max(TOL, CHAIN_DRIFT_FACTOR * drift)
    worst = max(res.decode_errs)
    _record("fullsize", name, rows=rows, prefill_layer_err=[round(e, 5) for e in res.layer_errs],
            prefill_chained_err=round(res.prefill_err, 5), chained_bound=round(bound, 5),
            oracle_fp32_drift=round(drift, 5), decode_max_err=round(worst, 5),
            decode_last_err=round(res.decode_errs[-1], 5),
            kv_max_code_delta=None if kv is None else max(m for m, _ in kv),
            kv_mismatch_rate=None if kv is None else max(r for _, r in kv))
    assert len(res.decode_errs) == c["S"] and len(res.layer_errs) == s.n_layers
    assert max(res.layer_errs) <= TOL
    assert worst <= TOL
    assert res.prefill_err <= bound
    if kv is not None:
        assert max(m for m, _ in kv) <= 1 and max(r for _, r in kv) <= 1e-3


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama2-7b-int8", "llama2-70b-tp8-int4"])
def test_full_size_kv_codes_bit_exact_for_same_quantiser_input(name):
    """The oracle's int8 KV quantiser applied to the GPU's own fp32 K (after the rotary
    embedding) and V reproduces the cache's codes and scales bit for bit: the whole batch,
    every layer, the full prompt and one decode step."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    c = CONFIGS[name]
    s = c["shape"]
    B, P, nkv, d = c["B"], c["P"], s.n_kv_heads, s.head_dim
    per = 2 * B * P * nkv * d
    with Fingerprint(s, c["wq"], c["kvq"], 0) as fp:
        dump = torch.zeros(s.n_layers * per, dtype=torch.float32, device="cuda")
        fp.set_debug_kv_dump(dump)
        x = torch.empty(B * P * s.hidden, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 0, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, B, P)
        torch.cuda.synchronize()
        checked = 0
        for l in range(s.n_layers):
            k, v, ks, vs = fp.export_kv(l)
            blk = dump[l * per:(l + 1) * per].cpu().numpy().reshape(2, B, P, nkv, d)
            for which, codes, scales in ((0, k, ks), (1, v, vs)):
                oc, osc = quant_kv_int8(blk[which].transpose(0, 2, 1, 3))
                assert np.array_equal(codes[:, :, :P, :], oc), (l, which)
                assert np.array_equal(scales[:, :, :P].astype(np.float32), osc), (l, which)
                checked += oc.size
        a = y.view(B, P, s.hidden)[:, -1, :].contiguous()
        b = torch.empty_like(a)
        dump.zero_()
        fp.decode_step(a, b)
        torch.cuda.synchronize()
        dm = dump.cpu().numpy()
        for l in range(s.n_layers):
            k, v, ks, vs = fp.export_kv(l)
            blk = dm[l * 2 * B * nkv * d:(l + 1) * 2 * B * nkv * d].reshape(2, B, nkv, d)
            for which, codes, scales in ((0, k, ks), (1, v, vs)):
                oc, osc = quant_kv_int8(blk[which])
                assert np.array_equal(codes[:, :, P, :], oc), (l, which)
                assert np.array_equal(scales[:, :, P].astype(np.float32), osc), (l, which)
    _record("kv_same_input", name, codes_checked=checked, mismatches=0)


def _oracle_rows(wq, seed, layer, name, N, K, rows):
    """The oracle's codes (and scales / zeros) of the given rows of one weight matrix, each
    row synthesised from its own slice of the generator stream."""
    w = np.stack([fpgen.bits_to_f32(fpgen.bf16_bits(seed, layer, TENSOR_ID[name], K, 0.0, 0.02, start=r * K))
                  for r in rows])
    if wq == "bf16":
        return (w.view(np.uint32) >> 16).astype(np.uint16), None, None
    if wq == "sp24":
        d = np.where(prune_2of4(w), w, np.float32(0)).astype(np.float32)
        return (d.view(np.uint32) >> 16).astype(np.uint16), None, None
    if wq == "int8":
        c, sc = quant_int8_channel(w)
        return c, sc, None
    q, sc, z = quant_int4_g128(w)
    return pack_int4(q), sc, z


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", [n for n in CONFIGS if n != "tiny"])
def test_full_size_weight_codes_sampled_rows(name):
    """Codes, scales and zeros of every matrix of every layer, on the first, the last and 24
    random rows, and the norm gains, equal the oracle's bit for bit."""
    from paper_2501_13111_amd import Fingerprint
    c = CONFIGS[name]
    s = c["shape"]
    rng = np.random.default_rng(17)
    nrows = 0
    with Fingerprint(s, c["wq"], c["kvq"], 0) as fp:
        for l in range(s.n_layers):
            for gname in ("attn_norm", "mlp_norm"):
                g, _, _ = fp.export_weight(l, gname)
                want = fpgen.bf16_bits(0, l, TENSOR_ID[gname], s.hidden, 1.0, 0.02)
                assert np.array_equal(g, want), (l, gname)
            for wname, (N, K) in weight_shapes(s).items():
                codes, sc, z = fp.export_weight(l, wname)
                rows = sorted({0, N - 1, *rng.integers(0, N, 24).tolist()})
                oc, osc, oz = _oracle_rows(c["wq"], 0, l, wname, N, K, rows)
                assert np.array_equal(codes[rows], oc), (l, wname)
                if osc is not None:
                    assert np.array_equal(sc[rows].astype(np.float32), osc), (l, wname)
                if oz is not None:
                    assert np.array_equal(z[rows].astype(np.float32), oz), (l, wname)
                nrows += len(rows)
    _record("weight_codes", name, rows_checked=nrows, mismatches=0)

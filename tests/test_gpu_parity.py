"""Parity of the HIP path with the oracle at reduced sizes (several tiles, ragged
tails, every weight / KV format, grouped-query attention, multi-chunk decode
attention).  Bars: bit-exact weight codes and device-generated data; KV codes
bit-exact for identical quantiser inputs; bf16 activations within 2e-2
normwise (teacher-forced decode)."""
import json

import numpy as np
import pytest

import fpgen
from fpgen.workloads import Shape, CONFIGS
from oracle.layer import Fingerprint as OracleFingerprint
from oracle.quant import quant_kv_int8
from tests.gpu_harness import TOL, log, run_parity, bf16_to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2501_13111_amd as P
    P.load()
    yield


def test_fill_normal_matches_generator():
    import torch
    from paper_2501_13111_amd import fill_normal
    for (seed, layer, tensor, mean, sigma, n) in [(0, -1, 15, 0.0, 1.0, 100003), (0, 0, 1, 0.0, 0.02, 65536),
                                                   (5, 3, 0, 1.0, 0.02, 4096), (2**63 + 1, 1, 8, 0.0, 0.02, 777)]:
        t = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        fill_normal(t, seed, layer, tensor, mean, sigma)
        got = t.view(torch.int16).cpu().numpy().view(np.uint16)
        want = fpgen.bf16_bits(seed, layer, tensor, n, mean, sigma)
        log(f"fill_normal seed={seed} layer={layer} tensor={tensor}")
        assert np.array_equal(got, want)


WSHAPE = Shape(n_layers=2, hidden=256, n_heads=4, n_kv_heads=2, head_dim=64, ffn=384,
               max_batch=2, max_prompt=16, max_seq=24)


@pytest.mark.parametrize("wq", ["bf16", "int8", "int4", "sp24"])
def test_weight_codes_bit_exact(wq):
    from paper_2501_13111_amd import Fingerprint
    log(f"weight codes {wq}")
    orc = OracleFingerprint(WSHAPE, wq, "bf16", seed=11)
    with Fingerprint(WSHAPE, wq, "bf16", seed=11) as fp:
        for l in range(WSHAPE.n_layers):
            for name in ("attn_norm", "mlp_norm"):
                g, _, _ = fp.export_weight(l, name)
                want = orc.layers[l][name].astype(np.float32).view(np.uint32) >> 16
                assert np.array_equal(g, want.astype(np.uint16)), (l, name)
            for name in ("q", "k", "v", "o", "gate", "up", "down"):
                c, s, z = fp.export_weight(l, name)
                oc, os_, oz = orc.export_weight(l, name)
                if wq in ("bf16", "sp24"):
                    assert np.array_equal(c, (oc.view(np.uint32) >> 16).astype(np.uint16)), (l, name)
                elif wq == "int8":
                    assert np.array_equal(c, oc), (l, name)
                    assert np.array_equal(s.astype(np.float32), os_), (l, name)
                else:
                    assert np.array_equal(c, oc), (l, name)
                    assert np.array_equal(s.astype(np.float32), os_), (l, name)
                    assert np.array_equal(z.astype(np.float32), oz), (l, name)


def _report(name, res):
    log(f"{name}: prefill {res.prefill_err:.3e} (l2 {res.prefill_err2:.3e}) per layer "
        f"{[f'{e:.2e}' for e in res.layer_errs]} decode max "
        f"{max(res.decode_errs) if res.decode_errs else 0:.3e}")
    # one machine-readable record per case (tests/parity_table.py collects them)
    log("PARITY " + json.dumps(dict(kind="reduced", workload=name,
                                    prefill_layer_err=[round(e, 5) for e in res.layer_errs],
                                    prefill_chained_err=round(res.prefill_err, 5),
                                    decode_max_err=round(max(res.decode_errs), 5) if res.decode_errs else None,
                                    decode_steps=len(res.decode_errs))))


def test_tiny_config_end_to_end():
    c = CONFIGS["tiny"]
    res = run_parity(c["shape"], c["wq"], c["kvq"], c["B"], c["P"], c["S"])
    _report("tiny", res)
    assert res.prefill_err <= TOL
    assert max(res.decode_errs) <= TOL


CASES = [
    # (name, shape, wq, kvq, B, P, S)
    ("mha-bf16", Shape(2, 512, 4, 4, 128, 640, 3, 77, 84), "bf16", "bf16", 3, 77, 5),
    ("mha-int8", Shape(2, 512, 4, 4, 128, 640, 3, 77, 84), "int8", "int8", 3, 77, 5),
    ("mha-int4-bf16kv", Shape(2, 512, 4, 4, 128, 640, 3, 77, 84), "int4", "bf16", 3, 77, 5),
    ("mha-int4-int8kv", Shape(2, 512, 4, 4, 128, 640, 3, 77, 84), "int4", "int8", 3, 77, 5),
    ("mha-bf16-int8kv", Shape(1, 512, 4, 4, 128, 640, 2, 77, 84), "bf16", "int8", 2, 77, 4),
    ("gqa8-d64-int4-int8", Shape(2, 512, 8, 1, 64, 384, 5, 130, 134), "int4", "int8", 5, 130, 4),
    ("gqa8-d128-int4-int8", Shape(1, 1024, 8, 1, 128, 512, 4, 100, 104), "int4", "int8", 4, 100, 4),
    ("gqa2-d64-int8", Shape(1, 256, 4, 2, 64, 688, 2, 40, 46), "int8", "bf16", 2, 40, 6),
    ("batch40-int8", Shape(1, 256, 2, 2, 128, 384, 40, 20, 23), "int8", "int8", 40, 20, 3),
    ("batch64-int4", Shape(1, 256, 2, 2, 128, 384, 64, 9, 12), "int4", "bf16", 64, 9, 3),
    ("long-ctx-bf16", Shape(1, 256, 2, 2, 128, 384, 2, 520, 530), "bf16", "bf16", 2, 520, 3),
    # batches of 17 to 64 on two-block waves take 32x32x16 MFMA tiles: bf16 weights, and
    # int8 with a wide qkv (42 tiles of 256 rows) over a ragged 64-row activation tile
    ("batch24-bf16", Shape(1, 256, 2, 2, 128, 384, 24, 12, 15), "bf16", "bf16", 24, 12, 3),
    # one sequence takes the single-sequence projections: int4 (its scale | zero words ride
    # with the weight loads) under GQA 4:1 with an int8 cache, and at head_dim 64
    ("single-int4-gqa4-int8kv", Shape(2, 1024, 8, 2, 128, 1408, 1, 70, 76), "int4", "int8", 1, 70, 4),
    ("single-int4-d64", Shape(1, 512, 8, 8, 64, 768, 1, 33, 40), "int4", "bf16", 1, 33, 5),
    # decode that ends exactly at the cache capacity (P + S = max_seq)
    ("full-capacity-int8", Shape(1, 256, 2, 2, 128, 384, 3, 29, 32), "int8", "int8", 3, 29, 3),
    ("batch33-int8-wide", Shape(1, 3584, 28, 28, 128, 512, 33, 8, 11), "int8", "int8", 33, 8, 3),
    # prefill GEMMs with too few 256 x 256 tiles run split-K with reduction kernels
    # (M >= 256; M = 300 leaves a ragged row tile)
    ("splitk-bf16", Shape(2, 512, 4, 4, 128, 1024, 2, 160, 164), "bf16", "bf16", 2, 160, 2),
    ("splitk-int4-int8kv", Shape(2, 1024, 8, 8, 128, 2048, 2, 160, 164), "int4", "int8", 2, 160, 2),
    ("splitk-int8-gqa", Shape(2, 1024, 8, 4, 128, 2048, 1, 300, 302), "int8", "int8", 1, 300, 2),
    # 2:4 sparse weights on the sparse MFMA: one sequence (batch schedule), a ragged 128-row
    # weight tile (hidden 576) under GQA 3:1, 40 sequences (two 32-token tiles in decode,
    # ragged 128-token prefill tiles), and an int8 cache
    ("sp24-single-gqa3", Shape(2, 576, 9, 3, 64, 704, 1, 70, 76), "sp24", "bf16", 1, 70, 4),
    ("sp24-batch3", Shape(1, 1024, 8, 8, 128, 2048, 3, 130, 134), "sp24", "bf16", 3, 130, 3),
    ("sp24-batch40-int8kv", Shape(2, 512, 4, 4, 128, 1024, 40, 50, 54), "sp24", "int8", 40, 50, 3),
    # short prompts on a bf16 cache (the key-split prefill attention): a one-token prompt
    # (three of the four waves without a block), and GQA 4:1 at head_dim 64 over a ragged
    # 45-token prompt (two blocks)
    ("prompt1-bf16", Shape(1, 256, 2, 2, 128, 384, 2, 1, 4), "bf16", "bf16", 2, 1, 3),
    ("gqa4-d64-bf16-short", Shape(1, 512, 8, 2, 64, 768, 3, 45, 48), "int8", "bf16", 3, 45, 3),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_parity_reduced(case):
    name, shape, wq, kvq, B, P, S = case
    log(f"case {name}: {shape} {wq}/{kvq} B={B} P={P} S={S}")
    res = run_parity(shape, wq, kvq, B, P, S, layerwise=shape.n_layers > 1)
    _report(name, res)
    assert res.prefill_err <= TOL
    assert all(e <= TOL for e in res.layer_errs)
    assert max(res.decode_errs) <= TOL


def test_graph_replay_matches_eager():
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    shape = Shape(2, 256, 4, 2, 64, 384, 2, 40, 48)
    outs = {}
    for graph in (False, True):
        with Fingerprint(shape, "int8", "int8", seed=3) as fp:
            fp.set_decode_graph(graph)
            x = torch.empty(2 * 40 * 256, dtype=torch.bfloat16, device="cuda")
            fill_normal(x, 3, -1, 15, 0.0, 1.0)
            y = torch.empty_like(x)
            fp.prefill(x, y, 2, 40)
            a = y.view(2, 40, 256)[:, -1, :].contiguous()
            b = torch.empty_like(a)
            res = []
            for s in range(6):
                fp.decode_step(a, b)
                torch.cuda.synchronize()
                res.append(b.clone())
                a, b = b, a
            outs[graph] = torch.stack(res).cpu()
    assert torch.equal(outs[False].view(torch.int16), outs[True].view(torch.int16))


@pytest.mark.parametrize("B,wq,kvq", [(3, "int4", "int8"), (1, "bf16", "bf16"), (1, "int8", "int8")],
                         ids=["batch3-int4-int8kv", "single-bf16", "single-int8-int8kv"])
def test_decode_steps_match_single_steps(B, wq, kvq):
    """n steps in one call (one graph) give bit for bit what n calls of fp_decode_step
    give, with the decode graph on and off, for odd and even n, the batch schedule and the
    single-sequence one; the last call ends exactly at the cache's capacity.  The last
    output is in y for odd n and in x for even n."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    shape = Shape(2, 256, 4, 2, 64, 384, 3, 30, 44)
    P = 30
    steps = (1, 4, 3, 1, 5)                   # odd and even n, up to max_seq = 44
    assert P + sum(steps) == shape.max_seq

    def start(fp):
        x = torch.empty(B * P * 256, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 5, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, B, P)
        return y.view(B, P, 256)[:, -1, :].contiguous()

    ref = []
    with Fingerprint(shape, wq, kvq, seed=5) as fp:
        a = start(fp)
        b = torch.empty_like(a)
        for _ in range(sum(steps)):
            fp.decode_step(a, b)
            a, b = b, a
            ref.append(a.clone())
    for graph in (True, False):
        with Fingerprint(shape, wq, kvq, seed=5) as fp:
            fp.set_decode_graph(graph)
            x = start(fp)
            y = torch.empty_like(x)
            done = 0
            for n in steps:
                out = fp.decode_steps(x, y, n)
                done += n
                torch.cuda.synchronize()
                assert torch.equal(out.view(torch.int16), ref[done - 1].view(torch.int16)), (graph, n)
                if out is y:                  # continue from the last output
                    x, y = y, x
            assert fp.position() == (shape.max_seq, B)


def test_kv_codes_bit_exact_for_same_quantiser_input():
    """The oracle's int8 KV quantiser applied to the GPU's own fp32 K/V (debug dump)
    reproduces the GPU's codes and scales bit for bit, prefill and decode."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    shape = Shape(2, 512, 8, 2, 64, 384, 3, 50, 53)
    B, P = 3, 50
    nkv, d = shape.n_kv_heads, shape.head_dim
    with Fingerprint(shape, "int4", "int8", seed=2) as fp:
        dump = torch.zeros(shape.n_layers * 2 * B * P * nkv * d, dtype=torch.float32, device="cuda")
        fp.set_debug_kv_dump(dump)
        x = torch.empty(B * P * shape.hidden, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 2, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, B, P)
        torch.cuda.synchronize()
        dm = dump.cpu().numpy()
        for l in range(shape.n_layers):
            k, v, ks, vs = fp.export_kv(l)
            blk = dm[l * 2 * B * P * nkv * d:(l + 1) * 2 * B * P * nkv * d].reshape(2, B, P, nkv, d)
            for which, codes, scales in ((0, k, ks), (1, v, vs)):
                pre = blk[which].transpose(0, 2, 1, 3)            # [B, nkv, P, d]
                oc, osc = quant_kv_int8(pre)
                assert np.array_equal(codes[:, :, :P, :], oc), (l, which)
                assert np.array_equal(scales[:, :, :P].astype(np.float32), osc), (l, which)
        # one decode step
        a = y.view(B, P, shape.hidden)[:, -1, :].contiguous()
        b = torch.empty_like(a)
        dump.zero_()
        fp.decode_step(a, b)
        torch.cuda.synchronize()
        dm = dump.cpu().numpy()
        for l in range(shape.n_layers):
            k, v, ks, vs = fp.export_kv(l)
            blk = dm[l * 2 * B * nkv * d:(l + 1) * 2 * B * nkv * d].reshape(2, B, nkv, d)
            for which, codes, scales in ((0, k, ks), (1, v, vs)):
                oc, osc = quant_kv_int8(blk[which])
                assert np.array_equal(codes[:, :, P, :], oc), (l, which)
                assert np.array_equal(scales[:, :, P].astype(np.float32), osc), (l, which)


def test_kv_codes_end_to_end_within_one():
    """End-to-end int8 KV codes against the oracle's: |delta code| <= 1, mismatch rate reported
    and bounded (the quantiser inputs come out of GEMMs with different summation orders)."""
    from paper_2501_13111_amd import Fingerprint
    import torch
    from paper_2501_13111_amd import fill_normal
    shape = Shape(1, 512, 4, 4, 128, 640, 2, 64, 64)
    B, P = 2, 64
    orc = OracleFingerprint(shape, "int8", "int8", seed=4)
    orc.prefill(fpgen.prompt(4, B, P, shape.hidden))
    with Fingerprint(shape, "int8", "int8", seed=4) as fp:
        x = torch.empty(B * P * shape.hidden, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 4, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, B, P)
        k, v, ks, vs = fp.export_kv(0)
    oc = orc.kv_codes[0]
    for mine, ref in ((k, oc["k"]), (v, oc["v"])):
        dlt = np.abs(mine[:, :, :P].astype(np.int32) - ref[:, :, :P].astype(np.int32))
        rate = float((dlt > 0).mean())
        log(f"kv code mismatch rate {rate:.2e}, max |delta| {dlt.max()}")
        assert dlt.max() <= 1
        assert rate <= 1e-3


def test_reprefill_with_another_batch_drops_stale_graphs():
    """Decode graphs are captured per (x, y, batch).  Prefill B = 3, graph decode steps,
    then prefill B = 2 and B = 1 on the same handle and the same x / y buffers (sized for
    the largest batch, with sentinel rows past the active batch): every decode output
    equals a fresh handle's bit for bit, and the rows past the active batch are never
    written."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    shape = Shape(2, 256, 4, 2, 64, 384, 3, 20, 40)
    H, P, Bmax = 256, 20, 3
    sentinel = torch.full((Bmax * H,), 7.0, dtype=torch.bfloat16, device="cuda")

    def prompt(B):
        x = torch.empty(B * P * H, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 8, -1, 15, 0.0, 1.0)
        return x

    def fresh(B, steps):
        with Fingerprint(shape, "int8", "int8", seed=8) as fp:
            x = prompt(B)
            y = torch.empty_like(x)
            fp.prefill(x, y, B, P)
            a = y.view(B, P, H)[:, -1, :].contiguous()
            b = torch.empty_like(a)
            outs = []
            for _ in range(steps):
                fp.decode_step(a, b)
                outs.append(b.clone())
                a, b = b, a
            torch.cuda.synchronize()
            return outs

    with Fingerprint(shape, "int8", "int8", seed=8) as fp:
        xa = sentinel.clone()
        xb = sentinel.clone()
        stream = torch.cuda.current_stream().cuda_stream
        for B in (3, 2, 1, 2):
            log(f"re-prefill B={B}")
            x = prompt(B)
            y = torch.empty_like(x)
            fp.prefill(x, y, B, P)
            xa.copy_(sentinel)
            xb.copy_(sentinel)
            xa[:B * H].copy_(y.view(B, P, H)[:, -1, :].reshape(-1))
            got = []
            for st in range(3):
                src, dst = (xa, xb) if st % 2 == 0 else (xb, xa)
                fp.decode_ptr(src.data_ptr(), dst.data_ptr(), stream)
                got.append(dst[:B * H].clone())
            # steps 4 and 5 in one call: step 4 reads xb and writes xa, step 5 writes xb
            fp.decode_steps_ptr(xb.data_ptr(), xa.data_ptr(), 2, stream)
            got.append(xb[:B * H].clone())
            torch.cuda.synchronize()
            want = fresh(B, 5)
            for st, g in enumerate(got[:3]):
                assert torch.equal(g.view(torch.int16), want[st].view(-1).view(torch.int16)), (B, st)
            assert torch.equal(got[3].view(torch.int16), want[4].view(-1).view(torch.int16)), B
            for buf in (xa, xb):
                assert torch.equal(buf[B * H:].view(torch.int16), sentinel[B * H:].view(torch.int16)), B


@pytest.mark.parametrize("kvq", ["bf16", "int8"])
def test_single_sequence_decode_steps_match_single_steps(kvq):
    """One sequence (the single-sequence schedule the 7B bf16 workload runs): n steps in
    one call equal n calls of fp_decode_step bit for bit, graph on and off, with the last
    call ending exactly at the cache capacity."""
    import torch
    from paper_2501_13111_amd import Fingerprint, fill_normal
    shape = Shape(2, 512, 4, 4, 128, 640, 1, 33, 42)
    P = 33

    def start(fp):
        x = torch.empty(P * 512, dtype=torch.bfloat16, device="cuda")
        fill_normal(x, 9, -1, 15, 0.0, 1.0)
        y = torch.empty_like(x)
        fp.prefill(x, y, 1, P)
        return y.view(1, P, 512)[:, -1, :].contiguous()

    ref = []
    with Fingerprint(shape, "bf16", kvq, seed=9) as fp:
        fp.set_decode_graph(False)
        a = start(fp)
        b = torch.empty_like(a)
        for _ in range(9):
            fp.decode_step(a, b)
            a, b = b, a
            ref.append(a.clone())
    for graph in (True, False):
        with Fingerprint(shape, "bf16", kvq, seed=9) as fp:
            fp.set_decode_graph(graph)
            x = start(fp)
            y = torch.empty_like(x)
            done = 0
            for n in (3, 2, 4):               # 9 steps: the last call ends at max_seq = 42
                out = fp.decode_steps(x, y, n)
                done += n
                torch.cuda.synchronize()
                assert torch.equal(out.view(torch.int16), ref[done - 1].view(torch.int16)), (graph, n)
                if out is y:
                    x, y = y, x
            assert fp.position() == (42, 1)


# prompts long enough for the 256 x 256 prefill tiling (>= 128 tiles) with its fused
# residual and SwiGLU epilogues: ragged last row tile (M = 8000) and column tile (hidden
# 1152), and a [gate; up] tile count that is not a multiple of the wave layout
BIG_CASES = [
    ("big-int4-ragged", Shape(1, 1152, 9, 9, 128, 2176, 8, 1000, 1002), "int4", "int8", 8, 1000, 2, (0, 7)),
    ("big-bf16", Shape(1, 1024, 8, 8, 128, 2560, 8, 1024, 1026), "bf16", "bf16", 8, 1024, 2, (3,)),
    ("big-int8-gqa", Shape(1, 1024, 8, 2, 128, 2048, 8, 1024, 1026), "int8", "int8", 8, 1024, 2, (5,)),
    # hidden and ffn not whole 64-input stages: tile counts of the large tiling, but the
    # projections that reduce over them take the small tiling (o, over n_heads * head_dim =
    # 1024, stays large)
    ("big-bf16-partial-stage", Shape(1, 1040, 8, 8, 128, 2080, 4, 1024, 1026), "bf16", "bf16", 4, 1024, 2, (2,)),
    # 2:4 weights on the large sparse tiling, with a ragged last column tile
    ("big-sp24-ragged", Shape(1, 1024, 8, 4, 128, 2112, 8, 1000, 1002), "sp24", "int8", 8, 1000, 2, (0, 7)),
]


@pytest.mark.parametrize("case", BIG_CASES, ids=[c[0] for c in BIG_CASES])
def test_parity_large_prefill_tiles(case):
    name, shape, wq, kvq, B, P, S, rows = case
    log(f"case {name}: {shape} {wq}/{kvq} B={B} P={P} S={S} rows={rows}")
    res = run_parity(shape, wq, kvq, B, P, S, rows=rows)
    _report(name, res)
    assert res.prefill_err <= TOL
    assert max(res.decode_errs) <= TOL


# Small grids with a bf16 cache take the short-prompt kernel (online softmax, no second
# pass; the limit does not apply there), so the bf16 repeat path is exercised by a grid of
# 256 workgroups (big-bf16-partial-stage, sampled rows); the int8 cases take the regular
# kernel at any size.
REPEAT_CASES = [c + (None,) for c in CASES if c[0] in ("mha-bf16", "gqa8-d128-int4-int8", "long-ctx-bf16",
                                                       "sp24-batch3")] + \
               [c for c in BIG_CASES if c[0] == "big-bf16-partial-stage"]


@pytest.mark.parametrize("case", REPEAT_CASES, ids=[c[0] for c in REPEAT_CASES])
def test_prefill_attention_repeat_path(case, monkeypatch):
    """The prefill attention's second pass (a probability against the first block's
    maximum passing the limit) forced from the host with a limit of 2: most workgroups of
    the regular kernel repeat their prompt with a larger reference, and the result still
    meets the bar."""
    name, shape, wq, kvq, B, P, S, rows = case
    monkeypatch.setenv("FP_ATTN_PROB_LIMIT_LOG2", "1")
    log(f"case {name} (probability limit 2): {shape} {wq}/{kvq} B={B} P={P} S={S} rows={rows}")
    if rows is not None:
        res = run_parity(shape, wq, kvq, B, P, S, rows=rows)
        _report(name + "-repeat", res)
        assert res.prefill_err <= TOL
        assert max(res.decode_errs) <= TOL
        return
    res = run_parity(shape, wq, kvq, B, P, S, layerwise=shape.n_layers > 1)
    _report(name + "-repeat", res)
    assert res.prefill_err <= TOL
    assert all(e <= TOL for e in res.layer_errs)
    assert max(res.decode_errs) <= TOL

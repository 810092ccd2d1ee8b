"""Host-side tests of the C ABI: the library loads, exports every declared symbol,
and validates arguments and state on the host (no GPU needed)."""
import ctypes

import pytest

from paper_2501_13111_amd import binding
from paper_2501_13111_amd.binding import Fingerprint, FpError, FpShape
from fpgen.workloads import Shape, CONFIGS


@pytest.fixture(scope="module")
def lib():
    return binding.load()


def test_every_declared_symbol_is_exported(lib):
    names = binding.header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code, name in binding.STATUS.items():
        assert lib.fp_status_str(code).decode() == name


def _create_status(shape, wq=0, kvq=0, unbacked=True):
    L = binding.load()
    s = FpShape.from_obj(shape)
    h = ctypes.c_void_p()
    fn = L.fp_layer_create_unbacked if unbacked else L.fp_layer_create
    rc = fn(ctypes.byref(s), wq, kvq, 0, ctypes.byref(h))
    if rc == 0:
        L.fp_layer_destroy(h)
    return rc


@pytest.mark.parametrize("kw,wq,code", [
    (dict(n_heads=6), 0, -1),                 # 6 heads not a multiple of 4 kv heads
    (dict(hidden=260), 0, -1),                # hidden not a multiple of 16
    (dict(hidden=320), 2, -1),                # int4 needs multiples of 128
    (dict(head_dim=96, hidden=384), 0, -6),   # head_dim 96 unsupported
    (dict(max_batch=65), 0, -6),
    (dict(max_prompt=64, max_seq=48), 0, -1),
    (dict(rms_eps=0.0), 0, -1),
    (dict(n_layers=0), 0, -1),
    (dict(hidden=288, n_heads=4, head_dim=64), 3, -1),   # 2:4 sparse: hidden 288 not a multiple of 64
    (dict(ffn=416), 3, -1),                              # nor ffn 416
])
def test_shape_validation(kw, wq, code):
    base = dict(n_layers=1, hidden=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn=384,
                max_batch=2, max_prompt=32, max_seq=48)
    base.update(kw)
    shape = Shape(**base)
    assert _create_status(shape, wq=wq, unbacked=True) == code
    # the real create performs the same checks before touching the device
    assert _create_status(shape, wq=wq, unbacked=False) == code


def test_bad_enums_and_null(lib):
    s = FpShape.from_obj(CONFIGS["tiny"]["shape"])
    h = ctypes.c_void_p()
    assert lib.fp_layer_create_unbacked(ctypes.byref(s), 7, 0, 0, ctypes.byref(h)) == -1
    assert lib.fp_layer_create_unbacked(ctypes.byref(s), 0, 5, 0, ctypes.byref(h)) == -1
    assert lib.fp_layer_create_unbacked(None, 0, 0, 0, ctypes.byref(h)) == -1
    assert lib.fp_layer_create_unbacked(ctypes.byref(s), 0, 0, 0, None) == -1
    assert lib.fp_prefill(None, 16, 1, 1, 32, None) == -1
    assert lib.fp_layer_destroy(None) == 0


def test_no_device_reports_hip_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert _create_status(CONFIGS["tiny"]["shape"], unbacked=False) == -5


def test_state_machine_on_unbacked_handle():
    c = CONFIGS["tiny"]
    s = c["shape"]        # max_batch 1, max_prompt 32, max_seq 48
    fp = Fingerprint(s, "bf16", "bf16", unbacked=True)
    X, Y = 1 << 20, 1 << 30          # fake, non-overlapping addresses: nothing is launched
    with pytest.raises(FpError) as e:
        fp.decode_ptr(X, Y)
    assert e.value.code == -2        # decode before prefill
    with pytest.raises(FpError) as e:
        fp.decode_steps_ptr(X, Y, 2)
    assert e.value.code == -2
    with pytest.raises(FpError) as e:
        fp.prefill_ptr(X, Y, 2, 8)
    assert e.value.code == -3        # batch beyond capacity
    with pytest.raises(FpError) as e:
        fp.prefill_ptr(X, Y, 1, 33)
    assert e.value.code == -3        # prompt beyond capacity
    with pytest.raises(FpError) as e:
        fp.prefill_ptr(X, X + 100, 1, 8)
    assert e.value.code == -1        # x and y overlap
    with pytest.raises(FpError) as e:
        fp.prefill_ptr(X, Y, 0, 8)
    assert e.value.code == -1
    assert fp.position() == (0, 0)
    fp.prefill_ptr(X, Y, 1, 32)
    assert fp.position() == (32, 1)
    for i in range(16):
        fp.decode_ptr(X, Y)
    assert fp.position() == (48, 1)
    with pytest.raises(FpError) as e:
        fp.decode_ptr(X, Y)
    assert e.value.code == -3        # cache full at max_seq
    assert fp.position() == (48, 1)  # nothing changed on error
    fp.prefill_ptr(X, Y, 1, 4)       # a new prefill resets the position
    assert fp.position() == (4, 1)
    # n steps at once: all or nothing against the capacity
    with pytest.raises(FpError) as e:
        fp.decode_steps_ptr(X, Y, 0)
    assert e.value.code == -1        # n < 1
    with pytest.raises(FpError) as e:
        fp.decode_steps_ptr(X, X + 100, 3)
    assert e.value.code == -1        # x and y overlap
    with pytest.raises(FpError) as e:
        fp.decode_steps_ptr(X, Y, 45)
    assert e.value.code == -3        # 4 + 45 > 48
    assert fp.position() == (4, 1)
    fp.decode_steps_ptr(X, Y, 44)
    assert fp.position() == (48, 1)
    with pytest.raises(FpError) as e:
        fp.export_kv(0)
    assert e.value.code == -2
    fp.close()


def test_last_error_message_is_set():
    L = binding.load()
    s = FpShape.from_obj(Shape(1, 260, 4, 4, 64, 384, 1, 8, 8))
    h = ctypes.c_void_p()
    assert L.fp_layer_create_unbacked(ctypes.byref(s), 0, 0, 0, ctypes.byref(h)) == -1
    assert b"multiples of 16" in L.fp_last_error()


def _planned_bytes(shape, wq, kvq):
    fp = Fingerprint(shape, wq, kvq, unbacked=True)
    try:
        return fp.memory_bytes()
    finally:
        fp.close()


def _hand_weight_bytes(s, wq):
    """Fused matrices [q;k;v], o, [gate;up], down stored fragment-major: 1 KiB per 16 rows
    and one k-step of 32 bf16 / 64 int8 / 128 int4 inputs (k padded to whole steps);
    int8 adds an fp16 scale per row; int4 an fp16 scale, an fp16 zero and a packed u32
    scale|zero word per (row, group of 128).  Plus two bf16 gains of hidden."""
    ks = {"bf16": 32, "int8": 64, "int4": 128, "sp24": 32}[wq]
    qd, kd = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
    mats = [(qd + 2 * kd, s.hidden), (s.hidden, qd), (2 * s.ffn, s.hidden), (s.hidden, s.ffn)]
    per_layer = 2 * s.hidden * 2
    for N, K in mats:
        if wq == "sp24":          # 32 x 32 blocks: 1 KiB of kept values + 128 B of index words
            per_layer += (N // 32) * (K // 32) * (1024 + 128)
            continue
        per_layer += (N // 16) * (-(-K // ks)) * 1024
        if wq == "int8":
            per_layer += N * 2
        elif wq == "int4":
            per_layer += N * (K // 128) * (2 + 2 + 4)
    return s.n_layers * per_layer


def _hand_kv_bytes(s, kvq):
    """Keys [B, nkv, R, d] and values in 32-position blocks [B, nkv, R/32, d, 32] with
    R = max_seq rounded up to 32; int8 adds fp16 key and value scales [B, nkv, R]."""
    R = -(-s.max_seq // 32) * 32
    esz = 1 if kvq == "int8" else 2
    per_layer = 2 * s.max_batch * s.n_kv_heads * R * s.head_dim * esz
    if kvq == "int8":
        per_layer += 2 * s.max_batch * s.n_kv_heads * R * 2
    return s.n_layers * per_layer


@pytest.mark.parametrize("name", ["tiny", "llama2-7b-bf16", "llama2-7b-int8", "llama2-13b-int4",
                                  "llama2-70b-tp8-int4", "llama2-7b-sp24"])
def test_memory_bytes_match_the_storage_layout(name):
    c = CONFIGS[name]
    s = c["shape"]
    w, kv, ws = _planned_bytes(s, c["wq"], c["kvq"])
    assert w == _hand_weight_bytes(s, c["wq"])
    assert kv == _hand_kv_bytes(s, c["kvq"])
    # workspace: at least the prefill activations (x, h, normalised input: 3 x [B*P, hidden]
    # bf16) and the fp32 q|k|v of the prompt
    M = s.max_batch * s.max_prompt
    qkv = s.n_heads * s.head_dim + 2 * s.n_kv_heads * s.head_dim
    assert ws >= 3 * M * s.hidden * 2 + M * qkv * 4


def test_memory_bytes_scale_with_weight_format_and_layers():
    """Sec. 3.2: INT8 weights halve and INT4 weights quarter the memory of 16-bit weights
    (plus their scales: 2 bytes per row for int8, 8 bytes per 128 inputs for int4), and
    the footprint grows linearly with the number of hidden layers (Sec. 5, Fig. 7)."""
    import dataclasses
    s = CONFIGS["llama2-7b-bf16"]["shape"]
    wb = _planned_bytes(s, "bf16", "bf16")[0]
    w8 = _planned_bytes(s, "int8", "bf16")[0]
    w4 = _planned_bytes(s, "int4", "bf16")[0]
    gains = s.n_layers * 2 * s.hidden * 2
    assert abs((w8 - gains) / (wb - gains) - 0.5) < 1e-3
    assert abs((w4 - gains) / (wb - gains) - (0.25 + 8 / 256)) < 1e-3
    # 2:4 sparsity (Sec. 3.3): half the bf16 values plus 2 bits per kept value
    ws = _planned_bytes(s, "sp24", "bf16")[0]
    assert abs((ws - gains) / (wb - gains) - 9 / 16) < 1e-9
    one = [_planned_bytes(dataclasses.replace(s, n_layers=n), "int4", "int8") for n in (1, 2, 3)]
    for i in range(2):       # weights and KV are linear; the workspace does not grow with layers
        assert one[2][i] - one[1][i] == one[1][i] - one[0][i]
    assert one[0][2] == one[1][2] == one[2][2]


@pytest.mark.parametrize("vocab,code", [(8, -1), (-16, -1), (32000, 0), (0, 0)])
def test_vocab_validation(vocab, code):
    import dataclasses
    s = dataclasses.replace(CONFIGS["tiny"]["shape"], vocab=vocab)
    assert _create_status(s, unbacked=True) == code


def test_head_calls_on_unbacked_handles():
    import dataclasses
    X, Y = 1 << 20, 1 << 30
    L = binding.load()
    plain = Fingerprint(CONFIGS["tiny"]["shape"], "bf16", "bf16", unbacked=True)
    assert L.fp_embed(plain._h, X, 4, Y, None) == -2            # no embedding (vocab = 0)
    assert L.fp_head(plain._h, X, 1, 1, None, Y, None) == -2
    assert L.fp_generate(plain._h, X, 1, 4, 2, Y, None, None, None, None) == -2
    plain.close()
    s = dataclasses.replace(CONFIGS["tiny"]["shape"], vocab=512)   # max_batch 1, prompt 32, seq 48
    fp = Fingerprint(s, "int8", "int8", unbacked=True)
    assert L.fp_embed(fp._h, X, 0, Y, None) == -1
    assert L.fp_embed(fp._h, None, 4, Y, None) == -1
    assert L.fp_embed(fp._h, X, 4, Y, None) == 0
    assert L.fp_head(fp._h, X, 2, 1, None, Y, None) == -3       # beyond max_batch
    assert L.fp_head(fp._h, X, 1, 0, None, Y, None) == -1
    assert L.fp_head(fp._h, X, 1, 5, None, None, None) == -1
    assert L.fp_generate(fp._h, X, 1, 33, 2, Y, None, None, None, None) == -3    # prompt
    assert L.fp_generate(fp._h, X, 1, 32, 17, Y, None, None, None, None) == -3   # 32 + 17 > 48
    assert L.fp_generate(fp._h, X, 1, 32, -1, Y, None, None, None, None) == -1
    assert L.fp_generate(fp._h, X, 1, 32, 16, Y, None, None, None, None) == 0
    assert fp.position() == (48, 1)
    fp.close()


def test_memory_bytes_with_the_other_blocks():
    """Embedding [vocab, hidden] and LM head [vocab, hidden] in bf16 plus the final gain,
    under every weight format."""
    import dataclasses
    for wq in ("bf16", "int4"):
        s0 = CONFIGS["llama2-7b-bf16"]["shape"]
        s1 = dataclasses.replace(s0, vocab=32000)
        w0 = _planned_bytes(s0, wq, "bf16")[0]
        w1 = _planned_bytes(s1, wq, "bf16")[0]
        assert w1 - w0 == 2 * 32000 * 4096 * 2 + 4096 * 2


def test_estimators_agree_with_the_oracle():
    import numpy as np
    from oracle import estimate as E
    rng = np.random.default_rng(5)
    for _ in range(20):
        layers = tuple(int(v) for v in rng.choice([1, 2, 3, 4, 8], size=2, replace=False))
        n_out = tuple(int(v) for v in rng.choice([8, 16, 50, 64, 100, 128], size=2, replace=False))
        lat = rng.uniform(5, 500, size=(2, 2)).tolist()
        got = binding.fit_latency_l2(layers, n_out, lat)
        want = E.fit_l2(layers, n_out, lat)
        for k in want:
            assert abs(got[k] - want[k]) <= 1e-9 * (1 + abs(want[k])), k
        n, o = int(rng.integers(1, 100)), int(rng.integers(0, 500))
        assert np.allclose(binding.predict_latency(got, n, o), E.predict(want, n, o), rtol=1e-10)
        t, p = binding.fit_ttft_tpot(n_out, lat[0])
        assert np.allclose((t, p), E.fit_ttft_tpot(n_out, lat[0]), rtol=1e-10, atol=1e-10)
        vals = rng.uniform(1e8, 1e10, size=2).tolist()
        m = int(rng.integers(1, 100))
        assert np.isclose(binding.extrapolate_layers(layers, vals, m), E.extrapolate_layers(layers, vals, m),
                          rtol=1e-12)
    with pytest.raises(FpError) as e:
        binding.fit_ttft_tpot((32, 32), (1.0, 2.0))
    assert e.value.code == -1
    with pytest.raises(FpError):
        binding.fit_latency_l2((2, 2), (16, 64), [[1.0, 2.0], [1.0, 2.0]])
    with pytest.raises(FpError):
        binding.extrapolate_layers((3, 3), (1.0, 2.0), 5)

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

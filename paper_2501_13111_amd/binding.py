"""ctypes binding of the C ABI in include/fp.h -- argument marshalling only.

Every step of the fingerprint forward pass runs in the HIP library
(``libfp_mi355x.so``); this module checks tensor arguments, passes their
device addresses and the current stream, and turns status codes into
exceptions.  It raises if the library has not been built: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfp_mi355x.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "fp.h")

WQ = {"bf16": 0, "int8": 1, "int4": 2, "sp24": 3}
KVQ = {"bf16": 0, "int8": 1}
TENSOR = {"attn_norm": 0, "q": 1, "k": 2, "v": 3, "o": 4, "mlp_norm": 5, "gate": 6, "up": 7,
          "down": 8, "input": 15, "embed": 16, "final_norm": 17, "lm_head": 18}
STATUS = {0: "FP_OK", -1: "FP_ERR_INVALID_ARG", -2: "FP_ERR_STATE", -3: "FP_ERR_CAPACITY",
          -4: "FP_ERR_OOM", -5: "FP_ERR_HIP", -6: "FP_ERR_UNSUPPORTED"}


class FpError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        self.code = code
        self.status = STATUS.get(code, str(code))
        super().__init__(f"{where}: {self.status}: {msg}")


class FpShape(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("max_prompt", ctypes.c_int32),
                ("max_seq", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float), ("vocab", ctypes.c_int32)]

    @classmethod
    def from_obj(cls, s):
        """Build from any object with the shape's attribute names (e.g. a dataclass); a
        missing vocab means 0 (hidden layers only)."""
        return cls(*(getattr(s, f, 0) for f, _ in cls._fields_))


class LatencyModel(ctypes.Structure):
    """fp_latency_model: the four unknowns of Eq. 2 and Eq. 3."""
    _fields_ = [("ttft_layer", ctypes.c_double), ("tpot_layer", ctypes.c_double),
                ("ttft_other", ctypes.c_double), ("tpot_other", ctypes.c_double)]


_lib = None


def lib_path() -> str:
    return LIB_PATH


def load(path: str | None = None):
    """Load the built HIP library (raises if it is missing).  The environment variable
    FP_MI355X_LIB selects another build of the same library (e.g. a tuning variant)."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or os.environ.get("FP_MI355X_LIB") or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"HIP library not built: {p} is missing (run __graft_entry__.build())")
    L = ctypes.CDLL(p)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "fp_layer_create": [ctypes.POINTER(FpShape), i32, i32, u64, ctypes.POINTER(vp)],
        "fp_layer_create_unbacked": [ctypes.POINTER(FpShape), i32, i32, u64, ctypes.POINTER(vp)],
        "fp_layer_destroy": [vp],
        "fp_prefill": [vp, vp, i32, i32, vp, vp],
        "fp_decode_step": [vp, vp, vp, vp],
        "fp_decode_steps": [vp, vp, vp, i32, vp],
        "fp_decode_step_noalloc": [vp, vp, vp, vp],
        "fp_set_decode_graph": [vp, i32],
        "fp_fill_normal": [vp, i64, u64, i32, i32, ctypes.c_float, ctypes.c_float, vp],
        "fp_export_weight": [vp, i32, i32, vp, vp, vp],
        "fp_export_kv": [vp, i32, vp, vp, vp, vp],
        "fp_set_debug_kv_dump": [vp, vp],
        "fp_set_debug_layer_dump": [vp, vp],
        "fp_memory_bytes": [vp, ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t),
                            ctypes.POINTER(ctypes.c_size_t)],
        "fp_get_position": [vp, ctypes.POINTER(i32), ctypes.POINTER(i32)],
        "fp_embed": [vp, vp, i64, vp, vp],
        "fp_head": [vp, vp, i32, i32, vp, vp, vp],
        "fp_generate": [vp, vp, i32, i32, i32, vp, vp, vp, ctypes.POINTER(ctypes.c_float), vp],
        "fp_fit_ttft_tpot": [ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double),
                             ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)],
        "fp_fit_latency_l2": [ctypes.POINTER(i32), ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(LatencyModel)],
        "fp_predict_latency": [ctypes.POINTER(LatencyModel), i32, i32, ctypes.POINTER(ctypes.c_double),
                               ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)],
        "fp_extrapolate_layers": [ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double), i32,
                                  ctypes.POINTER(ctypes.c_double)],
        "fp_device_memory": [ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.fp_status_str.argtypes = [ctypes.c_int]
    L.fp_status_str.restype = ctypes.c_char_p
    L.fp_last_error.argtypes = []
    L.fp_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def header_functions() -> list[str]:
    """Names of the functions include/fp.h declares."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(fp_\w+)\s*\(", text, re.M)))


def _check(code: int, where: str):
    if code != 0:
        msg = load().fp_last_error().decode(errors="replace")
        raise FpError(code, where, msg)


def _stream(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _dev_ptr(t, dtype_bits: int = 16, numel: int | None = None, name: str = "tensor") -> int:
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.element_size() * 8 != dtype_bits:
        raise ValueError(f"{name} must have {dtype_bits}-bit elements")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return t.data_ptr()


def _i32s(*v):
    return (ctypes.c_int32 * len(v))(*[int(x) for x in v])


def _f64s(*v):
    return (ctypes.c_double * len(v))(*[float(x) for x in v])


def fit_ttft_tpot(n_out, latency):
    """Eq. 1 at two output lengths -> (TTFT, TPOT)."""
    t, p = ctypes.c_double(), ctypes.c_double()
    _check(load().fp_fit_ttft_tpot(_i32s(*n_out), _f64s(*latency), ctypes.byref(t), ctypes.byref(p)),
           "fp_fit_ttft_tpot")
    return t.value, p.value


def fit_latency_l2(layers, n_out, latency):
    """L2 (Eq. 1-3): latency[i][j] of the fingerprint with layers[i] layers at length n_out[j]
    -> dict(ttft_layer, tpot_layer, ttft_other, tpot_other)."""
    m = LatencyModel()
    flat = [latency[0][0], latency[0][1], latency[1][0], latency[1][1]]
    _check(load().fp_fit_latency_l2(_i32s(*layers), _i32s(*n_out), _f64s(*flat), ctypes.byref(m)),
           "fp_fit_latency_l2")
    return {f: getattr(m, f) for f, _ in LatencyModel._fields_}


def predict_latency(model, n_layers, n_out):
    """(TTFT, TPOT, latency) of n_layers hidden layers at output length n_out."""
    m = LatencyModel(**model)
    t, p, l = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(load().fp_predict_latency(ctypes.byref(m), int(n_layers), int(n_out), ctypes.byref(t),
                                     ctypes.byref(p), ctypes.byref(l)), "fp_predict_latency")
    return t.value, p.value, l.value


def extrapolate_layers(layers, values, n_layers):
    """M2's linear extrapolation in the layer count."""
    v = ctypes.c_double()
    _check(load().fp_extrapolate_layers(_i32s(*layers), _f64s(*values), int(n_layers), ctypes.byref(v)),
           "fp_extrapolate_layers")
    return v.value


def device_memory():
    """(used, total) bytes of the current device (hipMemGetInfo)."""
    u, t = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().fp_device_memory(ctypes.byref(u), ctypes.byref(t)), "fp_device_memory")
    return u.value, t.value


def fill_normal(t, seed: int, layer: int, tensor: int, mean: float, sigma: float, stream=None):
    """Device synthetic data: t (bf16 / int16 CUDA tensor) <- bf16(mean + sigma*z)."""
    L = load()
    _check(L.fp_fill_normal(_dev_ptr(t, name="t"), t.numel(), seed & ((1 << 64) - 1), layer,
                            tensor, mean, sigma, _stream(stream)), "fp_fill_normal")


class Fingerprint:
    """One fingerprint on the current device (weights, KV cache, workspace)."""

    def __init__(self, shape, wq: str = "bf16", kvq: str = "bf16", seed: int = 0,
                 unbacked: bool = False):
        L = load()
        self.shape = shape
        self.wq, self.kvq, self.seed = wq, kvq, seed
        self._s = FpShape.from_obj(shape)
        h = ctypes.c_void_p()
        fn = L.fp_layer_create_unbacked if unbacked else L.fp_layer_create
        _check(fn(ctypes.byref(self._s), WQ[wq], KVQ[kvq], seed & ((1 << 64) - 1), ctypes.byref(h)),
               "fp_layer_create")
        self._h = h
        self.B = 0

    # lifetime ------------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            load().fp_layer_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    # forward -------------------------------------------------------------
    def prefill(self, x, y, B: int, P: int, stream=None):
        H = self.shape.hidden
        xp = _dev_ptr(x, numel=B * P * H, name="x")
        yp = _dev_ptr(y, numel=B * P * H, name="y")
        _check(load().fp_prefill(self._h, xp, B, P, yp, _stream(stream)), "fp_prefill")
        self.B = B

    def decode_step(self, x, y, stream=None):
        H = self.shape.hidden
        xp = _dev_ptr(x, numel=self.B * H, name="x")
        yp = _dev_ptr(y, numel=self.B * H, name="y")
        _check(load().fp_decode_step(self._h, xp, yp, _stream(stream)), "fp_decode_step")

    def decode_step_noalloc(self, x, y, stream=None):
        """fp_decode_step_noalloc: one eager decode step whose scratch lives in the library's
        static per-GPU region (no allocation of any kind)."""
        H = self.shape.hidden
        xp = _dev_ptr(x, numel=self.B * H, name="x")
        yp = _dev_ptr(y, numel=self.B * H, name="y")
        _check(load().fp_decode_step_noalloc(self._h, xp, yp, _stream(stream)), "fp_decode_step_noalloc")

    def decode_steps(self, x, y, n: int, stream=None):
        """n decode steps alternating between x and y (step 1 writes y); returns the
        buffer holding the last step's output (y for odd n, x for even n)."""
        H = self.shape.hidden
        xp = _dev_ptr(x, numel=self.B * H, name="x")
        yp = _dev_ptr(y, numel=self.B * H, name="y")
        _check(load().fp_decode_steps(self._h, xp, yp, int(n), _stream(stream)), "fp_decode_steps")
        return y if n % 2 == 1 else x

    def decode_steps_ptr(self, x_ptr: int, y_ptr: int, n: int, stream_ptr: int = 0):
        _check(load().fp_decode_steps(self._h, x_ptr, y_ptr, int(n), stream_ptr), "fp_decode_steps")

    def prefill_ptr(self, x_ptr: int, y_ptr: int, B: int, P: int, stream_ptr: int = 0):
        """Raw-pointer form (host-side tests with unbacked handles)."""
        _check(load().fp_prefill(self._h, x_ptr, B, P, y_ptr, stream_ptr), "fp_prefill")
        self.B = B

    def decode_ptr(self, x_ptr: int, y_ptr: int, stream_ptr: int = 0):
        _check(load().fp_decode_step(self._h, x_ptr, y_ptr, stream_ptr), "fp_decode_step")

    # blocks outside the hidden layers (vocab > 0) ------------------------
    def embed(self, ids, x, stream=None):
        """x [M, hidden] bf16 <- embedding rows of ids (int32 CUDA tensor [M])."""
        M = ids.numel()
        ip = _dev_ptr(ids, dtype_bits=32, name="ids")
        xp = _dev_ptr(x, numel=M * self.shape.hidden, name="x")
        _check(load().fp_embed(self._h, ip, M, xp, _stream(stream)), "fp_embed")

    def head(self, y, B: int, T: int, next_ids, logits=None, stream=None):
        """Final norm + LM head + greedy argmax of position T-1 of y [B, T, hidden]."""
        yp = _dev_ptr(y, numel=B * T * self.shape.hidden, name="y")
        ip = _dev_ptr(next_ids, dtype_bits=32, numel=B, name="next_ids")
        lp = None if logits is None else _dev_ptr(logits, dtype_bits=32, numel=B * self.shape.vocab,
                                                  name="logits")
        _check(load().fp_head(self._h, yp, B, T, lp, ip, _stream(stream)), "fp_head")

    def generate(self, prompt_ids, n_out: int, out_ids, logits=None, force_ids=None, timed=False,
                 stream=None):
        """One dummy request: prompt_ids int32 [B, P] -> out_ids int32 [n_out + 1, B] (and the
        logits [n_out + 1, B, vocab] when given).  Returns the device time in ms when timed."""
        B, P = prompt_ids.shape
        pp = _dev_ptr(prompt_ids, dtype_bits=32, name="prompt_ids")
        op = _dev_ptr(out_ids, dtype_bits=32, numel=(n_out + 1) * B, name="out_ids")
        lp = None if logits is None else _dev_ptr(logits, dtype_bits=32,
                                                  numel=(n_out + 1) * B * self.shape.vocab, name="logits")
        fp_ = None if force_ids is None else _dev_ptr(force_ids, dtype_bits=32, numel=n_out * B,
                                                      name="force_ids")
        ms = ctypes.c_float(-1.0)
        _check(load().fp_generate(self._h, pp, B, P, int(n_out), op, lp, fp_,
                                  ctypes.byref(ms) if timed else None, _stream(stream)), "fp_generate")
        self.B = B
        return ms.value if timed else None

    def set_decode_graph(self, enable: bool):
        _check(load().fp_set_decode_graph(self._h, 1 if enable else 0), "fp_set_decode_graph")

    def set_debug_kv_dump(self, buf=None):
        p = None if buf is None else _dev_ptr(buf, dtype_bits=32, name="dump")
        _check(load().fp_set_debug_kv_dump(self._h, p), "fp_set_debug_kv_dump")

    def set_debug_layer_dump(self, buf=None):
        p = None if buf is None else _dev_ptr(buf, dtype_bits=16, name="dump")
        _check(load().fp_set_debug_layer_dump(self._h, p), "fp_set_debug_layer_dump")

    # inspection ----------------------------------------------------------
    def position(self):
        pos, b = ctypes.c_int32(), ctypes.c_int32()
        _check(load().fp_get_position(self._h, ctypes.byref(pos), ctypes.byref(b)), "fp_get_position")
        return pos.value, b.value

    def memory_bytes(self):
        w, kv, ws = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        _check(load().fp_memory_bytes(self._h, ctypes.byref(w), ctypes.byref(kv), ctypes.byref(ws)),
               "fp_memory_bytes")
        return w.value, kv.value, ws.value

    def weight_shape(self, name: str):
        s = self.shape
        qd, kd = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
        return {"q": (qd, s.hidden), "k": (kd, s.hidden), "v": (kd, s.hidden), "o": (s.hidden, qd),
                "gate": (s.ffn, s.hidden), "up": (s.ffn, s.hidden), "down": (s.hidden, s.ffn)}[name]

    def export_weight(self, layer: int, name: str):
        """(codes, scales, zeros) as numpy arrays in the canonical layouts of fp.h (layer -1
        for the embedding, final norm and LM head)."""
        L = load()
        if name in ("embed", "lm_head"):
            c = np.empty((self.shape.vocab, self.shape.hidden), np.uint16)
            _check(L.fp_export_weight(self._h, -1, TENSOR[name], c.ctypes.data, None, None),
                   "fp_export_weight")
            return c, None, None
        if name in ("attn_norm", "mlp_norm", "final_norm"):
            g = np.empty(self.shape.hidden, np.uint16)
            _check(L.fp_export_weight(self._h, layer, TENSOR[name], g.ctypes.data, None, None),
                   "fp_export_weight")
            return g, None, None
        N, K = self.weight_shape(name)
        if self.wq in ("bf16", "sp24"):
            c = np.empty((N, K), np.uint16)
            _check(L.fp_export_weight(self._h, layer, TENSOR[name], c.ctypes.data, None, None),
                   "fp_export_weight")
            return c, None, None
        if self.wq == "int8":
            c = np.empty((N, K), np.int8)
            sc = np.empty(N, np.float16)
            _check(L.fp_export_weight(self._h, layer, TENSOR[name], c.ctypes.data, sc.ctypes.data, None),
                   "fp_export_weight")
            return c, sc, None
        c = np.empty((N, K // 8), np.int32)
        sc = np.empty((N, K // 128), np.float16)
        z = np.empty((N, K // 128), np.float16)
        _check(L.fp_export_weight(self._h, layer, TENSOR[name], c.ctypes.data, sc.ctypes.data,
                                  z.ctypes.data), "fp_export_weight")
        return c, sc, z

    def export_kv(self, layer: int):
        """(k, v, k_scales, v_scales) of the active batch: [B, nkv, max_seq, d] (+ scales)."""
        s = self.shape
        shp = (self.B, s.n_kv_heads, s.max_seq, s.head_dim)
        if self.kvq == "int8":
            k, v = np.empty(shp, np.int8), np.empty(shp, np.int8)
            ks, vs = np.empty(shp[:3], np.float16), np.empty(shp[:3], np.float16)
            _check(load().fp_export_kv(self._h, layer, k.ctypes.data, v.ctypes.data, ks.ctypes.data,
                                       vs.ctypes.data), "fp_export_kv")
            return k, v, ks, vs
        k, v = np.empty(shp, np.uint16), np.empty(shp, np.uint16)
        _check(load().fp_export_kv(self._h, layer, k.ctypes.data, v.ctypes.data, None, None),
               "fp_export_kv")
        return k, v, None, None

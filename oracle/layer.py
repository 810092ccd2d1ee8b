"""The fingerprint's decoder layer, prefill and KV-cached decode -- test infrastructure only.

Paper passages followed:
* a fingerprint keeps the LLM's components -- embedding, hidden layers,
  normalisation layer, activation -- with one or two hidden layers
  (Sec. 1, Sec. 5.1, Fig. 2);
* latency = TTFT + output_length x TPOT (Eq. 1): prefill produces the first
  token, then each output token is one decode step that reuses the KV cache,
  so per-token cost stays constant (Sec. 5.3);
* INT8 / INT4 weight-only quantisation and an INT8 KV cache are searched
  (Sec. 3.2, Table A.1), and so is pruning (Sec. 3.3, Table A.1), here the 2:4
  semi-structured form with magnitude scores ("sp24": every projection keeps 2 of
  every 4 consecutive weights of a row, bf16).

The paper writes none of the layer's math.  The reading (Llama-2 style, the
LLMs it profiles) is, per layer, with x bf16 [T, H]:
    xn = bf16(rmsnorm(x) * g_attn)
    q, k, v = xn W_q^T, xn W_k^T, xn W_v^T                (fp32/fp64, not rounded)
    q, k = rope(q, pos), rope(k, pos)
    K/V cache <- k, v  (bf16, or int8 per head and position)
    o = bf16(attention(q, K_cache, V_cache))              (causal, GQA h -> h*nkv/nh)
    h = bf16(x + o W_o^T)
    hn = bf16(rmsnorm(h) * g_mlp)
    a = bf16(silu(hn W_gate^T) * (hn W_up^T))
    y = bf16(h + a W_down^T)
Attention always reads K/V back from the cache (so KV-cached decode equals
full recompute).  Decode feeds the last layer's output at the last position
back as the next input.

With shape.vocab > 0 the fingerprint also keeps the blocks outside the hidden
layers (Sec. 5.1, Fig. 2: embedding, normalisation layer, LM head), and a
dummy request (Sec. 5.3) runs on token ids:
    x = E[ids]                                            (embedding gather)
    y = layers(x)                                         (prefill or decode step)
    logits = bf16(rmsnorm(y_last) * g_final) W_lm^T       (fp64 here)
    next id = argmax(logits), the lowest id among equal maxima (greedy)
The embedding, final gain and LM head stay 16-bit (bf16) under every weight
format: the weight-only quantisation applies to the hidden layers' projections.
A request with output length n runs the prefill (which yields the first token)
and n decode steps, each consuming the previous token.

Pins (tests/test_oracle_layer.py): RMSNorm against torch's rms_norm and the
closed form for constant rows; RoPE against complex multiplication and its
identity / norm / relative-position properties; attention against brute-force
loops and torch's scaled_dot_product_attention; SiLU against torch; the layer
against the identity special case, causality, batch independence and
KV-cached decode == full recompute; the whole two-layer stack against the same
layer composed from torch library routines (F.linear, F.rms_norm, complex
rotation, scaled_dot_product_attention, F.silu) for every weight format with a
bf16 and with an int8 cache; and the int8 cache's codes and scales against an
independent torch rebuild (keys quantised after the rotary embedding, both keys
and values from their fp32 values).
"""
from __future__ import annotations

import numpy as np

import fpgen
from .numerics import bf16_round
from .quant import (quant_int8_channel, dequant_int8_channel, quant_int4_g128,
                    dequant_int4_g128, pack_int4, quant_kv_int8, prune_2of4)

# The layer-stack shape and the five workloads live in the data-only table shared
# with the benchmark.
from fpgen.workloads import Shape, CONFIGS  # noqa: F401

F32 = np.float32

WEIGHT_NAMES = ("q", "k", "v", "o", "gate", "up", "down")
TENSOR_ID = {"attn_norm": 0, "q": 1, "k": 2, "v": 3, "o": 4, "mlp_norm": 5,
             "gate": 6, "up": 7, "down": 8}


def weight_shapes(s: Shape):
    """[N, K] (out x in) of each projection."""
    return {"q": (s.q_dim, s.hidden), "k": (s.kv_dim, s.hidden), "v": (s.kv_dim, s.hidden),
            "o": (s.hidden, s.q_dim), "gate": (s.ffn, s.hidden), "up": (s.ffn, s.hidden),
            "down": (s.hidden, s.ffn)}


# ------------------------------------------------------------------ components
def rmsnorm(x, g, eps, acc=np.float64):
    """y = x * (1 / sqrt(mean(x^2) + eps)) * g over the last axis, in ``acc``."""
    xa = np.asarray(x, dtype=acc)
    ms = np.mean(xa * xa, axis=-1, keepdims=True)
    r = acc(1.0) / np.sqrt(ms + acc(eps))
    return (xa * r) * np.asarray(g, dtype=acc)


def silu(z):
    """silu(z) = z / (1 + exp(-z))."""
    with np.errstate(over="ignore"):
        return z / (1 + np.exp(-z))


def rope_tables(max_seq: int, head_dim: int, theta: float):
    """cos / sin tables [max_seq, head_dim/2]: angle(p, i) = p * theta^(-2i/d),
    evaluated in float64 and rounded once to float32."""
    half = head_dim // 2
    inv = np.power(np.float64(theta), -2.0 * np.arange(half, dtype=np.float64) / head_dim)
    ang = np.arange(max_seq, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(F32), np.sin(ang).astype(F32)


def apply_rope(u, cos, sin, acc=np.float64):
    """Rotate-half rotary embedding of u [..., T, nh, d] with tables cos/sin [T, d/2].

    Element i pairs with i + d/2:  u'_i = u_i c - u_{i+d/2} s,
    u'_{i+d/2} = u_{i+d/2} c + u_i s  (each product and sum rounded in ``acc``)."""
    u = np.asarray(u, dtype=acc)
    half = u.shape[-1] // 2
    a, b = u[..., :half], u[..., half:]
    c = np.asarray(cos, dtype=acc)[:, None, :]
    s = np.asarray(sin, dtype=acc)[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention(q, K, V, q_pos, n_kv_heads, acc=np.float64):
    """Causal multi-head / grouped-query attention of one sequence.

    q [T, nh, d] at absolute positions q_pos [T]; K, V [nkv, S, d] hold the
    cached (stored) keys and values of positions 0..S-1.  Query head h reads kv
    head floor(h * nkv / nh) over positions j <= q_pos.  Scores are
    (q . k) * float32(1/sqrt(d)); softmax subtracts the row max over the
    allowed positions.  Returns o [T, nh, d] in ``acc``."""
    T, nh, d = q.shape
    S = K.shape[1]
    scale = acc(F32(1.0 / np.sqrt(d)))
    allowed = np.arange(S)[None, :] <= np.asarray(q_pos)[:, None]          # [T, S]
    out = np.empty((T, nh, d), dtype=acc)
    for h in range(nh):
        kvh = (h * n_kv_heads) // nh
        sc = (np.asarray(q[:, h, :], dtype=acc) @ np.asarray(K[kvh], dtype=acc).T) * scale
        sc = np.where(allowed, sc, -np.inf)
        m = sc.max(axis=-1, keepdims=True)
        p = np.exp(sc - m)                                                  # excluded -> 0
        out[:, h, :] = (p @ np.asarray(V[kvh], dtype=acc)) / p.sum(axis=-1, keepdims=True)
    return out


# ------------------------------------------------------------------ the model
class Fingerprint:
    """Fingerprint forward pass: ``prefill`` then one ``decode`` call per token.

    ``batch_rows`` selects which sequences of the full batch this instance runs
    (sequences are independent, so any subset gives the same per-row results as
    the whole batch); prompts come from ``fpgen.prompt`` with the same row
    numbering.  ``acc`` is the arithmetic type (float64 by default)."""

    def __init__(self, shape: Shape, wq: str = "bf16", kvq: str = "bf16", seed: int = 0,
                 acc=np.float64, weights=None):
        assert wq in ("bf16", "int8", "int4", "sp24") and kvq in ("bf16", "int8")
        self.s, self.wq, self.kvq, self.seed, self.acc = shape, wq, kvq, seed, acc
        s = shape
        assert s.n_heads % s.n_kv_heads == 0 and s.head_dim % 2 == 0
        self.cos, self.sin = rope_tables(s.max_seq, s.head_dim, s.rope_theta)
        self.layers = [self._make_layer(l, weights) for l in range(s.n_layers)]
        self.pos = None
        if s.vocab > 0:
            self.embed_table = fpgen.weight(seed, -1, fpgen.T_EMBED, (s.vocab, s.hidden))
            self.final_norm = fpgen.gain(seed, -1, fpgen.T_FINAL_NORM, s.hidden)
            self.lm_head = fpgen.weight(seed, -1, fpgen.T_LM_HEAD, (s.vocab, s.hidden))

    # weights -------------------------------------------------------------
    def _make_layer(self, l, weights):
        s = self.s
        L = {"attn_norm": fpgen.gain(self.seed, l, TENSOR_ID["attn_norm"], s.hidden),
             "mlp_norm": fpgen.gain(self.seed, l, TENSOR_ID["mlp_norm"], s.hidden)}
        quant = {}
        for name, shp in weight_shapes(s).items():
            if weights is not None and (l, name) in weights:
                w = np.asarray(weights[(l, name)], dtype=F32)
            else:
                w = fpgen.weight(self.seed, l, TENSOR_ID[name], shp)
            if self.wq == "bf16":
                deq = w
                quant[name] = (w, None, None)
            elif self.wq == "sp24":
                deq = np.where(prune_2of4(w), w, F32(0.0)).astype(F32)
                quant[name] = (deq, None, None)
            elif self.wq == "int8":
                c, sc = quant_int8_channel(w)
                deq = dequant_int8_channel(c, sc)
                quant[name] = (c, sc, None)
            else:
                q, sc, z = quant_int4_g128(w)
                deq = dequant_int4_g128(q, sc, z)
                quant[name] = (pack_int4(q), sc, z)
            L[name] = deq.astype(self.acc)
        L["quant"] = quant
        return L

    def export_weight(self, layer: int, name: str):
        """(codes, scales, zeros) in the canonical layouts: bf16 weights as float32
        values; int8 codes [N, K] with scales [N]; int4 packed words [N, K/8] int32
        with scales / zeros [N, K/128]; 2:4 sparse weights dense, pruned ones zero."""
        return self.layers[layer]["quant"][name]

    # cache ---------------------------------------------------------------
    def _reset_cache(self, B):
        s = self.s
        shp = (B, s.n_kv_heads, s.max_seq, s.head_dim)
        self.K = [np.zeros(shp, self.acc) for _ in range(s.n_layers)]
        self.V = [np.zeros(shp, self.acc) for _ in range(s.n_layers)]
        self.kv_codes = None
        if self.kvq == "int8":
            self.kv_codes = [dict(k=np.zeros(shp, np.int8), v=np.zeros(shp, np.int8),
                                  ks=np.zeros(shp[:3], F32), vs=np.zeros(shp[:3], F32))
                             for _ in range(s.n_layers)]
        self.pre_quant = [dict(k=None, v=None) for _ in range(s.n_layers)]

    def _store(self, l, k, v, pos):
        """Write k, v [B, T, nkv, d] at positions ``pos`` into layer l's cache."""
        kt = np.transpose(k, (0, 2, 1, 3))       # [B, nkv, T, d]
        vt = np.transpose(v, (0, 2, 1, 3))
        if self.kvq == "bf16":
            self.K[l][:, :, pos, :] = bf16_round(kt)
            self.V[l][:, :, pos, :] = bf16_round(vt)
        else:
            k32, v32 = kt.astype(F32), vt.astype(F32)     # the quantiser sees fp32 values
            kc, ks = quant_kv_int8(k32)
            vc, vs = quant_kv_int8(v32)
            cc = self.kv_codes[l]
            cc["k"][:, :, pos, :], cc["ks"][:, :, pos] = kc, ks
            cc["v"][:, :, pos, :], cc["vs"][:, :, pos] = vc, vs
            self.K[l][:, :, pos, :] = kc.astype(F32) * ks[..., None]
            self.V[l][:, :, pos, :] = vc.astype(F32) * vs[..., None]
            self.pre_quant[l] = dict(k=k32, v=v32)

    # forward -------------------------------------------------------------
    def _layer(self, l, x, pos):
        """x [B, T, H] bf16-valued; pos [T] absolute positions. Returns y [B, T, H]."""
        s, A, W = self.s, self.acc, self.layers[l]
        B, T, H = x.shape
        xn = bf16_round(rmsnorm(x, W["attn_norm"], s.rms_eps, A)).astype(A)
        q = (xn @ W["q"].T).reshape(B, T, s.n_heads, s.head_dim)
        k = (xn @ W["k"].T).reshape(B, T, s.n_kv_heads, s.head_dim)
        v = (xn @ W["v"].T).reshape(B, T, s.n_kv_heads, s.head_dim)
        if A is F32:
            q, k, v = q.astype(F32), k.astype(F32), v.astype(F32)
        c, sn = self.cos[pos], self.sin[pos]
        q = apply_rope(q, c, sn, A)
        k = apply_rope(k, c, sn, A)
        self._store(l, k, v, pos)
        end = int(pos[-1]) + 1
        o = np.empty((B, T, s.n_heads, s.head_dim), A)
        for b in range(B):
            o[b] = attention(q[b], self.K[l][b, :, :end], self.V[l][b, :, :end], pos,
                             s.n_kv_heads, A)
        ob = bf16_round(o.reshape(B, T, s.q_dim)).astype(A)
        h = bf16_round(x.astype(A) + ob @ W["o"].T).astype(A)
        hn = bf16_round(rmsnorm(h, W["mlp_norm"], s.rms_eps, A)).astype(A)
        g = hn @ W["gate"].T
        u = hn @ W["up"].T
        a = bf16_round(silu(g) * u).astype(A)
        y = bf16_round(h + a @ W["down"].T)
        return y

    def prefill(self, x):
        """x [B, P, H] bf16-valued prompt hidden states -> y [B, P, H] (float32)."""
        x = np.asarray(x, dtype=F32)
        B, P, H = x.shape
        assert H == self.s.hidden and P <= self.s.max_seq
        self._reset_cache(B)
        pos = np.arange(P)
        for l in range(self.s.n_layers):
            x = self._layer(l, x, pos)
        self.pos = P
        return x

    def prefill_layers(self, xs):
        """Layer-by-layer teacher forcing of a prefill: layer l runs on xs[l] (a given
        input [B, P, H] of that layer, e.g. another implementation's own) instead of on
        layer l-1's output here.  Returns the per-layer outputs; the cache afterwards
        holds what each layer stored from its given input."""
        xs = [np.asarray(x, dtype=F32) for x in xs]
        assert len(xs) == self.s.n_layers
        B, P, H = xs[0].shape
        assert H == self.s.hidden and P <= self.s.max_seq
        self._reset_cache(B)
        pos = np.arange(P)
        ys = [self._layer(l, xs[l], pos) for l in range(self.s.n_layers)]
        self.pos = P
        return ys

    def decode(self, x):
        """One decode step: x [B, H] (the previous output fed back) -> y [B, H]."""
        assert self.pos is not None and self.pos < self.s.max_seq
        x = np.asarray(x, dtype=F32)[:, None, :]
        pos = np.array([self.pos])
        for l in range(self.s.n_layers):
            x = self._layer(l, x, pos)
        self.pos += 1
        return x[:, 0, :]

    def run(self, x_prompt, steps, teacher=None):
        """Prefill then ``steps`` decode steps.  Free-running feeds each output back;
        with ``teacher`` (list of [B, H] inputs) step s takes teacher[s] instead.
        Returns (y_prefill, [y_step ...])."""
        y0 = self.prefill(x_prompt)
        xin = y0[:, -1, :]
        ys = []
        for st in range(steps):
            if teacher is not None:
                xin = teacher[st]
            y = self.decode(xin)
            ys.append(y)
            xin = y
        return y0, ys

    # ------------------------------------------------------------ other blocks
    def embed(self, ids):
        """Embedding gather: ids (int) [...] -> rows of the table [..., H] (bf16 values)."""
        ids = np.asarray(ids)
        assert self.s.vocab > 0 and ids.min() >= 0 and ids.max() < self.s.vocab
        return self.embed_table[ids]

    def head(self, y):
        """Final RMSNorm and LM head of the last hidden states y [B, H]: returns
        (logits [B, vocab] in the arithmetic type, next ids [B] by greedy argmax)."""
        A = self.acc
        yn = bf16_round(rmsnorm(y, self.final_norm, self.s.rms_eps, A)).astype(A)
        logits = yn @ self.lm_head.astype(A).T
        return logits, argmax_first(logits)

    def generate(self, ids, n_out, teacher=None):
        """One dummy request on token ids [B, P]: the prefill yields token 0, then n_out
        decode steps each consume the previous token (or teacher[i - 1] when given) and
        yield tokens 1..n_out.  Returns (tokens [n_out + 1, B], logits [n_out + 1, B, V])."""
        ids = np.asarray(ids)
        y = self.prefill(self.embed(ids))
        lg, tok = self.head(y[:, -1, :])
        toks, logits = [tok], [lg]
        for i in range(n_out):
            inp = tok if teacher is None else np.asarray(teacher[i])
            lg, tok = self.head(self.decode(self.embed(inp)))
            toks.append(tok)
            logits.append(lg)
        return np.stack(toks), np.stack(logits)


def argmax_first(logits):
    """Index of the largest value along the last axis; the lowest index among equal maxima."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.int32)

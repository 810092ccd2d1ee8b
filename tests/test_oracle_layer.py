"""Pins of the oracle's layer components and of the layer / decode loop as a whole."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fnn

import fpgen
from oracle.layer import (Shape, Fingerprint, rope_tables, apply_rope, rmsnorm, silu,
                          attention, weight_shapes, CONFIGS)
from oracle.numerics import bf16_round


# ------------------------------------------------------------------ components
def test_rmsnorm_matches_torch_and_closed_form():
    rng = np.random.default_rng(0)
    x = rng.normal(0, 2, (5, 96))
    g = rng.normal(1, 0.1, 96)
    ours = rmsnorm(x, g, 1e-5)
    ref = Fnn.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(ours, ref, rtol=1e-13, atol=0)
    for c in (0.0, 1e-3, 0.5, -3.0):
        y = rmsnorm(np.full((1, 64), c), g[:64], 1e-5)
        assert np.allclose(y, c / math.sqrt(c * c + 1e-5) * g[:64], rtol=1e-14, atol=0)


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 2001)
    assert np.allclose(silu(z), Fnn.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-300)
    assert silu(np.float64(0.0)) == 0.0


def test_rope_tables_match_complex_exponential():
    cos, sin = rope_tables(64, 16, 1e4)
    p = np.arange(64)[:, None]
    i = np.arange(8)[None, :]
    e = np.exp(1j * p * (1e4 ** (-(2.0 * i) / 16)))
    assert np.array_equal(cos, e.real.astype(np.float32)) or np.allclose(cos, e.real, atol=6e-8)
    assert np.allclose(sin, e.imag, atol=6e-8)
    assert np.all(cos[0] == 1) and np.all(sin[0] == 0)
    assert np.allclose(cos[:, 0], np.cos(np.arange(64)), atol=6e-8)       # inv freq of i=0 is 1


def test_rope_equals_complex_rotation_and_is_relative():
    rng = np.random.default_rng(1)
    d = 32
    cos, sin = rope_tables(40, d, 1e4)
    u = rng.normal(size=(40, 3, d))
    pos = np.arange(40)
    r = apply_rope(u, cos[pos], sin[pos])
    z = (u[..., :d // 2] + 1j * u[..., d // 2:]) * (cos[pos] + 1j * sin[pos].astype(np.float64))[:, None, :]
    assert np.allclose(r[..., :d // 2], z.real, rtol=0, atol=1e-12)
    assert np.allclose(r[..., d // 2:], z.imag, rtol=0, atol=1e-12)
    # position 0 is the identity; every (i, i+d/2) pair keeps its norm
    assert np.array_equal(r[0], u[0])
    n0 = u[..., :d // 2] ** 2 + u[..., d // 2:] ** 2
    n1 = r[..., :d // 2] ** 2 + r[..., d // 2:] ** 2
    assert np.allclose(n0, n1, rtol=1e-6)
    # q(m) . k(n) depends only on m - n
    q, k = rng.normal(size=d), rng.normal(size=d)

    def dot(m, n):
        a = apply_rope(q[None, None, :], cos[[m]], sin[[m]])[0, 0]
        b = apply_rope(k[None, None, :], cos[[n]], sin[[n]])[0, 0]
        return a @ b
    for m, n in [(5, 2), (20, 17), (39, 36)]:
        assert abs(dot(m, n) - dot(3, 0)) < 1e-5


def _attention_loops(q, K, V, q_pos, nkv):
    T, nh, d = q.shape
    out = np.zeros((T, nh, d))
    scale = float(np.float32(1.0 / math.sqrt(d)))
    for t in range(T):
        for h in range(nh):
            kv = h * nkv // nh
            js = range(int(q_pos[t]) + 1)
            sc = [sum(q[t, h, e] * K[kv, j, e] for e in range(d)) * scale for j in js]
            m = max(sc)
            w = [math.exp(s - m) for s in sc]
            tot = sum(w)
            for e in range(d):
                out[t, h, e] = sum(w[j] * V[kv, j, e] for j in js) / tot
    return out


@pytest.mark.parametrize("nh,nkv", [(2, 2), (4, 1), (4, 2)])
def test_attention_brute_force_and_sdpa(nh, nkv):
    rng = np.random.default_rng(nh * 10 + nkv)
    T, d = 6, 8
    q = rng.normal(size=(T, nh, d))
    K = rng.normal(size=(nkv, T, d))
    V = rng.normal(size=(nkv, T, d))
    pos = np.arange(T)
    ours = attention(q, K, V, pos, nkv)
    assert np.allclose(ours, _attention_loops(q, K, V, pos, nkv), rtol=1e-12, atol=1e-13)
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(K).repeat_interleave(nh // nkv, dim=0)[None]
    vt = torch.from_numpy(V).repeat_interleave(nh // nkv, dim=0)[None]
    ref = Fnn.scaled_dot_product_attention(qt, kt, vt, is_causal=True,
                                           scale=float(np.float32(1 / math.sqrt(d))))
    assert np.allclose(ours, ref[0].permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)
    # a decode query at position T-1 sees the whole prefix
    last = attention(q[-1:], K, V, np.array([T - 1]), nkv)
    assert np.allclose(last, ours[-1:], rtol=1e-13, atol=0)


def test_attention_special_cases():
    rng = np.random.default_rng(7)
    d = 16
    V = rng.normal(size=(1, 5, d))
    K = rng.normal(size=(1, 5, d))
    q = rng.normal(size=(1, 1, d))
    # one key -> output is that value
    assert np.allclose(attention(q, K, V, np.array([0]), 1)[0, 0], V[0, 0], rtol=0, atol=1e-15)
    # equal scores (q = 0) -> mean of the allowed values
    o = attention(np.zeros((1, 1, d)), K, V, np.array([3]), 1)
    assert np.allclose(o[0, 0], V[0, :4].mean(axis=0), rtol=1e-14, atol=1e-15)


def test_softmax_rows_sum_to_one_fp32():
    rng = np.random.default_rng(8)
    S, d = 300, 64
    q = rng.normal(size=(S, 1, d)).astype(np.float32)
    K = rng.normal(size=(1, S, d)).astype(np.float32)
    V = np.ones((1, S, d), np.float32)         # output = sum(p) / sum(p)
    o = attention(q, K, V, np.arange(S), 1, acc=np.float32)
    assert np.all(np.abs(o - 1) <= S * 2.0 ** -24)


# ------------------------------------------------------------------ the layer
SMALL = Shape(n_layers=2, hidden=128, n_heads=4, n_kv_heads=2, head_dim=32, ffn=256,
              max_batch=2, max_prompt=12, max_seq=20)


def _prompt(B, P, H, seed=0):
    return fpgen.prompt(seed, B, P, H)


def test_identity_when_output_projections_are_zero():
    s = SMALL
    zero = {(l, n): np.zeros(shp, np.float32) for l in range(s.n_layers)
            for n, shp in weight_shapes(s).items() if n in ("o", "down")}
    fp = Fingerprint(s, "bf16", "bf16", weights=zero)
    x = _prompt(2, 12, s.hidden)
    assert np.array_equal(fp.prefill(x), x)
    assert np.array_equal(fp.decode(x[:, -1]), x[:, -1])


def test_causality_and_batch_independence():
    s = SMALL
    fp = Fingerprint(s, "int8", "int8")
    x = _prompt(2, 12, s.hidden)
    y = fp.prefill(x)
    x2 = x.copy()
    x2[:, 7:] = bf16_round(x2[:, 7:] * 1.5 + 0.25)
    y2 = fp.prefill(x2)
    assert np.array_equal(y[:, :7], y2[:, :7])
    assert not np.array_equal(y[:, 7:], y2[:, 7:])
    y_b1 = fp.prefill(x[1:2])
    assert np.array_equal(y_b1[0], y[1])


@pytest.mark.parametrize("wq,kvq", [("bf16", "bf16"), ("int8", "int8"), ("int4", "bf16"),
                                    ("int4", "int8"), ("sp24", "int8")])
def test_kv_cached_decode_equals_full_recompute(wq, kvq):
    s = SMALL
    P, S = 8, 6
    fp = Fingerprint(s, wq, kvq)
    x = _prompt(2, P, s.hidden)
    y0, ys = fp.run(x, S)
    inputs = [y0[:, -1]] + ys[:-1]          # what each decode step consumed
    full_in = np.concatenate([x, np.stack(inputs, axis=1)], axis=1)
    yfull = fp.prefill(full_in)
    assert np.array_equal(yfull[:, :P], y0)
    dec = np.stack(ys, axis=1)
    err = np.abs(yfull[:, P:] - dec).max() / np.abs(dec).max()
    assert err <= 1e-9, err


def test_gqa_groups_share_kv_head():
    """With nkv = 1 every query head reads the same cache; permuting query heads of W_q
    permutes the attention output heads (checked through the layer with W_o = identity
    sized blocks)."""
    s = Shape(1, 64, 4, 1, 16, 128, 1, 6, 6)
    fp = Fingerprint(s, "bf16", "bf16")
    x = _prompt(1, 6, 64)
    W = fp.layers[0]
    xn = bf16_round(rmsnorm(x, W["attn_norm"], s.rms_eps)).astype(np.float64)
    q = (xn @ W["q"].T).reshape(1, 6, 4, 16)
    k = (xn @ W["k"].T).reshape(1, 6, 1, 16)
    v = (xn @ W["v"].T).reshape(1, 6, 1, 16)
    cos, sin = rope_tables(6, 16, 1e4)
    q = apply_rope(q, cos, sin)
    k = apply_rope(k, cos, sin)
    K = bf16_round(k[0].transpose(1, 0, 2)).astype(np.float64)
    V = bf16_round(v[0].transpose(1, 0, 2)).astype(np.float64)
    o = attention(q[0], K, V, np.arange(6), 1)
    perm = [2, 0, 3, 1]
    o_perm = attention(q[0][:, perm], K, V, np.arange(6), 1)
    assert np.array_equal(o_perm, o[:, perm])


def test_teacher_forcing_hook_reproduces_free_run():
    s = SMALL
    fp = Fingerprint(s, "bf16", "bf16")
    x = _prompt(1, 8, s.hidden)
    y0, ys = fp.run(x, 4)
    inputs = [y0[:, -1]] + ys[:-1]
    y0b, ysb = fp.run(x, 4, teacher=inputs)
    assert all(np.array_equal(a, b) for a, b in zip(ys, ysb))


@pytest.mark.parametrize("kvq", ["bf16", "int8"])
def test_layerwise_prefill_reproduces_chain(kvq):
    """Fed its own chain's layer inputs, the layer-by-layer prefill is the chained
    prefill, and decode continues from the same cache."""
    import dataclasses
    s = SMALL
    x = _prompt(2, 8, s.hidden)
    one = Fingerprint(dataclasses.replace(s, n_layers=1), "bf16", kvq)   # layer 0 alone
    y0 = one.prefill(x)
    fp = Fingerprint(s, "bf16", kvq)
    assert s.n_layers == 2
    y = fp.prefill(x)
    d = fp.decode(y[:, -1])
    fp2 = Fingerprint(s, "bf16", kvq)
    ys = fp2.prefill_layers([x, y0])
    assert np.array_equal(ys[0], y0) and np.array_equal(ys[1], y)
    assert np.array_equal(fp2.decode(y[:, -1]), d)
    # a different input to layer 1 changes only layer 1's output
    ys3 = Fingerprint(s, "bf16", kvq).prefill_layers([x, y0 * 0.5])
    assert np.array_equal(ys3[0], y0) and not np.array_equal(ys3[1], y)


def test_configs_are_the_workloads():
    assert set(CONFIGS) == {"tiny", "llama2-7b-bf16", "llama2-7b-int8", "llama2-13b-int4",
                            "llama2-70b-tp8-int4", "llama2-7b-sp24"}
    c5 = CONFIGS["llama2-70b-tp8-int4"]
    assert c5["shape"].hidden == 8192 and c5["shape"].n_heads == 8 and c5["shape"].n_kv_heads == 1


def _torch_kv_int8(u):
    """int8 KV store written with torch ops: u [B, P, n, d] fp32 (keys after the rotary
    embedding, or values) -> dequantised float64 values, with the codes and scales.
    One fp16 scale per (sequence, position, head): absmax / 127 rounded to fp16;
    codes = round-half-even(u / scale) clamped to +-127."""
    u = u.to(torch.float32)
    amax = u.abs().amax(dim=-1, keepdim=True)
    sc = (amax / 127.0).to(torch.float16).to(torch.float32)
    safe = torch.where(sc == 0, torch.ones_like(sc), sc)
    codes = torch.clamp(torch.round(u / safe), -127, 127)
    codes = torch.where(sc == 0, torch.zeros_like(codes), codes)
    return (codes * sc).double(), codes.to(torch.int8), sc[..., 0]


def _torch_layer_stack(fp, x, P, kvq="bf16", kv_out=None):
    """The same layer built from torch library routines: F.linear (weight [out, in]),
    F.rms_norm, rotary embedding as complex multiplication (torch.polar),
    F.scaled_dot_product_attention and F.silu, rounding to bf16 at the same points.
    With kvq = "int8" the keys (after the rotary embedding) and values go through the
    int8 store of ``_torch_kv_int8`` from fp32; ``kv_out`` collects its codes and scales."""
    s = fp.s
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    rb = lambda a: torch.from_numpy(bf16_round(a.numpy()).astype(np.float64))
    inv = 1e4 ** (-torch.arange(0, s.head_dim // 2, dtype=torch.float64) * 2 / s.head_dim)
    ang = torch.arange(P, dtype=torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)
    rot = torch.complex(rot.real.float().double(), rot.imag.float().double())   # fp32 tables

    def rope(u):                       # u [B, P, n, d]
        d2 = s.head_dim // 2
        z = torch.complex(u[..., :d2], u[..., d2:]) * rot[None, :, None, :]
        return torch.cat([z.real, z.imag], dim=-1)

    xx = t(x)
    B = xx.shape[0]
    for L in fp.layers:
        xn = rb(Fnn.rms_norm(xx, (s.hidden,), weight=t(L["attn_norm"]), eps=s.rms_eps))
        q = rope(Fnn.linear(xn, t(L["q"])).view(B, P, s.n_heads, s.head_dim))
        k = rope(Fnn.linear(xn, t(L["k"])).view(B, P, s.n_kv_heads, s.head_dim))
        v = Fnn.linear(xn, t(L["v"])).view(B, P, s.n_kv_heads, s.head_dim)
        if kvq == "int8":
            k, kc, ksc = _torch_kv_int8(k)
            v, vc, vsc = _torch_kv_int8(v)
            if kv_out is not None:
                kv_out.append((kc, ksc, vc, vsc))
        else:
            k, v = rb(k), rb(v)
        g = s.n_heads // s.n_kv_heads
        o = Fnn.scaled_dot_product_attention(
            q.transpose(1, 2), k.transpose(1, 2).repeat_interleave(g, 1),
            v.transpose(1, 2).repeat_interleave(g, 1), is_causal=True,
            scale=float(np.float32(1 / math.sqrt(s.head_dim))))
        o = rb(o.transpose(1, 2).reshape(B, P, -1))
        h = rb(xx + Fnn.linear(o, t(L["o"])))
        hn = rb(Fnn.rms_norm(h, (s.hidden,), weight=t(L["mlp_norm"]), eps=s.rms_eps))
        a = rb(Fnn.silu(Fnn.linear(hn, t(L["gate"]))) * Fnn.linear(hn, t(L["up"])))
        xx = rb(h + Fnn.linear(a, t(L["down"])))
    return xx.numpy()


@pytest.mark.parametrize("wq,kvq", [("bf16", "bf16"), ("int8", "bf16"), ("int4", "bf16"),
                                    ("bf16", "int8"), ("int8", "int8"), ("int4", "int8"),
                                    ("sp24", "bf16")])
def test_layer_matches_torch_functional_composition(wq, kvq):
    s = Shape(2, 128, 4, 2, 32, 256, 2, 10, 10)
    fp = Fingerprint(s, wq, kvq)
    x = _prompt(2, 10, s.hidden, seed=3)
    ours = fp.prefill(x)
    ref = _torch_layer_stack(fp, x, 10, kvq)
    err = np.abs(ours - ref).max() / np.abs(ref).max()
    assert err <= 1e-6, err


def test_int8_kv_codes_rebuilt_from_torch_ops():
    """The int8 cache the oracle writes (codes and fp16 scales per sequence, position and
    kv head) equals the one rebuilt independently with torch ops: keys quantised after
    the rotary embedding, both keys and values quantised from their fp32 values (no
    bf16 rounding first), for every layer of a two-layer stack."""
    s = Shape(2, 256, 4, 2, 64, 256, 2, 12, 12)
    for wq in ("bf16", "int4"):
        fp = Fingerprint(s, wq, "int8")
        x = _prompt(2, 12, s.hidden, seed=6)
        fp.prefill(x)
        kv = []
        _torch_layer_stack(fp, x, 12, "int8", kv_out=kv)
        for l, (kc, ksc, vc, vsc) in enumerate(kv):
            cc = fp.kv_codes[l]
            # torch [B, P, nkv, d] -> oracle layout [B, nkv, P, d]
            assert np.array_equal(cc["k"][:, :, :12], kc.permute(0, 2, 1, 3).numpy()), (wq, l)
            assert np.array_equal(cc["v"][:, :, :12], vc.permute(0, 2, 1, 3).numpy()), (wq, l)
            assert np.array_equal(cc["ks"][:, :, :12], ksc.permute(0, 2, 1).numpy()), (wq, l)
            assert np.array_equal(cc["vs"][:, :, :12], vsc.permute(0, 2, 1).numpy()), (wq, l)


def test_sp24_layer_weights_are_the_pruned_generator_weights():
    """Each projection of a 2:4 fingerprint is the bf16 generator weight with the magnitude
    2:4 mask applied: half of every row zero, the kept values unchanged."""
    from oracle.quant import prune_2of4
    s = Shape(1, 128, 4, 2, 32, 256, 1, 8, 8)
    fp = Fingerprint(s, "sp24", "bf16")
    for name, shp in weight_shapes(s).items():
        w = fpgen.weight(0, 0, {"q": 1, "k": 2, "v": 3, "o": 4, "gate": 6, "up": 7, "down": 8}[name], shp)
        got = fp.export_weight(0, name)[0]
        assert np.array_equal(got, np.where(prune_2of4(w), w, 0)), name
        assert np.count_nonzero(got == 0) >= got.size // 2

"""CPU tests of bench.py's contract and measurement model (no GPU needed).

The decode-step byte counts are pinned to the per-step algorithmic bytes of the four
full-size workloads (weights and norm gains, the cached keys and values read and the new
ones written, and the activations each projection reads and writes), averaged over the
100 decode positions after the prompt.  The prefill flop count is checked against a
direct count of the projection and causal-attention multiply-adds.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from fpgen.workloads import CONFIGS  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


@pytest.mark.parametrize("name,mb", [("llama2-7b-bf16", 828.2), ("llama2-7b-int8", 558.0),
                                     ("llama2-13b-int4", 3508.4), ("llama2-70b-tp8-int4", 388.6)])
def test_decode_step_bytes_match_the_workload_table(name, mb):
    c = CONFIGS[name]
    s, B, P, S = c["shape"], c["B"], c["P"], 100
    mean = sum(bench.decode_step_bytes(s, c["wq"], c["kvq"], B, P + i) for i in range(S)) / S
    assert abs(mean / 1e6 - mb) < 0.05


def test_decode_step_bytes_by_hand_for_the_7b_bf16_step():
    # two layers; weights [N, K] bf16; gains 2 x hidden bf16; bf16 cache of 32 heads x 128
    s = CONFIGS["llama2-7b-bf16"]["shape"]
    H, F, t = 4096, 11008, 512
    w = (3 * H * H + H * H + 2 * F * H + H * F) * 2 + 2 * H * 2
    kv_tok = 2 * 32 * 128 * 2
    act = 2 * (4 * H + 2 * H + 2 * F)
    per_layer = w + (t + 1) * kv_tok + kv_tok + act
    assert bench.decode_step_bytes(s, "bf16", "bf16", 1, t) == 2 * per_layer


def test_prefill_flops_by_hand():
    s = CONFIGS["llama2-7b-bf16"]["shape"]
    H, F, P = 4096, 11008, 512
    proj = 2 * P * (3 * H * H + H * H + 2 * F * H + H * F)
    attn = 4 * 128 * 32 * (P * (P + 1) // 2)       # q.k and p.v over the causal pairs
    assert bench.prefill_flops(s, 1, P) == 2 * (proj + attn)


def test_traffic_is_reported_only_for_the_sources_it_was_measured_on(monkeypatch):
    h = bench.src_hash("prefill_gemm")
    assert h != bench.src_hash("decode_proj")
    monkeypatch.setattr(bench, "TRAFFIC", {("prefill_gemm", "w"): {"src": h, "bytes_per_launch": 123}})
    assert bench.measured_traffic("prefill_gemm", "w") == 123
    assert bench.measured_traffic("prefill_gemm", "other") is None
    assert bench.measured_traffic("decode_proj", "w") is None
    monkeypatch.setattr(bench, "TRAFFIC", {("prefill_gemm", "w"): {"src": "0" * 16, "bytes_per_launch": 123}})
    assert bench.measured_traffic("prefill_gemm", "w") is None


def test_headline_is_the_largest_single_gpu_workload():
    head, names = bench.workload_names()
    assert head == "llama2-70b-tp8-int4" and names[0] == head and len(names) == len(CONFIGS)
    big = max(CONFIGS, key=lambda n: (CONFIGS[n]["B"] * CONFIGS[n]["P"], CONFIGS[n]["shape"].hidden))
    assert big == head


def test_cpu_baseline_sample_reports_the_host(monkeypatch):
    """The CPU baseline times the oracle's float32 mode on a one-layer, one-sequence
    sample and scales the rate to the workload's layer count."""
    import dataclasses
    from fpgen.workloads import Shape
    cfg = dict(shape=Shape(3, 128, 2, 2, 64, 256, 4, 8, 12), wq="int8", kvq="int8", B=4, P=8, S=4)
    r = bench.cpu_baseline(cfg, 0, 0.01)
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s" and r["value"] > 0
    assert r["cores"] >= 1 and r["nproc"] >= 1 and isinstance(r["cpu_model"], str)
    assert "1 of 3 layers" in r["sample"] and "float32" in r["sample"]


def test_sparse_bytes_and_flops_by_hand():
    """2:4 sparse weights: half the weights kept as bf16 with a 2-bit position each (9/16 of
    the dense bf16 bytes); the prefill's projection work is that of the kept half."""
    c = CONFIGS["llama2-7b-sp24"]
    s = c["shape"]
    H, F = 4096, 11008
    w_dense = (3 * H * H + H * H + 2 * F * H + H * F)
    assert bench.weight_bytes(3 * H, H, "sp24") == 3 * H * H * 1.125
    b_sp = bench.decode_step_bytes(s, "sp24", "bf16", 1, 512)
    b_bf = bench.decode_step_bytes(s, "bf16", "bf16", 1, 512)
    assert b_bf - b_sp == 2 * w_dense * (2 - 1.125)
    P = 512
    attn = 4 * 128 * 32 * (P * (P + 1) // 2)
    assert bench.prefill_flops(s, 1, P, "sp24") == 2 * (2 * P * w_dense // 2 + attn)

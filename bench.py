#!/usr/bin/env python
"""Benchmark of the fingerprint forward pass on one MI355X.

One "step" is one pass of the whole hot path over one batch: a prefill over the
prompt (the time to first token) followed by S KV-cached decode steps, each
feeding its output back as the next input (the time per output token) -- the
dummy request iServe's Profiler sends to a fingerprint (paper Sec. 4.2, Sec. 5.3,
Eq. 1).  Inputs are synthetic and already resident in HBM when timing starts.

By default every workload of the table is measured in one invocation and the
headline is the largest one that fits one GPU (the 70B model's 1/8
tensor-parallel shard: the largest model, prompt, batch and prefill).  Prints ONE
JSON line: ``value`` is the headline's decode tokens/s = B * S * steps / (total
decode time); its prefill time, MFMA utilisation, step rate against HBM peak, the
dominant kernel's roofline and the CPU oracle's rate sit beside it, and
``workloads`` holds the same figures for every workload.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "fingerprint decode tokens/s + % HBM roofline; prefill MFMA utilisation"
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
MFMA16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 / fp16 MFMA
# weight bytes per dense weight; 2:4 sparse: half the weights kept as bf16 plus a 2-bit
# position each (1.125 B), the algorithmic multiply work is that of the kept half
WBYTES = {"bf16": 2.0, "int8": 1.0, "int4": 0.5, "sp24": 1.125}
WFLOPS = {"bf16": 1.0, "int8": 1.0, "int4": 1.0, "sp24": 0.5}

KIND = {0: "rmsnorm", 1: "qkv", 2: "rope_kv", 3: "attn", 4: "o", 5: "resid_norm", 6: "gate_up",
        7: "swiglu", 8: "down", 9: "pos"}
PROJ = {"qkv", "o", "gate_up", "down"}

# Measured HBM bytes per launch of a kernel family on a workload, from two rocprofv3
# --pmc passes (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0, the factors a 1 GiB device copy
# gives), averaged over the family's launches.  Valid only for the kernel sources they
# were taken on (hash of the kernel's source files and of its argument block in
# fp_internal.h); the summaries and commands are in profiles/.
TRAFFIC = {
    ("prefill_gemm", "llama2-70b-tp8-int4"): {"src": "ef13af709f851df1", "bytes_per_launch": 8605742090},
    ("prefill_attn", "llama2-70b-tp8-int4"): {"src": "4c143c5591b38ef6", "bytes_per_launch": 1622333522},
    ("decode_proj", "llama2-70b-tp8-int4"): {"src": "7bbc74de5f69e243", "bytes_per_launch": 27162882},
    ("decode_attn", "llama2-70b-tp8-int4"): {"src": "3348a08a368fc693", "bytes_per_launch": 47377051},
    ("decode_proj", "llama2-7b-bf16"): {"src": "7bbc74de5f69e243", "bytes_per_launch": 102930905},
}
FAMILY_SRC = {
    "decode_proj": (("skinny.hip", "fp_device.h"), r"enum XForm \{.*?\n\};\n.*?struct SkinnyArgs \{.*?\n\};"),
    "prefill_gemm": (("gemm.hip", "fp_device.h"), r"struct GemmArgs \{.*?\n\};"),
    "prefill_attn": (("attn_prefill.hip", "fp_device.h"), r"struct AttnPreArgs \{.*?\n\};"),
    "decode_attn": (("attn_decode.hip", "fp_device.h"), r"struct AttnDecArgs \{.*?\n\};"),
}


def src_hash(family="decode_proj"):
    import hashlib
    import re
    files, pat = FAMILY_SRC[family]
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2501_13111_amd", "csrc")
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(csrc, "fp_internal.h")) as fh:
        hdr = fh.read()
    m = re.search(pat, hdr, re.S)
    h.update(m.group(0).encode() if m else b"")
    return h.hexdigest()[:16]


def skinny_src_hash():
    return src_hash("decode_proj")


def measured_traffic(family, config):
    """Measured bytes per launch, or None when not measured for this workload or the
    kernel sources changed since the counters were taken."""
    t = TRAFFIC.get((family, config))
    if t is None or t["src"] != src_hash(family):
        return None
    return t["bytes_per_launch"]


def skinny_traffic(config):
    return measured_traffic("decode_proj", config)


def cfg_of(name):
    from fpgen.workloads import CONFIGS
    return CONFIGS[name]


def workload_names():
    from fpgen.workloads import CONFIGS, HEADLINE
    return HEADLINE, [HEADLINE] + [n for n in CONFIGS if n != HEADLINE]


def proj_dims(s):
    """(N, K) of the fused projections of one layer."""
    qd, kd = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
    return {"qkv": (qd + 2 * kd, s.hidden), "o": (s.hidden, qd), "gate_up": (2 * s.ffn, s.hidden),
            "down": (s.hidden, s.ffn)}


def weight_bytes(N, K, wq):
    b = N * K * WBYTES[wq]
    if wq == "int8":
        b += N * 2                     # fp16 row scales
    elif wq == "int4":
        b += N * (K // 128) * 4        # fp16 scale + zero per group
    return b


def proj_bytes(kind, s, wq, M):
    """Algorithmic bytes of one decode projection launch: weights + input + output."""
    N, K = proj_dims(s)[kind]
    return weight_bytes(N, K, wq) + M * K * 2 + M * N * 2


def kv_tok_bytes(s, kvq):
    return 2 * s.n_kv_heads * s.head_dim * (1 if kvq == "int8" else 2) + (4 * s.n_kv_heads if kvq == "int8" else 0)


def decode_step_bytes(s, wq, kvq, B, t):
    """Algorithmic HBM bytes of one decode step at position t (the new token's index)."""
    per_layer = sum(weight_bytes(N, K, wq) for N, K in proj_dims(s).values()) + 2 * s.hidden * 2
    kvt = kv_tok_bytes(s, kvq)
    per_layer += B * (t + 1) * kvt + B * kvt
    per_layer += B * 2 * (4 * s.hidden + 2 * s.n_heads * s.head_dim + 2 * s.ffn)
    return s.n_layers * per_layer


def prefill_flops(s, B, P, wq="bf16"):
    params = sum(N * K for N, K in proj_dims(s).values()) * WFLOPS[wq]
    return s.n_layers * int(2 * B * P * params + 4 * s.head_dim * s.n_heads * B * P * (P + 1) // 2)


def profile_decode(fp, x, y, stream_ptr):
    """One eager decode step, timed per launch on the bench stream: the library stamps a
    start / stop HIP event pair from each kernel's own dispatch (hipExtLaunchKernel), so an
    interval is that kernel's execution."""
    import ctypes
    from paper_2501_13111_amd import binding

    class KT(ctypes.Structure):
        _fields_ = [("kind", ctypes.c_int32), ("layer", ctypes.c_int32), ("ms", ctypes.c_float)]
    L = binding.load()
    L.fp_profile_decode_step.argtypes = [ctypes.c_void_p] * 4 + [ctypes.POINTER(KT), ctypes.c_int32,
                                                                 ctypes.POINTER(ctypes.c_int32)]
    L.fp_profile_decode_step.restype = ctypes.c_int
    recs = (KT * 512)()
    n = ctypes.c_int32()
    rc = L.fp_profile_decode_step(fp._h, x.data_ptr(), y.data_ptr(), stream_ptr, recs, 512, ctypes.byref(n))
    if rc != 0:
        raise RuntimeError(f"fp_profile_decode_step: {L.fp_last_error().decode()}")
    return [(KIND[recs[i].kind], recs[i].layer, recs[i].ms) for i in range(n.value)]


def profile_prefill(fp, x, y, B, P, stream_ptr):
    import ctypes
    from paper_2501_13111_amd import binding

    class KT(ctypes.Structure):
        _fields_ = [("kind", ctypes.c_int32), ("layer", ctypes.c_int32), ("ms", ctypes.c_float)]
    L = binding.load()
    L.fp_profile_prefill.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(KT), ctypes.c_int32,
                                     ctypes.POINTER(ctypes.c_int32)]
    L.fp_profile_prefill.restype = ctypes.c_int
    recs = (KT * 512)()
    n = ctypes.c_int32()
    rc = L.fp_profile_prefill(fp._h, x.data_ptr(), B, P, y.data_ptr(), stream_ptr, recs, 512, ctypes.byref(n))
    if rc != 0:
        raise RuntimeError(f"fp_profile_prefill: {L.fp_last_error().decode()}")
    fp.B = B
    return [(KIND[recs[i].kind], recs[i].layer, recs[i].ms) for i in range(n.value)]


def host_info():
    """CPU model, logical CPUs visible and the BLAS threads numpy runs with."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info()), default=None)
    except Exception:
        pass
    return model, nproc, threads or nproc


def cpu_baseline(cfg, seed, budget_s):
    """The oracle, as it stands, in its float32 (BLAS sgemm) mode on a bounded sample of
    the workload: a one-layer fingerprint of the same shape and formats, one sequence,
    the full prompt, then decode steps until about ``budget_s`` seconds of decode have
    run.  Decode time scales linearly with the number of layers (every layer does the
    same work), so the rate is quoted for the workload's layer count: tokens/s =
    steps / (decode seconds x layers)."""
    import dataclasses
    import numpy as np
    import fpgen
    from oracle.layer import Fingerprint as OracleFingerprint
    s = cfg["shape"]
    L = s.n_layers
    s1 = dataclasses.replace(s, n_layers=1, max_batch=1)
    orc = OracleFingerprint(s1, cfg["wq"], cfg["kvq"], seed, acc=np.float32)
    x = fpgen.prompt(seed, cfg["B"], cfg["P"], s.hidden, b_start=0, b_count=1)
    t0 = time.perf_counter()
    y = orc.prefill(x)
    t_pre = time.perf_counter() - t0
    xin = y[:, -1, :]
    n, t_dec = 0, 0.0
    while n < cfg["S"] and (t_dec < budget_s or n < 2):
        t0 = time.perf_counter()
        xin = orc.decode(xin)
        t_dec += time.perf_counter() - t0
        n += 1
    model, nproc, threads = host_info()
    return {"value": round(n / (t_dec * L), 3), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"1 of {L} layers and 1 of {cfg['B']} sequences: prefill of {cfg['P']} tokens "
                      f"({t_pre:.2f} s) then {n} decode steps ({t_dec:.2f} s), float32 numpy/BLAS "
                      f"oracle, rate scaled to {L} layers",
            "prefill_tokens_per_s": round(cfg["P"] / (t_pre * L), 2),
            "cpu_model": model, "nproc": nproc, "blas_threads": threads}


def gemm_flops(kind, s, M, wq="bf16"):
    N, K = proj_dims(s)[kind]
    return int(2 * M * N * K * WFLOPS[wq])


def attn_kv_bytes(s, kvq, B, t):
    """Algorithmic bytes of one decode attention launch at position t: the cached keys
    and values read (t + 1 positions) and the new row written."""
    return B * (t + 2) * kv_tok_bytes(s, kvq)


def roofline_entry(kernel, bound, achieved, peak, unit, avg_ms, per_launch, traffic):
    return {"kernel": kernel, "bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic,
            "avg_launch_us": round(1e3 * avg_ms, 3),
            ("flops_per_launch_avg" if unit == "TFLOP/s" else "bytes_per_launch_avg"): int(per_launch)}


def run_workload(name, args, torch, timed_out=None):
    """Measure one workload: W warm-up passes, K timed passes (a pass is a prefill and S
    decode steps in one fp_decode_steps call), one pass with a graph per decode step for
    the step-time distribution, and one eagerly profiled prefill and eight decode steps
    for the per-kernel figures."""
    from paper_2501_13111_amd import Fingerprint, fill_normal
    cfg = cfg_of(name)
    s, wq, kvq, B, Pp, S = cfg["shape"], cfg["wq"], cfg["kvq"], cfg["B"], cfg["P"], cfg["S"]
    H = s.hidden
    print(f"bench: {name} (B={B} P={Pp} S={S})", file=sys.stderr, flush=True)
    fp = Fingerprint(s, wq, kvq, args.seed)
    fp.set_decode_graph(not args.no_graph)
    stream = torch.cuda.current_stream()
    sp = int(stream.cuda_stream)
    x = torch.empty(B * Pp * H, dtype=torch.bfloat16, device="cuda")
    fill_normal(x, args.seed, -1, 15, 0.0, 1.0)
    y = torch.empty_like(x)
    bufs = [torch.empty(B * H, dtype=torch.bfloat16, device="cuda") for _ in range(2)]

    def one_pass(events=None):
        fp.prefill(x, y, B, Pp)
        if events is not None:
            events[0].record(stream)
        bufs[0].copy_(y.view(B, Pp, H)[:, -1, :].reshape(-1))
        fp.decode_steps(bufs[0], bufs[1], S)          # the S steps in one call (one graph replay)
        if events is not None:
            events[1].record(stream)

    for _ in range(args.warmup):
        one_pass()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        one_pass(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    prefill_ms = [starts[k].elapsed_time(evs[k][0]) for k in range(args.steps)]
    decode_ms = [evs[k][0].elapsed_time(evs[k][1]) for k in range(args.steps)]
    pass_step_ms = [d / S for d in decode_ms]          # per pass: the mean step of its S steps
    dec_total_s = sum(decode_ms) / 1e3
    value = B * S * args.steps / dec_total_s
    mean_bytes = statistics.fmean(decode_step_bytes(s, wq, kvq, B, Pp + i) for i in range(S))
    step_frac = mean_bytes / (statistics.fmean(pass_step_ms) / 1e3) / 1e9 / HBM_PEAK_GBS

    # ---- step-time distribution: one pass with one graph replay per decode step
    fp.prefill(x, y, B, Pp)
    bufs[0].copy_(y.view(B, Pp, H)[:, -1, :].reshape(-1))
    sev = [torch.cuda.Event(enable_timing=True) for _ in range(S + 1)]
    sev[0].record(stream)
    for st in range(S):
        fp.decode_step(bufs[st % 2], bufs[(st + 1) % 2])
        sev[st + 1].record(stream)
    torch.cuda.synchronize()
    single = sorted(sev[i].elapsed_time(sev[i + 1]) for i in range(S))
    pct = lambda q: single[min(S - 1, int(round(q * (S - 1))))]

    # ---- per-kernel profile of a prefill and a decode step (eager, HIP events per launch)
    pre_prof = profile_prefill(fp, x, y, B, Pp, sp)
    bufs[0].copy_(y.view(B, Pp, H)[:, -1, :].reshape(-1))
    dec_profs = []
    for st in range(min(S, 8)):
        dec_profs.append(profile_decode(fp, bufs[st % 2], bufs[(st + 1) % 2], sp))
    fp.close()
    by_kind = {}
    for prof in dec_profs:
        for kind, layer, ms in prof:
            by_kind.setdefault(kind, []).append(ms)
    pre_kinds = {}
    for kind, _, ms in pre_prof:
        pre_kinds[kind] = pre_kinds.get(kind, 0.0) + ms

    # decode projections (the weight-streaming kernels): bytes per launch over time per launch
    proj_ms = [ms for prof in dec_profs for kind, _, ms in prof if kind in PROJ]
    proj_b = [proj_bytes(kind, s, wq, B) for prof in dec_profs for kind, _, _ in prof if kind in PROJ]
    dec_kernel = "sp24_gemv_kernel" if wq == "sp24" else ("skinny_kernel" if B == 1 else "skinny_batch_kernel")
    roof_dec = roofline_entry(f"{dec_kernel} (decode projections qkv/o/gate_up/down)", "hbm",
                              sum(proj_b) / (sum(proj_ms) / 1e3) / 1e9, HBM_PEAK_GBS, "GB/s",
                              statistics.fmean(proj_ms), statistics.fmean(proj_b),
                              measured_traffic("decode_proj", name))
    # decode attention: cached K/V bytes read per launch (positions Pp .. Pp+7 of the profile)
    att_ms = [ms for prof in dec_profs for kind, _, ms in prof if kind == "attn"]
    att_b = [attn_kv_bytes(s, kvq, B, Pp + i) for i, prof in enumerate(dec_profs)
             for kind, _, _ in prof if kind == "attn"]
    roof_att = roofline_entry("attn_decode_kernel (+ merge)", "hbm", sum(att_b) / (sum(att_ms) / 1e3) / 1e9,
                              HBM_PEAK_GBS, "GB/s", statistics.fmean(att_ms), statistics.fmean(att_b),
                              measured_traffic("decode_attn", name))
    # prefill GEMMs: flops per launch over time per launch (the kinds' split-K reductions
    # included when a GEMM is split)
    g_ms = [ms for kind, _, ms in pre_prof if kind in PROJ]
    g_fl = [gemm_flops(kind, s, B * Pp, wq) for kind, _, _ in pre_prof if kind in PROJ]
    gemm_kernel = ("gemm_sp24_kernel (sparse MFMA)" if wq == "sp24" else
                   "gemm_big_kernel" if B * Pp >= 4096 else "gemm_kernel / gemm_big_kernel split-K")
    roof_gemm = roofline_entry(f"{gemm_kernel} (prefill projections qkv/o/gate_up/down)", "mfma",
                               sum(g_fl) / (sum(g_ms) / 1e3) / 1e12, MFMA16_PEAK_TFLOPS, "TFLOP/s",
                               statistics.fmean(g_ms), statistics.fmean(g_fl),
                               measured_traffic("prefill_gemm", name))
    pa_ms = [ms for kind, _, ms in pre_prof if kind == "attn"]
    pa_fl = 4 * s.head_dim * s.n_heads * B * Pp * (Pp + 1) // 2
    roof_pattn = roofline_entry("attn_prefill_kernel (attn_prefill_ks_kernel on grids smaller than the CU count)", "mfma", pa_fl * len(pa_ms) / (sum(pa_ms) / 1e3) / 1e12,
                                MFMA16_PEAK_TFLOPS, "TFLOP/s", statistics.fmean(pa_ms), pa_fl,
                                measured_traffic("prefill_attn", name))
    # the dominant kernel family: the most time in one pass (prefill once, S decode steps)
    n_prof = len(dec_profs)
    pass_time = {"prefill_gemm": sum(g_ms), "prefill_attn": sum(pa_ms),
                 "decode_proj": S * sum(proj_ms) / n_prof, "decode_attn": S * sum(att_ms) / n_prof}
    roofs = {"prefill_gemm": roof_gemm, "prefill_attn": roof_pattn, "decode_proj": roof_dec,
             "decode_attn": roof_att}
    dom = max(pass_time, key=pass_time.get)
    roof = dict(roofs[dom])
    roof["family"] = dom
    roof["share_of_pass"] = round(pass_time[dom] / (statistics.median(prefill_ms) + statistics.median(decode_ms)), 4)

    pflops = prefill_flops(s, B, Pp, wq)
    pre_med = statistics.median(prefill_ms)
    out = {
        "value": round(value, 2), "unit": "tokens/s",
        "ms_per_step": round(1e3 * wall / args.steps, 4),
        "dtype": "bf16" if wq == "bf16" else "f16",
        "config": {"workload": name, "layers": s.n_layers, "hidden": H, "heads": s.n_heads,
                   "kv_heads": s.n_kv_heads, "head_dim": s.head_dim, "ffn": s.ffn, "weights": wq,
                   "kv_cache": kvq, "batch": B, "prompt": Pp, "decode_steps": S,
                   "decode_graph": not args.no_graph, "decode_steps_per_call": S},
        "decode_step_us": round(1e3 * statistics.median(pass_step_ms), 2),
        "decode_step_timing": "median over passes of the pass's mean step (the S steps run as one call)",
        "decode_step_us_p10_p50_p90": [round(1e3 * pct(q), 2) for q in (0.1, 0.5, 0.9)],
        "decode_step_single_timing": "one pass, one graph replay per step (adds one graph launch per step)",
        "decode_step_hbm_frac": round(step_frac, 4),
        "decode_step_algorithmic_MB": round(mean_bytes / 1e6, 2),
        "prefill_ms": round(pre_med, 4),
        "prefill_tflops": round(pflops / (pre_med / 1e3) / 1e12, 1),
        "prefill_mfma_frac": round(pflops / (pre_med / 1e3) / 1e12 / MFMA16_PEAK_TFLOPS, 4),
        "prefill_gemm_mfma_frac": roof_gemm["frac"],
        "tokens_per_s_incl_prefill": round(B * S * args.steps / (sum(prefill_ms) / 1e3 + dec_total_s), 2),
        "roofline": roof,
        "rooflines": roofs,
        "decode_kernel_us": {k: round(1e3 * statistics.fmean(v), 2) for k, v in sorted(by_kind.items())},
        "prefill_kernel_ms": {k: round(v, 4) for k, v in sorted(pre_kinds.items())},
    }
    if not args.no_cpu_baseline:
        print(f"bench: {name} cpu baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cfg, args.seed, args.cpu_budget)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="all",
                    help="a workload name, or 'all' (every workload; the headline is the largest)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=4.0,
                    help="seconds of oracle decode per workload for the CPU baseline")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device once (the reference kernel that "
                         "calibrates rocprofv3's FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this benchmark runs on one GPU; --gpus {args.gpus} is not supported "
              f"(the multi-GPU sharding is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2501_13111_amd as P
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe > 0:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n}), flush=True)
        return
    P.load()

    headline, names = workload_names()
    if args.config != "all":
        cfg_of(args.config)
        headline, names = args.config, [args.config]
    results = {n: run_workload(n, args, torch) for n in names}
    h = results[headline]
    out = {
        "metric": METRIC, "value": h["value"], "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": h["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": h["dtype"],
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) prompt hidden states; no checkpoint)",
    }
    for k, v in h.items():
        if k not in out:
            out[k] = v
    if len(names) > 1:
        out["workloads"] = {n: {k: v for k, v in r.items() if k not in ("rooflines",)}
                            for n, r in results.items()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

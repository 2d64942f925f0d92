"""Benchmark: tiled exact attention on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-gemm]
    python bench.py --config NAME      # one workload only (own JSON line)

A step is one pass of the whole hot path over one batch of synthetic input,
on the four full-size workloads:
  1. prefill B=1 H=32 Sq=Skv=8192 d=128, non-causal, inputs x0.5 (attn_fwd) --
     the largest prefill workload, the line's headline;
  2. prefill B=4 H=16 Sq=Skv=2048 d=128, causal (attn_fwd);
  3. Flash-Decode B=16 H=32 Skv=8192 d=128 (attn_decode: split partials +
     combine);
  4. Flash-Decode B=1 H=32 Skv=131072 d=128 (attn_decode).
Inputs are seeded bf16 tensors resident in HBM before the timed region.  Each
call is bracketed by HIP events on the stream it runs on; the step wall time
is bracketed by device synchronisation.  Before the W warmup steps the step
runs until --prewarm-ms of event-timed GPU work have passed (the clocks leave
their idle state only after some tens of ms), so the timed steps measure the
steady state whatever W is.

Printed (one JSON line): value = the headline prefill's TFLOP/s
(algorithmic flops: 4*d per unmasked (query, key) pair) with its MFMA
roofline; every leg with its own rate and roofline (MFMA for prefill, HBM
for decode: K, V, Q read once, O written once); the fp64 CPU oracle's rate on
a bounded sample of the headline workload, timed on this host's cores; and,
timed separately after the steps, the GEMM workload (C = A B at
M = N = K = 8192, bf16 in, fp32 out) with its MFMA roofline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 4096 flop/clk x 2.4 GHz (dense bf16 MFMA)
PEAK_HBM_GBS = 8000.0      # HBM3E

PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2609_29219_amd", "csrc")
# sources that decide which kernel runs and what it does
KERNEL_SOURCES = {
    "prefill": ("fwd_kernel.h", "fwd_d128.hip", "fwd_d64.hip", "lds_dma.h", "plan.cpp", "api.hip",
                "common.h"),
    "decode": ("decode.hip", "plan.cpp", "api.hip", "common.h"),
    "gemm": ("gemm.hip", "lds_dma.h", "plan.cpp", "api.hip", "common.h"),
}
GEMM_WORKLOAD = "gemm_m8192_n8192_k8192"
GEMM_SHAPE = (8192, 8192, 8192)


def source_hash(kind: str) -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kind]:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _profile_fields(kind: str, name: str):
    """key = value lines of a committed rocprofv3 summary, or None if it is
    missing or the kernel sources changed since the counters were taken."""
    path = os.path.join(PROFILES, name)
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, _, v = line.strip().partition("=")
                fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != source_hash(kind):
        return None
    return fields


def profiled_traffic(kind: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 summary (None if stale)."""
    fields = _profile_fields(kind, f"traffic_{workload}.txt")
    return None if fields is None else int(fields["traffic_bytes_per_launch"])


def profiled_mfma_busy(workload: str):
    """The prefill kernel's MFMA-busy share of SIMD cycles from the committed
    counter summary (None if stale or absent)."""
    fields = _profile_fields("prefill", f"mfma_{workload}.txt")
    return None if fields is None else float(fields["mfma_busy_fraction"])


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    # the clocks leave their idle state only after some tens of ms of GPU
    # work (the first steps after idle run ~20% slower), so the step first
    # runs for this much event-timed GPU time, whatever --warmup says
    ap.add_argument("--prewarm-ms", type=float, default=200.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm", action="store_true", help="skip the GEMM leg")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time for the oracle sample")
    ap.add_argument("--config", default=None, help="bench a single named workload")
    return ap.parse_args()


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def _prewarm(fn, prewarm_ms: float):
    """Run fn until prewarm_ms of event-timed GPU work have passed (the clocks
    leave their idle state); returns (GPU ms, calls)."""
    import torch
    done_ms, calls = 0.0, 0
    while done_ms < prewarm_ms:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(8):
            fn()
        e1.record()
        torch.cuda.synchronize()
        done_ms += e0.elapsed_time(e1)
        calls += 8
    return done_ms, calls


def _time_calls(fn, steps: int, warmup: int, prewarm_ms: float = 0.0):
    """Per-call device time (ms) from HIP events on the current stream."""
    import torch
    _prewarm(fn, prewarm_ms)
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    t0 = time.perf_counter()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    return sum(ms) / len(ms), ms[len(ms) // 2], wall


def _load_workload(w, dev):
    from attn_inputs import make_inputs
    q, k, v = make_inputs(w)
    return q, k, v, q.to(dev), k.to(dev), v.to(dev)


def cpu_baseline(w, q, k, v, target_s: float) -> dict:
    """The fp64 oracle on whole (b, h) slabs of the prefill workload."""
    import oracle
    import numpy as np
    heads = w.B * w.H
    qs, ks, vs = (t.reshape(heads, 1, t.shape[2], w.d) for t in (q, k, v))

    def run(n):
        t0 = time.perf_counter()
        oracle.attn(qs[:n].contiguous(), ks[:n].contiguous(), vs[:n].contiguous(), n, 1, w.Sq,
                    w.Skv, w.d, w.scale, w.causal)
        return time.perf_counter() - t0

    t1 = run(1)
    n = int(max(1, min(heads, target_s / max(t1, 1e-6))))
    t = run(n) if n > 1 else t1
    # when the whole workload takes less than the target, repeat whole passes
    # over it until the target is reached (a steadier rate)
    passes = 1
    while n == heads and t < target_s and passes < 64:
        t += run(n)
        passes += 1
    sample = w.with_(B=1, H=n)
    flops = sample.flops() * passes
    reps = f" x {passes} passes" if passes > 1 else ""
    return {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{n} of {heads} (b,h) slabs of {w.name}{reps} ({flops / 1e9:.2f} GFLOP "
                      f"in {t:.2f} s, fp64, {_cpu_model()})",
            "seconds": t}


HEADLINE = "prefill_b1_h32_s8192_d128"
STEP = (HEADLINE, "prefill_b4_h16_s2048_d128_causal", "decode_b16_h32_s8192_d128",
        "decode_b1_h32_s131072_d128")


def _leg(pa, w, dev):
    """(callable, plan line) for one workload on inputs resident in HBM."""
    import torch
    _, _, _, qd, kd, vd = _load_workload(w, dev)
    if w.kind == "fwd":
        o = torch.empty((w.B, w.H, w.Sq, w.d), dtype=torch.float32, device=dev)
        plan = pa.get_plan(pa.KIND_FWD, w.B, w.H, w.Sq, w.Skv, w.d, w.causal)
        return (lambda: pa.attn_fwd(qd, kd, vd, o=o, scale=w.scale, causal=w.causal)), plan
    o = torch.empty((w.B, w.H, w.d), dtype=torch.float32, device=dev)
    plan = pa.get_plan(pa.KIND_DECODE, w.B, w.H, 1, w.Skv, w.d)
    return (lambda: pa.attn_decode(qd, kd, vd, o=o)), plan


def _leg_record(w, ms: float, plan: str) -> dict:
    """Rate and roofline of one leg from its mean per-call device time."""
    shape = {"B": w.B, "H": w.H, "Sq": w.Sq, "Skv": w.Skv, "d": w.d, "causal": w.causal}
    if w.kind == "fwd":
        tflops = w.flops() / (ms * 1e-3) / 1e12
        return {"value": tflops, "unit": "TFLOP/s", "ms_per_call": ms, **shape, "plan": plan,
                "roofline": {"bound": "mfma", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                             "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS,
                             "traffic": profiled_traffic("prefill", w.name),
                             "algorithmic_bytes": w.hbm_bytes(), "kernel": "fwd_kernel",
                             "ms_per_launch": ms, "flops_per_launch": w.flops(),
                             "mfma_busy_fraction": profiled_mfma_busy(w.name)}}
    gbs = w.hbm_bytes() / (ms * 1e-3) / 1e9
    return {"value": gbs, "unit": "GB/s", "ms_per_call": ms, **shape, "plan": plan,
            "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": gbs / PEAK_HBM_GBS,
                         "traffic": profiled_traffic("decode", w.name),
                         "kernel": "decode_partial_kernel + split_combine_kernel",
                         "bytes_per_call": w.hbm_bytes()}}


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {a.gpus}); the attention path "
              "has no multi-GPU form", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2609_29219_amd as pa
    from attn_inputs import BY_NAME

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if a.config == GEMM_WORKLOAD:
        print(json.dumps(gemm_leg(pa, dev, steps=a.steps, warmup=a.warmup,
                                  prewarm_ms=a.prewarm_ms)), flush=True)
        return
    if a.config:
        w = BY_NAME[a.config]
        fn, plan = _leg(pa, w, dev)
        mean_ms, med_ms, wall = _time_calls(fn, a.steps, a.warmup, a.prewarm_ms)
        rec = {"workload": w.name, "ms_mean": mean_ms, "ms_median": med_ms,
               "ms_wall_per_call": wall, "plan": plan}
        if w.kind == "fwd":
            rec["tflops"] = w.flops() / (mean_ms * 1e-3) / 1e12
            rec["frac_mfma_peak"] = rec["tflops"] / PEAK_BF16_TFLOPS
        rec["gbs"] = w.hbm_bytes() / (mean_ms * 1e-3) / 1e9
        rec["frac_hbm_peak"] = rec["gbs"] / PEAK_HBM_GBS
        print(json.dumps(rec), flush=True)
        return

    ws = [BY_NAME[n] for n in STEP]
    legs = [_leg(pa, w, dev) for w in ws]
    fns = [fn for fn, _ in legs]

    def step():
        for fn in fns:
            fn()

    # pre-warm by GPU time, then the warmup steps
    pre_ms, pre_steps = _prewarm(step, a.prewarm_ms)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
          for _ in range(a.steps)]
    t0 = time.perf_counter()
    for marks in ev:
        marks[0].record()
        for i, fn in enumerate(fns):
            fn()
            marks[i + 1].record()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) / a.steps * 1e3
    leg_ms = [sum(m[i].elapsed_time(m[i + 1]) for m in ev) / a.steps for i in range(len(fns))]

    recs = {w.name: _leg_record(w, ms, plan) for w, ms, (_, plan) in zip(ws, leg_ms, legs)}
    head = recs[HEADLINE]
    wh = BY_NAME[HEADLINE]
    roof = dict(head["roofline"])
    roof["peak_from_device"] = device_peak(pa)
    rec = {
        "metric": "Attention TFLOP/s + % MFMA peak (prefill); KV HBM GB/s + % peak (decode)",
        "value": head["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "prewarm_ms": pre_ms,
        "prewarm_steps": pre_steps,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded bf16 N(0,1), x0.5 for the long prefill; resident in HBM)",
        "config": {"workload": HEADLINE, "step": list(STEP),
                   "B": wh.B, "H": wh.H, "Sq": wh.Sq, "Skv": wh.Skv, "d": wh.d,
                   "causal": wh.causal, "plan": head["plan"]},
        "roofline": roof,
        "legs": recs,
    }
    if not a.no_gemm:
        # the same time-based pre-warm as the attention step
        rec["gemm"] = gemm_leg(pa, dev, prewarm_ms=a.prewarm_ms)
    if not a.no_cpu_baseline:
        from attn_inputs import make_inputs
        q, k, v = make_inputs(wh)
        rec["cpu_baseline"] = cpu_baseline(wh, q, k, v, a.cpu_seconds)
    print(json.dumps(rec), flush=True)


def device_peak(pa) -> dict:
    """The dense bf16 MFMA peak recomputed from the properties this device
    reports (CUs x SIMDs x 1024 flop/clk x maximum clock), next to the
    published figure the roofline uses."""
    d = pa.query_device()
    tflops = d["num_cus"] * d["simds_per_cu"] * 1024 * d["clock_ghz"] / 1e3
    return {"value": tflops, "unit": "TFLOP/s", "cus": d["num_cus"],
            "simds_per_cu": d["simds_per_cu"], "clock_ghz": d["clock_ghz"]}


def gemm_leg(pa, dev, steps=20, warmup=10, prewarm_ms=0.0) -> dict:
    """The GEMM workload (C = A B, bf16 in, fp32 out) timed on its own after
    the attention step, outside its timed region."""
    import torch
    from attn_inputs import random_bf16
    M, N, K = GEMM_SHAPE
    a = random_bf16((M, K), 31).to(dev)
    b = random_bf16((K, N), 32).to(dev)
    c = torch.empty((M, N), dtype=torch.float32, device=dev)
    _prewarm(lambda: pa.gemm(a, b, c), prewarm_ms)
    for _ in range(warmup):
        pa.gemm(a, b, c)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        pa.gemm(a, b, c)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tflops = 2.0 * M * N * K / (ms * 1e-3) / 1e12
    plan = pa.gemm_plan(M, N, K)
    # the 256 x 256 tile on 2 x 2 waves is the hand-scheduled kernel
    kernel = "gemm_sched_kernel" if all(f in plan.split() for f in (
        "BLOCK_M=256", "BLOCK_N=256", "WAVES_M=2", "WAVES_N=2")) else "gemm_kernel"
    return {"workload": GEMM_WORKLOAD, "M": M, "N": N, "K": K, "value": tflops,
            "unit": "TFLOP/s", "ms_per_call": ms, "plan": plan,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS,
                         "traffic": profiled_traffic("gemm", GEMM_WORKLOAD),
                         "algorithmic_bytes": gemm_bytes(), "kernel": kernel}}


def gemm_bytes() -> int:
    """Algorithmic HBM bytes of the GEMM workload: A and B read once, C (fp32) written once."""
    M, N, K = GEMM_SHAPE
    return 2 * M * K + 2 * K * N + 4 * M * N


if __name__ == "__main__":
    main()

"""Planner validation on the device: the block-size ablation.

    python paper_2609_29219_amd/plan_ablation.py [--save FILE] [--load FILE] [--fit]
                                                 [--only-calibration] [--markdown FILE] [--gemm]

For each workload every feasible prefill candidate (block sizes, waves,
pipeline knob, key splits) is run through the ATTN_FORCE_PLAN hook and timed, and set
against the planner's modelled time: where the planner's pick ranks among the
measured times, how far it is from the measured best, how far the pick of the
analytic model alone (without the per-variant tile costs) is from it, whether
the best is in the modelled top five, the rank correlation of modelled and
measured times, and the pick's rank among its legal one-step neighbours
(block width one step up or down, the other wave count, the neighbouring
pipeline knob, the neighbouring key-split count).  Two workloads are the
calibration shapes (the analytic fields are fitted and the tile costs
characterised on them); every other row, the benchmarked workloads among
them, is held out.  The two benchmarked decode workloads are timed at every
split count the planner considers and set against the modelled time.  The
paper validates its model the same way (top-k candidates and block-size
neighbourhoods); measurement here validates, it never selects.

--gemm runs the same validation for the GEMM over the paper's shape range
(256 to 16384, square and skewed): every feasible tile (BM, BN, BK, wave
grid, pipe) is timed; the report gives the planner pick's measured and
modelled TFLOP/s, its rank, and its rank among the tiles one legal step away
in BM, BN, BK and pipe (the paper's local block-size perturbation).

--fit refits the four offline-calibrated fields of the device description
(issue_cycles_per_score, valu_mfma_overlap, tile_sync_cycles,
tile_latency_cycles) to the measured times of the calibration workloads by
least squares on log time, using the library's own analytic model (the
calibration is done once per architecture and then frozen into the built-in
description).  --load reuses
a saved measurement instead of timing; the candidates' register and
occupancy footprint still comes from the compiled kernels on the device.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import paper_2609_29219_amd as pa  # noqa: E402

# (name, B, H, Sq, Skv, d, causal)
WORKLOADS = [
    # the calibration shapes: the analytic fields are fitted and the per-variant
    # tile costs characterised on these two only
    ("b2_h16_s4096_d128", 2, 16, 4096, 4096, 128, False),
    ("b2_h16_s4096_d128_causal", 2, 16, 4096, 4096, 128, True),
    # the benchmarked prefill workloads (their own seeded inputs), held out
    ("single_head_s256_d64", 1, 1, 256, 256, 64, False),
    ("prefill_b4_h16_s2048_d128_causal", 4, 16, 2048, 2048, 128, True),
    ("prefill_b1_h32_s8192_d128", 1, 32, 8192, 8192, 128, False),
    # further held-out shapes
    ("b4_h16_s2048_d64", 4, 16, 2048, 2048, 64, False),
    ("b8_h8_s1024_d128", 8, 8, 1024, 1024, 128, False),
    # long causal at d = 64, where the VALU binds and another schedule wins
    ("b4_h16_s8192_d64_causal", 4, 16, 8192, 8192, 64, True),
    # few heads / few queries against many keys: key splits fill the CUs
    ("b1_h2_s8192_d128", 1, 2, 8192, 8192, 128, False),
    ("b1_h32_q256_kv32768_d128", 1, 32, 256, 32768, 128, False),
]
CALIBRATION = ("b2_h16_s4096_d128", "b2_h16_s4096_d128_causal")
# the benchmarked decode workloads: (name, B, H, Skv, d)
DECODE_WORKLOADS = [("decode_b16_h32_s8192_d128", 16, 32, 8192, 128),
                    ("decode_b1_h32_s131072_d128", 1, 32, 131072, 128)]
DECODE_SPLITS = (1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 192, 256, 384, 512)
SPLITS = (1, 2, 3, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 192, 256)
CALIBRATED = ("issue_cycles_per_score", "valu_mfma_overlap", "tile_sync_cycles",
              "tile_latency_cycles")


def key(c: dict) -> tuple:
    return (c["BLOCK_N"], c["WAVES"], c["PIPE"], c["KV_SPLITS"])


def time_variant(w, variant, iters=10, reps=3) -> float:
    """Best-of-reps mean time (us) of `iters` back-to-back launches."""
    import torch
    from attn_inputs import random_bf16
    from attn_inputs import BY_NAME, make_inputs
    name, B, H, Sq, Skv, d, causal = w
    if not hasattr(time_variant, "cache") or time_variant.cache[0] != name:
        if name in BY_NAME:  # a benchmarked workload: its own inputs
            q, k, v = (t.cuda() for t in make_inputs(BY_NAME[name]))
        else:
            q = random_bf16((B, H, Sq, d), 11).cuda()
            k = random_bf16((B, H, Skv, d), 12).cuda()
            v = random_bf16((B, H, Skv, d), 13).cuda()
        o = torch.empty((B, H, Sq, d), dtype=torch.float32, device="cuda")
        time_variant.cache = (name, q, k, v, o)
    _, q, k, v, o = time_variant.cache
    bn, nw, pipe, ns = variant
    os.environ["ATTN_FORCE_PLAN"] = f"bn={bn},waves={nw},pipe={pipe},splits={ns}"
    try:
        for _ in range(3):
            pa.attn_fwd(q, k, v, o=o, causal=causal)
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(iters):
                pa.attn_fwd(q, k, v, o=o, causal=causal)
            b.record()
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b) / iters * 1e3)
        return best
    finally:
        os.environ.pop("ATTN_FORCE_PLAN", None)


def neighbours(pick: tuple, feasible: set) -> list:
    """Feasible candidates at most one step from pick in every symbol."""
    domains = ((32, 64, 128), (4, 8), (0, 1, 2, 3), SPLITS)
    out = []
    for c in feasible:
        steps = [abs(dom.index(a) - dom.index(b)) for dom, a, b in zip(domains, c, pick)]
        if max(steps) <= 1 and sum(steps) > 0:
            out.append(c)
    return sorted(out)


def spearman(a, b) -> float:
    def ranks(x):
        order = sorted(range(len(x)), key=lambda i: x[i])
        r = [0.0] * len(x)
        for pos, i in enumerate(order):
            r[i] = pos
        return r
    ra, rb = ranks(a), ranks(b)
    n = len(a)
    if n < 2:
        return float("nan")
    ma, mb = sum(ra) / n, sum(rb) / n
    num = sum((x - ma) * (y - mb) for x, y in zip(ra, rb))
    den = math.sqrt(sum((x - ma) ** 2 for x in ra) * sum((y - mb) ** 2 for y in rb))
    return num / den if den else float("nan")


def summarise(w, cands: list, meas: dict, analytic: list) -> dict:
    rows = [(c["modeled_us"], meas[key(c)], key(c)) for c in cands if key(c) in meas]
    by_model = sorted(rows)
    by_meas = sorted(rows, key=lambda r: r[1])
    pick, best = by_model[0], by_meas[0]
    # the analytic model alone (without the per-variant tile costs)
    arows = sorted((c["modeled_us"], meas[key(c)], key(c)) for c in analytic if key(c) in meas)
    apick = arows[0]
    feasible = {r[2] for r in rows}
    nb = neighbours(pick[2], feasible)
    nb_times = [meas[n] for n in nb]
    return {
        "workload": w[0], "candidates": len(rows), "calibration": w[0] in CALIBRATION,
        "analytic_pick": apick[2], "analytic_pick_us": apick[1],
        "analytic_over_best": apick[1] / best[1] - 1.0,
        "pick": pick[2], "pick_us": pick[1], "pick_modeled_us": pick[0],
        "best": best[2], "best_us": best[1],
        "pick_over_best": pick[1] / best[1] - 1.0,
        "pick_measured_rank": [r[2] for r in by_meas].index(pick[2]) + 1,
        "best_in_model_top5": best[2] in [r[2] for r in by_model[:5]],
        "spearman": spearman([r[0] for r in rows], [r[1] for r in rows]),
        "neighbours": len(nb),
        "pick_rank_in_neighbourhood": 1 + sum(t < pick[1] for t in nb_times),
        "rows": [{"variant": r[2], "modeled_us": r[0], "measured_us": r[1]} for r in by_meas],
    }


def fit(data: dict) -> dict:
    """Least squares on log(modeled / measured) over every measured candidate
    of the calibration workloads, with the analytic model alone (the
    per-variant tile costs are characterised against it afterwards)."""
    from scipy.optimize import least_squares
    base = pa.DeviceDesc()
    pa.lib.attn_query_device(ctypes.byref(base))

    def resid(x):
        desc = pa.DeviceDesc()
        ctypes.memmove(ctypes.byref(desc), ctypes.byref(base), ctypes.sizeof(desc))
        for name, val in zip(CALIBRATED, x):
            setattr(desc, name, float(val))
        out = []
        for w in WORKLOADS:
            meas = data.get(w[0])
            if not meas or w[0] not in CALIBRATION:
                continue
            for c in pa.fwd_candidates(*w[1:], desc=desc, device_footprint=True,
                                       analytic_only=True):
                t = meas.get(key(c))
                if t:
                    out.append(math.log(c["modeled_us"]) - math.log(t))
        return out

    x0 = [getattr(base, n) for n in CALIBRATED]
    sol = least_squares(resid, x0, bounds=([1.0, 0.0, 0.0, 0.0], [400.0, 0.95, 5000.0, 20000.0]),
                        diff_step=1e-3)
    r = resid(sol.x)
    return {"fields": dict(zip(CALIBRATED, map(float, sol.x))),
            "rms_log_error": math.sqrt(sum(v * v for v in r) / len(r)), "points": len(r)}


def markdown(summaries: list, fitted: dict | None, decode: list | None = None) -> str:
    out = ["| workload | role | candidates | analytic-only pick vs best | planner pick (BN, waves, "
           "pipe, splits) | pick vs measured best | pick's measured rank | best in model top-5 | "
           "Spearman | pick's rank among its neighbours |",
           "|---|---|---|---|---|---|---|---|---|---|"]
    for s in summaries:
        out.append(f"| {s['workload']} | {'calibration' if s['calibration'] else 'held out'} | "
                   f"{s['candidates']} | {s['analytic_pick']} {s['analytic_over_best']:+.1%} | "
                   f"{s['pick']} {s['pick_us']:.1f} us "
                   f"(modelled {s['pick_modeled_us']:.1f}) | {s['pick_over_best']:+.1%} "
                   f"(best {s['best']} {s['best_us']:.1f} us) | {s['pick_measured_rank']} | "
                   f"{'yes' if s['best_in_model_top5'] else 'no'} | {s['spearman']:.2f} | "
                   f"{s['pick_rank_in_neighbourhood']} of {s['neighbours'] + 1} |")
    if decode:
        out.append("")
        out.append("| decode workload | split counts | planner pick: splits, measured (modelled) | "
                   "modelled / measured | pick vs measured best | Spearman |")
        out.append("|---|---|---|---|---|---|")
        for s in decode:
            out.append(f"| {s['workload']} | {s['candidates']} | {s['pick']}: "
                       f"{s['pick_us']:.1f} us ({s['pick_modeled_us']:.1f}) | "
                       f"{s['pick_modeled_us'] / s['pick_us']:.3f} | {s['pick_over_best']:+.1%} "
                       f"(best {s['best']} splits, {s['best_us']:.1f} us) | "
                       f"{s['spearman']:.2f} |")
    if fitted:
        out.append("")
        out.append(f"Refit of the calibrated fields ({fitted['points']} points, rms log error "
                   f"{fitted['rms_log_error']:.3f}): " +
                   ", ".join(f"{k} = {v:.3g}" for k, v in fitted["fields"].items()))
    return "\n".join(out)


# ---------------------------------------------------------------- decode --
def time_decode(w, n, iters=10, reps=3) -> float:
    """Best-of-reps mean time (us) of back-to-back decode calls with n splits."""
    import torch
    from attn_inputs import BY_NAME, make_inputs
    name = w[0]
    if not hasattr(time_decode, "cache") or time_decode.cache[0] != name:
        time_decode.cache = None  # free the previous workload's 2 GiB first
        q, k, v = (t.cuda() for t in make_inputs(BY_NAME[name]))
        o = torch.empty((w[1], w[2], w[4]), dtype=torch.float32, device="cuda")
        time_decode.cache = (name, q, k, v, o)
    _, q, k, v, o = time_decode.cache
    for _ in range(3):
        pa.attn_decode(q, k, v, o=o, n_splits=n)
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(iters):
            pa.attn_decode(q, k, v, o=o, n_splits=n)
        b.record()
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b) / iters * 1e3)
    return best


def decode_summary(w, meas: dict) -> dict:
    """The split count the planner picks against every split count timed."""
    _, B, H, Skv, d = w
    model = {}
    for n in meas:
        model[n] = pa.parse_plan(pa.get_plan(pa.KIND_DECODE, B, H, 1, Skv, d,
                                             n_splits=n))["modeled_us"]
    pick = pa.parse_plan(pa.get_plan(pa.KIND_DECODE, B, H, 1, Skv, d))
    pn = pick["N_SPLITS"]
    best = min(meas, key=meas.get)
    ns = sorted(meas)
    return {"workload": w[0], "candidates": len(meas), "pick": pn, "pick_us": meas[pn],
            "pick_modeled_us": pick["modeled_us"], "best": best, "best_us": meas[best],
            "pick_over_best": meas[pn] / meas[best] - 1.0,
            "spearman": spearman([model[n] for n in ns], [meas[n] for n in ns]),
            "rows": [{"splits": n, "modeled_us": model[n], "measured_us": meas[n]} for n in ns]}


def decode_ablation(data: dict, load: bool) -> list:
    out = []
    for w in DECODE_WORKLOADS:
        _, B, H, Skv, d = w
        if not load:
            meas = {}
            for n in DECODE_SPLITS:
                plan = pa.parse_plan(pa.get_plan(pa.KIND_DECODE, B, H, 1, Skv, d, n_splits=n))
                if plan["N_SPLITS"] in meas:  # clamped to an already-timed count
                    continue
                meas[plan["N_SPLITS"]] = time_decode(w, n)
                print(f"{w[0]} splits={plan['N_SPLITS']} modelled {plan['modeled_us']:.1f} us "
                      f"measured {meas[plan['N_SPLITS']]:.1f} us", flush=True)
            data[w[0]] = meas
        if w[0] in data:
            out.append(decode_summary(w, data[w[0]]))
    time_decode.cache = None
    return out


# ------------------------------------------------------------------ GEMM --
# (M, N, K): squares across the paper's range and its skewed shapes
GEMM_SHAPES = [(256, 256, 256), (1024, 1024, 1024), (2048, 2048, 2048), (4096, 4096, 4096),
               (8192, 8192, 8192), (16384, 16384, 16384), (16384, 256, 2048), (256, 256, 2048),
               (16384, 256, 16384), (2048, 2048, 16384)]
GEMM_DOMAINS = ((64, 128, 256), (64, 128, 256), (32, 64), (0, 1, 2, 3),
                (1, 2, 3, 4, 6, 8))  # BM, BN, BK, pipe, K splits


def gemm_key(c: dict) -> tuple:
    return (c["BLOCK_M"], c["BLOCK_N"], c["BLOCK_K"], c["WAVES_M"], c["WAVES_N"], c["PIPE"],
            c.get("K_SPLITS", 1))


def time_gemm(shape, variant, reps=3) -> float:
    """Best-of-reps mean time (us) of back-to-back launches of one forced tile."""
    import torch
    from attn_inputs import random_bf16
    M, N, K = shape
    if not hasattr(time_gemm, "cache") or time_gemm.cache[0] != shape:
        a = random_bf16((M, K), 21).cuda()
        b = random_bf16((K, N), 22).cuda()
        c = torch.empty((M, N), dtype=torch.float32, device="cuda")
        time_gemm.cache = (shape, a, b, c)
    _, a, b, c = time_gemm.cache
    iters = 3 if M * N * K > 2 ** 40 else 10
    os.environ["ATTN_FORCE_GEMM"] = "bm=%d,bn=%d,bk=%d,wm=%d,wn=%d,pipe=%d,splits=%d" % variant
    try:
        for _ in range(3):
            pa.gemm(a, b, c)
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(iters):
                pa.gemm(a, b, c)
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) / iters * 1e3)
        return best
    finally:
        os.environ.pop("ATTN_FORCE_GEMM", None)


def gemm_neighbours(pick: tuple, feasible: set) -> list:
    """Feasible tiles whose BM, BN, BK, pipe and K split are each at most one
    legal step from the pick's (the paper's local block-size perturbation)."""
    out = []
    for c in feasible:
        steps = [abs(dom.index(x) - dom.index(y))
                 for dom, x, y in zip(GEMM_DOMAINS, (c[0], c[1], c[2], c[5], c[6]),
                                      (pick[0], pick[1], pick[2], pick[5], pick[6]))]
        if max(steps) <= 1 and c != pick:
            out.append(c)
    return sorted(out)


def gemm_summary(shape, cands: list, meas: dict) -> dict:
    M, N, K = shape
    flops = 2.0 * M * N * K
    rows = [(c["modeled_us"], meas[gemm_key(c)], gemm_key(c)) for c in cands
            if gemm_key(c) in meas]
    by_model = sorted(rows)
    by_meas = sorted(rows, key=lambda r: r[1])
    pick, best = by_model[0], by_meas[0]
    nb = gemm_neighbours(pick[2], {r[2] for r in rows})
    return {
        "shape": shape, "candidates": len(rows), "pick": pick[2], "pick_us": pick[1],
        "pick_tflops": flops / pick[1] / 1e6, "pick_modeled_tflops": flops / pick[0] / 1e6,
        "best": best[2], "best_us": best[1], "pick_over_best": pick[1] / best[1] - 1.0,
        "pick_measured_rank": [r[2] for r in by_meas].index(pick[2]) + 1,
        "spearman": spearman([r[0] for r in rows], [r[1] for r in rows]),
        "neighbours": len(nb),
        "pick_rank_in_neighbourhood": 1 + sum(meas[n] < pick[1] for n in nb),
    }


def gemm_markdown(summaries: list) -> str:
    out = ["| M, N, K | candidates | planner pick (BM, BN, BK, WM, WN, pipe) | measured TFLOP/s "
           "(modelled) | pick vs measured best | pick's measured rank | Spearman | pick's rank "
           "among its block-size neighbours |", "|---|---|---|---|---|---|---|---|"]
    for s in summaries:
        out.append(f"| {s['shape']} | {s['candidates']} | {s['pick']} | {s['pick_tflops']:.0f} "
                   f"({s['pick_modeled_tflops']:.0f}) | {s['pick_over_best']:+.1%} (best "
                   f"{s['best']}) | {s['pick_measured_rank']} | {s['spearman']:.2f} | "
                   f"{s['pick_rank_in_neighbourhood']} of {s['neighbours'] + 1} |")
    return "\n".join(out)


def main_gemm(a):
    data = {}
    if a.load:
        with open(a.load) as f:
            raw = json.load(f)
        data = {tuple(map(int, s.split(","))): {(tuple(map(int, k.split(","))) + (1,))[:7]: t
                                               for k, t in m.items()} for s, m in raw.items()}
    cands = {shape: pa.gemm_candidates(*shape) for shape in GEMM_SHAPES}
    if not a.load:
        for shape in GEMM_SHAPES:
            meas = {}
            for c in cands[shape]:
                meas[gemm_key(c)] = time_gemm(shape, gemm_key(c))
                print(f"{shape} {gemm_key(c)} modelled {c['modeled_us']:.1f} us measured "
                      f"{meas[gemm_key(c)]:.1f} us", flush=True)
            data[shape] = meas
    # saved before summarising, so a summary error loses no measurement
    if a.save:
        with open(a.save, "w") as f:
            json.dump({",".join(map(str, s)): {",".join(map(str, k)): t for k, t in m.items()}
                       for s, m in data.items()}, f, indent=1)
    summaries = [gemm_summary(shape, cands[shape], data[shape]) for shape in GEMM_SHAPES
                 if shape in data]
    text = gemm_markdown(summaries)
    print(text)
    if a.markdown:
        with open(a.markdown, "w") as f:
            f.write(text + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--save", help="write the measurements (JSON)")
    ap.add_argument("--load", help="reuse measurements (JSON) instead of timing")
    ap.add_argument("--fit", action="store_true", help="refit the calibrated description fields")
    ap.add_argument("--markdown", help="write the summary table here")
    ap.add_argument("--gemm", action="store_true",
                    help="the GEMM block-size ablation instead of the prefill one")
    ap.add_argument("--only-calibration", action="store_true",
                    help="time the calibration workloads only (for --fit)")
    ap.add_argument("--fit-out", help="write the refitted fields here (JSON)")
    a = ap.parse_args()
    import torch
    # torch's HIP runtime must initialise the device before this library's
    # first HIP call (the plan query below makes one)
    assert torch.cuda.is_available(), "the ablation needs a HIP device"
    if a.gemm:
        return main_gemm(a)
    data = {}
    if a.load:
        with open(a.load) as f:
            raw = json.load(f)
        # keys "bn,waves,pipe[,splits]" (measurements from before key splits: 1 split)
        data = {w: {(tuple(map(int, k.split(","))) + (1,))[:4]: t for k, t in m.items()}
                for w, m in raw.items() if w != "decode"}
    summaries = []
    workloads = [w for w in WORKLOADS if not a.only_calibration or w[0] in CALIBRATION]
    for w in workloads:
        cands = pa.fwd_candidates(*w[1:])
        if not a.load:
            meas = {}
            for c in cands:
                meas[key(c)] = time_variant(w, key(c))
                print(f"{w[0]} {key(c)} modelled {c['modeled_us']:.1f} us measured "
                      f"{meas[key(c)]:.1f} us", flush=True)
            data[w[0]] = meas
        if w[0] in data:
            summaries.append(summarise(w, cands, data[w[0]],
                                       pa.fwd_candidates(*w[1:], analytic_only=True)))
    decode_data = {}
    if a.load and "decode" in raw:
        decode_data = {w: {int(n): t for n, t in m.items()} for w, m in raw["decode"].items()}
    decode = None if a.only_calibration else decode_ablation(decode_data, bool(a.load))
    if a.save:
        out = {w: {",".join(map(str, k)): t for k, t in m.items()} for w, m in data.items()}
        out["decode"] = {w: {str(n): t for n, t in m.items()} for w, m in decode_data.items()}
        with open(a.save, "w") as f:
            json.dump(out, f, indent=1)
    fitted = fit(data) if a.fit else None
    if fitted and a.fit_out:
        with open(a.fit_out, "w") as f:
            json.dump(fitted, f, indent=1)
    text = markdown(summaries, fitted, decode)
    print(text)
    if a.markdown:
        with open(a.markdown, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()

"""Characterise the compiled prefill tile kernels once on a gfx950 device.

    python paper_2609_29219_amd/calibrate_primitives.py [--gemm] [--write [--out FILE]]
    python paper_2609_29219_amd/calibrate_primitives.py --device [FILE]

For each head dimension and masking mode, every valid tile variant (block
width, waves, pipeline knob) is timed on one calibration shape -- B2 H16
Sq = Skv = 4096, non-causal and causal, which is none of the benchmarked
workloads -- and its time is divided by the analytic model's time for it
(the model without these factors).  The ratio
is the variant's per-tile cost factor: the planner multiplies the modelled
tile cost by it.  This is the paper's primitive characterisation (its
latency model takes the cost of each primitive from isolated measurements,
collected once per architecture), applied to the compiled tile kernels; no
shape is tuned.  --write regenerates csrc/fwd_primitives.inc.  --gemm does the
same for the GEMM tile kernels (each B layout and pipe setting, alone on a CU
-- one tile per CU, K = 8192 -- and sharing CUs at M = N = K = 4096) into
csrc/gemm_primitives.inc.  --device runs the library's isolated
microbenchmarks instead (attn_measure_device: MFMA, fp32 VALU, v_exp_f32, LDS
read and HBM stream rates) and prints the device description as JSON (and
writes it to FILE); the planner's built-in gfx950 performance properties are
the values it measured on an MI355X.
"""
from __future__ import annotations

import argparse
import ctypes
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import paper_2609_29219_amd as pa  # noqa: E402

# B, H, Sq, Skv of the calibration shapes (disjoint from the benchmarked workloads)
SHAPES = {False: (2, 16, 4096, 4096), True: (2, 16, 4096, 4096)}
BNS, WAVES, PIPES = (32, 64, 128), (4, 8), (0, 1, 2, 3)
INC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "fwd_primitives.inc")


def time_variant(q, k, v, o, causal, bn, nw, pipe, iters=10, reps=3) -> float:
    import torch
    os.environ["ATTN_FORCE_PLAN"] = f"bn={bn},waves={nw},pipe={pipe}"
    try:
        for _ in range(3):
            pa.attn_fwd(q, k, v, o=o, causal=causal)
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(iters):
                pa.attn_fwd(q, k, v, o=o, causal=causal)
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) / iters * 1e3)
        return best
    finally:
        os.environ.pop("ATTN_FORCE_PLAN", None)


GEMM_SHAPE = (4096, 4096, 4096)
GEMM_INC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "gemm_primitives.inc")
# the planner's kGemmTiles order: (BM, BN, BK, WM, WN)
GEMM_TILES = [(64, 64, 64, 2, 2), (128, 128, 32, 2, 2), (128, 128, 64, 2, 2),
              (256, 128, 32, 2, 2), (256, 128, 64, 2, 2), (128, 256, 32, 2, 2),
              (128, 256, 64, 2, 2), (256, 256, 32, 2, 4), (256, 256, 64, 2, 4),
              (256, 256, 32, 2, 2), (256, 256, 64, 2, 2)]
GEMM_PIPES = 4  # pipe settings 0..3 (LDS slots - 1)


def time_gemm_tile(a, b, c, b_nk, tile, pipe) -> float:
    import torch
    os.environ["ATTN_FORCE_GEMM"] = "bm=%d,bn=%d,bk=%d,wm=%d,wn=%d" % tile + f",pipe={pipe}"
    try:
        for _ in range(3):
            pa.gemm(a, b, c, b_nk=b_nk)
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(10):
                pa.gemm(a, b, c, b_nk=b_nk)
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1) / 10 * 1e3)
        return best
    finally:
        os.environ.pop("ATTN_FORCE_GEMM", None)


def calibrate_gemm(write: bool, out: str) -> None:
    """Every valid GEMM tile kernel (both B layouts, every pipe), alone on a
    CU and sharing CUs (M = N = K = 4096).  Alone: one tile per CU (M = 16 BM,
    N = 16 BN, K = 8192), or, for a tile that only ever runs one workgroup
    per CU, two rounds of them (M = 32 BM): in a single round every
    workgroup starts at once and contends for the same panels, which large
    GEMMs (many rounds, desynchronised) do not see.  The candidates of a
    shape are timed in three interleaved passes, median per candidate, so
    drift of the clock under the power limit does not favour one of them."""
    import torch
    from attn_inputs import random_bf16
    desc = pa.DeviceDesc()
    pa.lib.attn_query_device(ctypes.byref(desc))
    side = int(round(desc.num_cus ** 0.5))
    table = {}
    for shared in (False, True):
        for b_nk in (False, True):
            for ti, tile in enumerate(GEMM_TILES):
                if shared:
                    M, N, K = GEMM_SHAPE
                else:
                    M, N, K = side * tile[0], (desc.num_cus // side) * tile[1], 8192
                    one_per_cu = [c["wg_per_cu"] == 1 for c in pa.gemm_candidates(
                        M, N, K, b_nk, device_footprint=True, analytic_only=True)
                        if (c["BLOCK_M"], c["BLOCK_N"], c["BLOCK_K"], c["WAVES_M"],
                            c["WAVES_N"]) == tile]
                    if one_per_cu and all(one_per_cu):
                        M *= 2
                # (unsplit K: the factor is the per-k-tile cost of the tile kernel)
                cands = [c for c in pa.gemm_candidates(M, N, K, b_nk, device_footprint=True,
                                                       analytic_only=True)
                         if (c["BLOCK_M"], c["BLOCK_N"], c["BLOCK_K"], c["WAVES_M"],
                             c["WAVES_N"]) == tile and c.get("K_SPLITS", 1) == 1
                         and (not shared or c["wg_per_cu"] >= 2)]
                if not cands:
                    continue  # (sharing: a tile that cannot share a CU has the alone setting only)
                a = random_bf16((M, K), 51).cuda()
                b = random_bf16((N, K) if b_nk else (K, N), 52).cuda()
                c = torch.empty((M, N), dtype=torch.float32, device="cuda")
                times = {cand["PIPE"]: [] for cand in cands}
                for _ in range(3):
                    for cand in cands:
                        times[cand["PIPE"]].append(time_gemm_tile(a, b, c, b_nk, tile, cand["PIPE"]))
                for cand in cands:
                    t = sorted(times[cand["PIPE"]])[1]
                    f = t / cand["modeled_us"]
                    table[(ti, b_nk, cand["PIPE"], shared)] = f
                    print(f"gemm {'shared' if shared else 'alone '} b_nk={int(b_nk)} {tile} "
                          f"pipe={cand['PIPE']} at {M}x{N}x{K}: measured {t:.1f} us, analytic "
                          f"{cand['modeled_us']:.1f} us, factor {f:.3f}", flush=True)
                del a, b, c
    if write:
        with open(GEMM_INC) as f:
            head = f.read().split("static const float")[0]
        rows = []
        for i in range(len(GEMM_TILES)):
            cells = ", ".join(
                "{" + ", ".join("{" + ", ".join(f"{table.get((i, b_nk, p, sh), 0.0):.4f}f"
                                                for sh in (False, True)) + "}"
                                for p in range(GEMM_PIPES)) + "}" for b_nk in (False, True))
            rows.append(f"    {{{cells}}},  // {GEMM_TILES[i]}")
        with open(out, "w") as f:
            f.write(head + f"static const float kGemmPrimScale[{len(GEMM_TILES)}][2]"
                    f"[{GEMM_PIPES}][2] = {{\n" +
                    "\n".join(rows) + "\n};\n")
        print(f"wrote {out}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--write", action="store_true", help="regenerate csrc/fwd_primitives.inc")
    ap.add_argument("--out", default=None, help="where --write puts the table")
    ap.add_argument("--gemm", action="store_true", help="the GEMM tile kernels instead")
    ap.add_argument("--device", nargs="?", const="", default=None, metavar="FILE",
                    help="measure the device description (microbenchmarks) instead")
    ap.add_argument("--fields", metavar="FILE",
                    help="JSON {'fields': {name: value}} (as plan_ablation.py --fit-out "
                         "writes) overriding description fields of the analytic model")
    a = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "characterisation needs a HIP device"
    if a.device is not None:
        import json
        text = json.dumps(pa.measure_device(), indent=1)
        print(text)
        if a.device:
            with open(a.device, "w") as f:
                f.write(text + "\n")
        return None
    if a.gemm:
        return calibrate_gemm(a.write, a.out or GEMM_INC)
    a.out = a.out or INC
    from attn_inputs import random_bf16
    desc = None
    if a.fields:
        import json
        desc = pa.DeviceDesc()
        pa.lib.attn_query_device(ctypes.byref(desc))
        with open(a.fields) as f:
            for name, val in json.load(f)["fields"].items():
                setattr(desc, name, float(val))
    table = {}
    for d in (64, 128):
        for causal in (False, True):
            B, H, Sq, Skv = SHAPES[causal]
            q = random_bf16((B, H, Sq, d), 41).cuda()
            k = random_bf16((B, H, Skv, d), 42).cuda()
            v = random_bf16((B, H, Skv, d), 43).cuda()
            o = torch.empty((B, H, Sq, d), dtype=torch.float32, device="cuda")
            for c in pa.fwd_candidates(B, H, Sq, Skv, d, causal, desc=desc,
                                       device_footprint=True, analytic_only=True):
                if c["KV_SPLITS"] != 1:
                    continue
                bn, nw, pipe = c["BLOCK_N"], c["WAVES"], c["PIPE"]
                t = time_variant(q, k, v, o, causal, bn, nw, pipe)
                table[(d, bn, nw, pipe, causal)] = t / c["modeled_us"]
                print(f"d={d} causal={int(causal)} ({bn}, {nw}, {pipe}): measured {t:.1f} us, "
                      f"analytic {c['modeled_us']:.1f} us, factor {t / c['modeled_us']:.3f}",
                      flush=True)
            del q, k, v, o
    if a.write:
        if a.out != INC:
            with open(INC) as f, open(a.out, "w") as g:
                g.write(f.read())
        write_inc(table, a.out)
        print(f"wrote {a.out}")


def write_inc(table: dict, path: str = INC) -> None:
    """The factor table as C: [d == 128][BN][waves][pipe][causal], 0 = none."""
    with open(path) as f:
        head = f.read().split("static const float")[0]
    dims = []
    for d in (64, 128):
        bns = []
        for bn in BNS:
            ws = []
            for nw in WAVES:
                ps = ", ".join("{" + ", ".join(f"{table.get((d, bn, nw, p, c), 0.0):.4f}f"
                                               for c in (False, True)) + "}" for p in PIPES)
                ws.append("{" + ps + "}")
            bns.append("{" + ", ".join(ws) + "}")
        dims.append(f"    {{  // d = {d}: BN 32, 64, 128\n     " + ",\n     ".join(bns) + "}")
    with open(path, "w") as f:
        f.write(head + "static const float kFwdPrimScale[2][3][2][4][2] = {\n" +
                ",\n".join(dims) + "};\n")


if __name__ == "__main__":
    main()

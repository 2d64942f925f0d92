"""Characterise the compiled prefill tile kernels once on a gfx950 device.

    python paper_2609_29219_amd/calibrate_primitives.py [--write [--out FILE]]

For each head dimension and masking mode, every valid tile variant (block
width, waves, pipeline knob) is timed on one calibration shape -- B1 H32
S8192 non-causal, B2 H16 S4096 causal -- and its time is divided by the
analytic model's time for it (the model without these factors).  The ratio
is the variant's per-tile cost factor: the planner multiplies the modelled
tile cost by it.  This is the paper's primitive characterisation (its
latency model takes the cost of each primitive from isolated measurements,
collected once per architecture), applied to the compiled tile kernels; no
shape is tuned.  --write regenerates csrc/fwd_primitives.inc.
"""
from __future__ import annotations

import argparse
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import paper_2609_29219_amd as pa  # noqa: E402

SHAPES = {False: (1, 32, 8192, 8192), True: (2, 16, 4096, 4096)}  # B, H, Sq, Skv
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--write", action="store_true", help="regenerate csrc/fwd_primitives.inc")
    ap.add_argument("--out", default=INC, help="where --write puts the table")
    a = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "characterisation needs a HIP device"
    from attn_inputs import random_bf16
    table = {}
    for d in (64, 128):
        for causal in (False, True):
            B, H, Sq, Skv = SHAPES[causal]
            q = random_bf16((B, H, Sq, d), 41).cuda()
            k = random_bf16((B, H, Skv, d), 42).cuda()
            v = random_bf16((B, H, Skv, d), 43).cuda()
            o = torch.empty((B, H, Sq, d), dtype=torch.float32, device="cuda")
            for c in pa.fwd_candidates(B, H, Sq, Skv, d, causal, device_footprint=True,
                                       analytic_only=True):
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

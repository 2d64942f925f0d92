"""Write tests/golden/oracle_small.json from the oracle (and nothing else).

Usage: python tests/golden/make_golden.py

The paper prints no attention values (its Flash Attention and Flash Decode
results are speedup bars in figures), so no fixture here is the paper's.
This file records the oracle's own output on small seeded inputs shaped like
each workload, as a regression guard on the oracle's arithmetic.  The oracle
itself is pinned by the checks in tests/oracle_pins.py.
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from attn_inputs import CONFIGS, make_inputs  # noqa: E402

CASES = [  # (config index, B, H, Sq, Skv, seed)
    (0, 1, 1, 256, 256, 1234),
    (1, 1, 2, 160, 160, 1235),
    (2, 1, 1, 96, 200, 1236),
    (3, 2, 2, 1, 300, 1237),
]


def main():
    out = {"source": "oracle/oracle_attn.c via oracle.attn; inputs from attn_inputs",
           "cases": []}
    for ci, B, H, Sq, Skv, seed in CASES:
        w = CONFIGS[ci].with_(B=B, H=H, Sq=Sq, Skv=Skv, seed=seed)
        q, k, v = make_inputs(w)
        if w.kind == "decode":
            o = oracle.attn(q.reshape(B, H, 1, w.d), k, v, B, H, 1, Skv, w.d, w.scale, False)
        else:
            o = oracle.attn(q, k, v, B, H, Sq, Skv, w.d, w.scale, w.causal)
        flat = o.reshape(-1)
        idx = np.random.default_rng(seed).choice(flat.size, size=12, replace=False)
        out["cases"].append({"config": ci, "B": B, "H": H, "Sq": Sq, "Skv": Skv, "seed": seed,
                             "index": [int(i) for i in idx],
                             "value": [float(x) for x in flat[idx]],
                             "abs_sum": float(np.abs(o).sum())})
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_small.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()

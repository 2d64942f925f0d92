"""Characterise the current device and print its description as JSON.

    python paper_2609_29219_amd/measure_device.py [out.json]

Runs the library's microbenchmarks (attn_measure_device) on device 0.  The
planner's built-in gfx950 performance properties are the values this wrote
on an MI355X.
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import paper_2609_29219_amd as pa  # noqa: E402

if __name__ == "__main__":
    desc = pa.measure_device()
    text = json.dumps(desc, indent=1)
    print(text)
    if len(sys.argv) > 1:
        with open(sys.argv[1], "w") as f:
            f.write(text + "\n")

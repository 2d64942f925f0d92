"""Build tests/c_abi/abi_check, a C++ caller of libattn.so's C ABI that uses
the HIP runtime alone (no Python, no torch).  Run by __graft_entry__.build()
after the library; the GPU test test_gpu_c_abi.py runs the binary."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_2609_29219_amd")
BIN = os.path.join(HERE, "abi_check")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build() -> str:
    cmd = [HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "abi_check.cpp"),
           "-L", PKG, "-lattn", "-Wl,-rpath,$ORIGIN/../../paper_2609_29219_amd",
           "-o", BIN + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"abi_check build failed:\n{r.stderr}")
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())

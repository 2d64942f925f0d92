"""Helpers for the GPU parity tests (tolerances, comparisons, case logging)."""
from __future__ import annotations

import os
import sys

import numpy as np
import torch

# Tolerances for bf16 inputs with fp32 accumulation, taken over all compared
# output elements in fp64.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def announce(msg: str) -> None:
    """Name the case on stdout before a GPU step (flushed)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def compare(got, want, what: str, max_abs: float = MAX_ABS, mean_abs: float = MEAN_ABS,
            rel_fro: float | None = None) -> dict:
    g = got.detach().cpu().double().numpy() if isinstance(got, torch.Tensor) else np.asarray(got)
    w = np.asarray(want, dtype=np.float64)
    assert g.shape == w.shape, f"{what}: shape {g.shape} vs {w.shape}"
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    err = np.abs(g - w)
    stats = {"max_abs": float(err.max()), "mean_abs": float(err.mean()),
             "rel_fro": float(np.linalg.norm(g - w) / max(np.linalg.norm(w), 1e-300))}
    assert stats["max_abs"] <= max_abs, f"{what}: max abs err {stats}"
    assert stats["mean_abs"] <= mean_abs, f"{what}: mean abs err {stats}"
    if rel_fro is not None:
        assert stats["rel_fro"] <= rel_fro, f"{what}: relative error {stats}"
    return stats


class forced_plan:
    """Context manager fixing the prefill tile (the ablation hook)."""

    def __init__(self, bn: int, waves: int, pipe: int):
        self.value = f"bn={bn},waves={waves},pipe={pipe}"

    def __enter__(self):
        self.old = os.environ.get("ATTN_FORCE_PLAN")
        os.environ["ATTN_FORCE_PLAN"] = self.value
        return self

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("ATTN_FORCE_PLAN", None)
        else:
            os.environ["ATTN_FORCE_PLAN"] = self.old

"""Seeded synthetic inputs for the attention workloads.

This module is shared by the tests, the benchmark and the smoke check.  It
draws random numbers and rounds them to bf16; it holds none of the attention
arithmetic, and it imports neither the oracle nor the HIP library.

The paper's Flash Attention / Flash Decode shapes live in figures whose data
is not in the text (Evaluation, "Flash Attention" and "Flash Decode"
paragraphs; the captions only name the axes B, L, N and B, N, L, D).  The five
workloads below stand in for them.  Recipe (identical for every config):
  * ``g = torch.Generator('cpu').manual_seed(1234 + index)``;
  * draw q, then k, then v as float32 ``randn``, one (b, h) slab at a time,
    in (b, h) row-major order;
  * multiply by ``input_scale`` (0.5 for the long-sequence config, else 1);
  * round to bf16 with round-to-nearest-even (``Tensor.to(torch.bfloat16)``).
The same bf16 host tensors feed the oracle (as uint16 bit patterns) and the
GPU (after ``.to('cuda')``).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    kind: str            # "fwd" (prefill) or "decode"
    B: int
    H: int
    Sq: int
    Skv: int
    d: int
    causal: bool
    input_scale: float
    seed: int

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(d), as the fp32 value both sides use."""
        return float(np.float32(1.0 / math.sqrt(self.d)))

    def allowed_pairs(self) -> int:
        """Number of (query, key) pairs inside the mask, over all (b, h)."""
        per_head = self.Sq * self.Skv
        if self.causal:
            off = self.Skv - self.Sq
            per_head = sum(min(i + off + 1, self.Skv) for i in range(self.Sq))
        return self.B * self.H * per_head

    def flops(self) -> int:
        """Algorithmic FLOP: 4*d per allowed (query, key) pair (QK^T and PV)."""
        return 4 * self.d * self.allowed_pairs()

    def hbm_bytes(self) -> int:
        """Algorithmic bytes: Q, K, V read once (bf16), O written once (fp32)."""
        q = self.B * self.H * self.Sq * self.d * 2
        kv = 2 * self.B * self.H * self.Skv * self.d * 2
        o = self.B * self.H * self.Sq * self.d * 4
        return q + kv + o

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five configurations, index k seeds the generator with 1234 + k.
CONFIGS = [
    Workload("single_head_s256_d64", "fwd", 1, 1, 256, 256, 64, False, 1.0, 1234),
    Workload("prefill_b4_h16_s2048_d128_causal", "fwd", 4, 16, 2048, 2048, 128, True, 1.0, 1235),
    Workload("prefill_b1_h32_s8192_d128", "fwd", 1, 32, 8192, 8192, 128, False, 0.5, 1236),
    Workload("decode_b16_h32_s8192_d128", "decode", 16, 32, 1, 8192, 128, False, 1.0, 1237),
    Workload("decode_b1_h32_s131072_d128", "decode", 1, 32, 1, 131072, 128, False, 1.0, 1238),
]

BY_NAME = {w.name: w for w in CONFIGS}


def _draw(g: torch.Generator, B: int, H: int, S: int, d: int, scale: float) -> torch.Tensor:
    out = torch.empty((B, H, S, d), dtype=torch.bfloat16)
    for b in range(B):
        for h in range(H):
            x = torch.randn((S, d), dtype=torch.float32, generator=g)
            if scale != 1.0:
                x.mul_(scale)
            out[b, h].copy_(x.to(torch.bfloat16))
    return out


def make_inputs(w: Workload, seed: int | None = None):
    """Return (q, k, v) as CPU bf16 tensors.

    fwd: q [B,H,Sq,d]; decode: q [B,H,d].  k, v: [B,H,Skv,d].
    """
    g = torch.Generator("cpu").manual_seed(w.seed if seed is None else seed)
    q = _draw(g, w.B, w.H, w.Sq, w.d, w.input_scale)
    k = _draw(g, w.B, w.H, w.Skv, w.d, w.input_scale)
    v = _draw(g, w.B, w.H, w.Skv, w.d, w.input_scale)
    if w.kind == "decode":
        q = q.reshape(w.B, w.H, w.d)
    return q, k, v


def random_bf16(shape, seed: int, scale: float = 1.0) -> torch.Tensor:
    """Generic seeded N(0, scale^2) tensor rounded to bf16 (CPU)."""
    g = torch.Generator("cpu").manual_seed(seed)
    x = torch.randn(shape, dtype=torch.float32, generator=g)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(torch.bfloat16)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """uint16 bit patterns of a CPU bf16 tensor (no copy of values changed)."""
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def from_float(a) -> torch.Tensor:
    """Round a float array to a bf16 tensor (RNE)."""
    return torch.as_tensor(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)

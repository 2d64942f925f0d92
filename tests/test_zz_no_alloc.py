"""GPU test of attn_decode_noalloc, the decode entry point that allocates
nothing (its split partials live in the library's static device scratch).

Each case calls it through the C ABI and compares its output with the
allocating entry point attn_decode_ex on the same inputs and split count
(same plan and kernels, so the same bits), and both with the fp64 oracle at
the parity tolerance.  Calls come in pairs, the second on a smaller input, so
the second reuses scratch that still holds the first call's partials.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from attn_inputs import random_bf16
from tests.gpu_common import announce, compare

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


def _case(pa, B, Hq, Hkv, Skv, d, n_splits, seed):
    q = random_bf16((B, Hq, d), seed)
    k = random_bf16((B, Hkv, Skv, d), seed + 1)
    v = random_bf16((B, Hkv, Skv, d), seed + 2)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    announce(f"attn_decode_noalloc B={B} Hq={Hq} Hkv={Hkv} Skv={Skv} d={d} n_splits={n_splits} "
             f"({pa.decode_workspace_bytes(B, Hq, Hkv, Skv, d, n_splits)} bytes of partials)")
    o = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_decode_noalloc(qd, kd, vd, o, n_splits=n_splits, lse=lse)
    want_o, want_lse = pa.attn_decode(qd, kd, vd, n_splits=n_splits, return_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o, want_o), "differs from attn_decode_ex with the library workspace"
    assert torch.equal(lse, want_lse)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    ref, ref_lse = oracle.attn_gqa(q.reshape(B, Hq, 1, d).contiguous(), k, v, B, Hq, Hkv, 1, Skv,
                                   d, sc, False)
    compare(o, ref.reshape(B, Hq, d), f"noalloc decode {B, Hq, Hkv, Skv, d, n_splits}")
    if Hq // Hkv < 4:
        # the VALU kernel sums unrounded fp32 probabilities: fp32-accurate lse
        compare(lse, ref_lse.reshape(B, Hq), "noalloc decode lse", max_abs=1e-4, mean_abs=2e-5)
    else:
        # the matrix-core kernel sums the bf16-rounded probabilities (each
        # within 2^-8 relative of exact), as prefill does
        compare(lse, ref_lse.reshape(B, Hq), "noalloc decode lse", max_abs=5e-3, mean_abs=1e-3)


@pytest.mark.parametrize("pair", [
    # (larger call, then a smaller one) -- B, Hq, Hkv, Skv, d, n_splits
    ((16, 32, 32, 2048, 128, 4), (2, 4, 4, 300, 128, 3)),      # VALU kernel, partials in the scratch
    ((4, 32, 4, 5000, 128, 16), (1, 8, 1, 777, 128, 5)),       # grouped heads, matrix cores
    ((3, 8, 8, 4099, 64, 64), (1, 2, 2, 17, 64, 0)),           # d = 64, many splits; then one
                                                               # split, which bypasses the scratch
], ids=["mha", "gqa_mfma", "d64"])
def test_noalloc_matches_allocating_decode(pa, pair):
    for i, (B, Hq, Hkv, Skv, d, n) in enumerate(pair):
        _case(pa, B, Hq, Hkv, Skv, d, n, seed=4000 + 10 * i + Skv)


def test_noalloc_rejects_calls_over_the_scratch(pa):
    # 64 x 64 rows x 8 splits x (128 + 2) floats = 17,039,360 bytes > 16 MiB
    B, H, Skv, d, n = 64, 64, 64, 128, 8
    assert B * H * n * (d + 2) * 4 > pa.NOALLOC_SCRATCH_BYTES
    assert pa.decode_workspace_bytes(B, H, H, Skv, d, n) > pa.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, H, d), dtype=torch.bfloat16, device=DEV)
    kv = torch.zeros((B, H, Skv, d), dtype=torch.bfloat16, device=DEV)
    o = torch.full((B, H, d), 7.0, dtype=torch.float32, device=DEV)
    announce("attn_decode_noalloc over the scratch limit")
    with pytest.raises(pa.AttnError) as e:
        pa.attn_decode_noalloc(q, kv, kv, o, n_splits=n)
    assert e.value.code == pa.ATTN_ENOMEM
    assert "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (o == 7.0).all(), "a rejected call launched work"
    # one split less fits, and runs
    o2 = pa.attn_decode_noalloc(q, kv, kv, torch.empty_like(o), n_splits=7)
    torch.cuda.synchronize()
    assert torch.isfinite(o2).all()

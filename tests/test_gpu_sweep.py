"""GPU parity over a seeded random sweep of the public calls' input space.

Each case draws batch, query and key/value heads (grouped-query included),
sequence lengths (log-uniform, so ragged tails of every size and lengths below
one tile occur), head dimension, causality, scale, input magnitude, output
dtype, log-sum-exp and, for decode, the split count, then compares every
output element of the planned call (whatever tile, schedule and key split the
planner picks for that shape) with the fp64 oracle on the same bf16 inputs.
The draws are fixed by the seed, so a failing case names a reproducible shape.
Tolerances as the other parity tests: outputs max-abs 2e-2, mean-abs 2e-3; the
log-sum-exp within the bf16-normaliser bound (max-abs 5e-3, mean-abs 1e-3).
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
LSE_MAX_ABS = 5e-3
LSE_MEAN_ABS = 1e-3


def _log_uniform(g, lo, hi):
    return int(round(math.exp(g.uniform(math.log(lo), math.log(hi)))))


def _prefill_cases(n, seed=20261202):
    g = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(g.integers(1, 4))
        Hkv = int(g.choice([1, 2, 3, 4]))
        Hq = Hkv * int(g.choice([1, 1, 2, 3, 4, 8]))
        if B * Hq > 24:  # bound the oracle's work: no grouping, then fewer batches
            Hq = Hkv
            B = min(B, 24 // Hq)
        d = int(g.choice([64, 128]))
        causal = bool(g.integers(0, 2))
        Sq = _log_uniform(g, 1, 1100)
        Skv = Sq + _log_uniform(g, 1, 1000) - 1 if causal else _log_uniform(g, 1, 2100)
        scale = float(np.float32(1.0 / math.sqrt(d) * g.choice([1.0, 0.5, 2.0])))
        mag = float(g.choice([1.0, 0.5]))
        out = "bf16" if g.integers(0, 2) else "fp32"
        lse = bool(g.integers(0, 2))
        cases.append((i, B, Hq, Hkv, Sq, Skv, d, causal, scale, mag, out, lse))
    return cases


def _decode_cases(n, seed=20261203):
    g = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        B = int(g.integers(1, 5))
        Hkv = int(g.choice([1, 2, 4, 8]))
        Hq = Hkv * int(g.choice([1, 2, 3, 4, 6, 8, 16]))
        Hq = min(Hq, 64 // Hkv * Hkv)
        d = int(g.choice([64, 128]))
        Skv = _log_uniform(g, 1, 20000)
        n_splits = 0 if g.integers(0, 2) else int(g.integers(1, min(Skv, 64) + 1))
        lse = bool(g.integers(0, 2))
        cases.append((i, B, Hq, Hkv, Skv, d, n_splits, lse))
    return cases


PREFILL = _prefill_cases(64)
DECODE = _decode_cases(32)


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


@pytest.mark.parametrize("case", PREFILL, ids=[
    f"{c[0]}-B{c[1]}-Hq{c[2]}-Hkv{c[3]}-Sq{c[4]}-Skv{c[5]}-d{c[6]}-{'causal' if c[7] else 'full'}"
    for c in PREFILL])
def test_fwd_sweep(pa, case):
    i, B, Hq, Hkv, Sq, Skv, d, causal, scale, mag, out, want_lse = case
    q = random_bf16((B, Hq, Sq, d), 3000 + 3 * i, scale=mag)
    k = random_bf16((B, Hkv, Skv, d), 3001 + 3 * i, scale=mag)
    v = random_bf16((B, Hkv, Skv, d), 3002 + 3 * i, scale=mag)
    dt = torch.bfloat16 if out == "bf16" else torch.float32
    announce(f"sweep attn_fwd_ex {case}")
    res = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=scale, causal=causal,
                      out_dtype=dt, return_lse=want_lse)
    torch.cuda.synchronize()
    o, lse = res if want_lse else (res, None)
    assert o.dtype == dt
    ref, ref_lse = oracle.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, scale, causal)
    compare(o.float(), ref, f"sweep fwd {case}")
    if want_lse:
        compare(lse, ref_lse, f"sweep fwd lse {case}", max_abs=LSE_MAX_ABS,
                mean_abs=LSE_MEAN_ABS)


@pytest.mark.parametrize("case", DECODE, ids=[
    f"{c[0]}-B{c[1]}-Hq{c[2]}-Hkv{c[3]}-Skv{c[4]}-d{c[5]}-n{c[6]}" for c in DECODE])
def test_decode_sweep(pa, case):
    i, B, Hq, Hkv, Skv, d, n_splits, want_lse = case
    q = random_bf16((B, Hq, d), 4000 + 3 * i)
    k = random_bf16((B, Hkv, Skv, d), 4001 + 3 * i)
    v = random_bf16((B, Hkv, Skv, d), 4002 + 3 * i)
    announce(f"sweep attn_decode_ex {case}")
    res = pa.attn_decode(q.to(DEV), k.to(DEV), v.to(DEV), n_splits=n_splits,
                         return_lse=want_lse)
    torch.cuda.synchronize()
    o, lse = res if want_lse else (res, None)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    ref, ref_lse = oracle.attn_gqa(q.reshape(B, Hq, 1, d).contiguous(), k, v, B, Hq, Hkv, 1,
                                   Skv, d, sc, False)
    compare(o, ref.reshape(B, Hq, d), f"sweep decode {case}")
    if want_lse:
        compare(lse, ref_lse.reshape(B, Hq), f"sweep decode lse {case}", max_abs=LSE_MAX_ABS,
                mean_abs=LSE_MEAN_ABS)

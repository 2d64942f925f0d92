"""GPU parity of the path's variants (through the C ABI) against the fp64 oracle.

Grouped-query heads (prefill and decode), bf16 output, the row log-sum-exp,
a caller-provided decode workspace, and prefill with split key ranges.  Inputs are seeded bf16 N(0,1).
Tolerances: outputs as the main parity tests (max-abs 2e-2, mean-abs 2e-3);
the log-sum-exp within 5e-3 (the kernel's normaliser sums bf16-rounded
probabilities, each within a relative 2^-8 of its exact value, so log l is
within 2^-8 = 3.9e-3 of exact, plus fp32 accumulation of the scores).
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from attn_inputs import random_bf16
from tests.gpu_common import announce, compare, forced_plan

pytestmark = pytest.mark.gpu

DEV = "cuda"
LSE_MAX_ABS = 5e-3
LSE_MEAN_ABS = 1e-3


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


def _qkv(B, Hq, Hkv, Sq, Skv, d, seed):
    return (random_bf16((B, Hq, Sq, d), seed), random_bf16((B, Hkv, Skv, d), seed + 1),
            random_bf16((B, Hkv, Skv, d), seed + 2))


GQA_SHAPES = [  # B, Hq, Hkv, Sq, Skv, d, causal
    (2, 4, 2, 77, 130, 128, False),
    (1, 8, 2, 200, 200, 128, True),
    (1, 6, 1, 65, 300, 64, False),
    (2, 8, 8, 130, 130, 64, True),
    (1, 16, 2, 33, 257, 128, True),
]


@pytest.mark.parametrize("shape", GQA_SHAPES, ids=[str(s) for s in GQA_SHAPES])
def test_fwd_gqa_lse(pa, shape):
    B, Hq, Hkv, Sq, Skv, d, causal = shape
    q, k, v = _qkv(B, Hq, Hkv, Sq, Skv, d, 700 + Hq + Sq)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    announce(f"attn_fwd_ex gqa {shape}")
    o, lse = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, causal=causal,
                         return_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, sc, causal)
    compare(o, ref, f"gqa out {shape}")
    compare(lse, ref_lse, f"gqa lse {shape}", max_abs=LSE_MAX_ABS, mean_abs=LSE_MEAN_ABS)


@pytest.mark.parametrize("variant", [(64, 8, 1), (128, 8, 1), (64, 4, 0), (64, 8, 2), (64, 8, 3),
                                     (32, 4, 3)])
def test_fwd_gqa_every_schedule(pa, variant):
    B, Hq, Hkv, Sq, Skv, d = 1, 8, 2, 290, 290, 128
    q, k, v = _qkv(B, Hq, Hkv, Sq, Skv, d, 800)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    with forced_plan(*variant):
        for causal in (False, True):
            announce(f"attn_fwd_ex gqa variant {variant} causal={causal}")
            o, lse = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, causal=causal,
                                 return_lse=True)
            torch.cuda.synchronize()
            ref, ref_lse = oracle.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, sc, causal)
            compare(o, ref, f"variant {variant}")
            compare(lse, ref_lse, f"variant {variant} lse", max_abs=LSE_MAX_ABS,
                    mean_abs=LSE_MEAN_ABS)


@pytest.mark.parametrize("causal", [False, True])
def test_fwd_bf16_output_is_the_rounded_fp32_output(pa, causal):
    B, H, Sq, Skv, d = 2, 3, 150, 150, 128
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 900)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    announce(f"attn_fwd_ex bf16 output causal={causal}")
    o32 = pa.attn_fwd(qd, kd, vd, causal=causal)
    o16 = pa.attn_fwd(qd, kd, vd, causal=causal, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert o16.dtype == torch.bfloat16
    # same arithmetic, then round to nearest even: bit-exact
    assert torch.equal(o16.cpu(), o32.cpu().to(torch.bfloat16))
    ref = oracle.attn(q, k, v, B, H, Sq, Skv, d, float(np.float32(1 / math.sqrt(d))), causal)
    compare(o16.float(), ref, "bf16 output")


CAUSAL_SCHEDULES = [(32, 4, 0), (32, 8, 1), (64, 4, 1), (64, 8, 1), (32, 4, 3), (64, 8, 3),
                    (128, 8, 0), (64, 8, 2)]


@pytest.mark.parametrize("variant", CAUSAL_SCHEDULES, ids=[str(v) for v in CAUSAL_SCHEDULES])
@pytest.mark.parametrize("d", [64, 128])
def test_fwd_causal_rows_stored_early_every_schedule(pa, variant, d):
    # A causal wave whose last key tile comes before its q-tile's last one
    # stores its rows straight from registers while the other waves still
    # compute.  Ragged Sq < Skv (the diagonal is offset), and several q-tiles
    # so that workgroups run two passes; fp32 and bf16 rows and the LSE.
    B, H, Sq, Skv = 1, 3, 600, 633
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 950 + d)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    with forced_plan(*variant):
        announce(f"attn_fwd_ex causal early stores {variant} d={d}")
        o, lse = pa.attn_fwd(qd, kd, vd, scale=sc, causal=True, return_lse=True)
        o16 = pa.attn_fwd(qd, kd, vd, scale=sc, causal=True, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.attn_gqa(q, k, v, B, H, H, Sq, Skv, d, sc, True)
    compare(o, ref, f"causal {variant} d={d}")
    compare(lse, ref_lse, f"causal {variant} d={d} lse", max_abs=LSE_MAX_ABS,
            mean_abs=LSE_MEAN_ABS)
    assert torch.equal(o16.cpu(), o.cpu().to(torch.bfloat16))


def test_fwd_lse_special_cases(pa):
    # Q = 0: every allowed score is 0, lse = log(#allowed keys) (exact up to fp32)
    B, H, Sq, Skv, d = 1, 2, 100, 160, 64
    k, v = random_bf16((B, H, Skv, d), 950), random_bf16((B, H, Skv, d), 951)
    q0 = torch.zeros((B, H, Sq, d), dtype=torch.bfloat16)
    announce("attn_fwd_ex lse with Q = 0")
    for causal in (False, True):
        _, lse = pa.attn_fwd(q0.to(DEV), k.to(DEV), v.to(DEV), causal=causal, return_lse=True)
        torch.cuda.synchronize()
        n = np.full(Sq, Skv) if not causal else np.arange(Sq) + (Skv - Sq) + 1
        np.testing.assert_allclose(lse.cpu().double().numpy(),
                                   np.broadcast_to(np.log(n), (B, H, Sq)), atol=2e-6, rtol=0)


def test_fwd_ex_rejects_before_launch(pa):
    q = torch.zeros((1, 4, 8, 64), dtype=torch.bfloat16, device=DEV)
    k = torch.zeros((1, 3, 8, 64), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:
        pa.attn_fwd(q, k, k)  # 3 key/value heads do not divide 4 query heads
    assert e.value.code == pa.ATTN_EINVAL


DECODE_GQA = [  # B, Hq, Hkv, Skv, d, n_splits  (group >= 4: the matrix-core kernel)
    (2, 8, 2, 1000, 128, 0),
    (1, 32, 4, 4096, 128, 0),
    (3, 6, 2, 777, 64, 5),
    (1, 16, 1, 2049, 128, 0),
    (2, 12, 4, 300, 128, 3),
    (1, 32, 2, 8192, 64, 0),
    (2, 32, 1, 1500, 128, 0),   # MQA: two query blocks of 16
    (1, 48, 2, 700, 128, 4),    # group 24: a full and a partial query block
    (3, 8, 2, 33, 128, 0),      # fewer keys than one 32-key step per wave
    (2, 20, 4, 1, 64, 0),       # a single key
    (1, 64, 8, 65536, 128, 0),  # long context, group 8
    (2, 8, 2, 1000, 128, 1),    # one split: the matrix-core kernel writes o and lse itself
    (3, 6, 2, 777, 64, 1),      # one split, the VALU kernel (group 3)
]


@pytest.mark.parametrize("shape", DECODE_GQA, ids=[str(s) for s in DECODE_GQA])
def test_decode_gqa_lse(pa, shape):
    B, Hq, Hkv, Skv, d, n = shape
    q = random_bf16((B, Hq, d), 1000 + Hq)
    k, v = random_bf16((B, Hkv, Skv, d), 1001 + Hq), random_bf16((B, Hkv, Skv, d), 1002 + Hq)
    announce(f"attn_decode_ex gqa {shape}")
    o, lse = pa.attn_decode(q.to(DEV), k.to(DEV), v.to(DEV), n_splits=n, return_lse=True)
    torch.cuda.synchronize()
    sc = float(np.float32(1.0 / math.sqrt(d)))
    ref, ref_lse = oracle.attn_gqa(q.reshape(B, Hq, 1, d).contiguous(), k, v, B, Hq, Hkv, 1, Skv,
                                   d, sc, False)
    compare(o, ref.reshape(B, Hq, d), f"decode gqa {shape}")
    if Hq // Hkv < 4:
        # the VALU kernel sums unrounded fp32 probabilities: fp32-accurate lse
        compare(lse, ref_lse.reshape(B, Hq), f"decode gqa lse {shape}", max_abs=1e-4,
                mean_abs=2e-5)
    else:
        # the matrix-core kernel sums the bf16-rounded probabilities (as prefill)
        compare(lse, ref_lse.reshape(B, Hq), f"decode gqa lse {shape}", max_abs=LSE_MAX_ABS,
                mean_abs=LSE_MEAN_ABS)


@pytest.mark.parametrize("d", [64, 128])
def test_decode_gqa_closed_forms(pa, d):
    # matrix-core decode: identical V rows give that row exactly (the weights
    # are an exact convex combination); Q = 0 gives the column mean of V and
    # lse = log(Skv)
    B, Hq, Hkv, Skv = 2, 16, 2, 777
    q = random_bf16((B, Hq, d), 1600)
    k = random_bf16((B, Hkv, Skv, d), 1601)
    row = random_bf16((B, Hkv, 1, d), 1602)
    v_same = row.expand(B, Hkv, Skv, d).contiguous()
    announce(f"attn_decode_ex gqa closed forms d={d}")
    o = pa.attn_decode(q.to(DEV), k.to(DEV), v_same.to(DEV))
    v = random_bf16((B, Hkv, Skv, d), 1603)
    o0, lse0 = pa.attn_decode(torch.zeros_like(q).to(DEV), k.to(DEV), v.to(DEV), return_lse=True)
    torch.cuda.synchronize()
    want = row.float().repeat_interleave(Hq // Hkv, dim=1).reshape(B, Hq, d)
    np.testing.assert_allclose(o.cpu().double().numpy(), want.double().numpy(), atol=2e-6,
                               rtol=1e-6)
    mean = v.double().mean(dim=2).repeat_interleave(Hq // Hkv, dim=1)
    compare(o0, mean.numpy(), "Q = 0 gives the mean of V", max_abs=2e-3, mean_abs=2e-4)
    np.testing.assert_allclose(lse0.cpu().double().numpy(), math.log(Skv), atol=2e-6, rtol=0)


def test_decode_gqa_split_invariance(pa):
    B, Hq, Hkv, Skv, d = 1, 16, 2, 5000, 128
    q = random_bf16((B, Hq, d), 1700).to(DEV)
    k = random_bf16((B, Hkv, Skv, d), 1701).to(DEV)
    v = random_bf16((B, Hkv, Skv, d), 1702).to(DEV)
    announce("attn_decode_ex gqa split counts")
    outs = {n: pa.attn_decode(q, k, v, n_splits=n) for n in (1, 3, 16, 40)}
    torch.cuda.synchronize()
    ref, _ = oracle.attn_gqa(q.cpu().reshape(B, Hq, 1, d).contiguous(), k.cpu(), v.cpu(), B, Hq,
                             Hkv, 1, Skv, d, float(np.float32(1.0 / math.sqrt(d))), False)
    for n, o in outs.items():
        compare(o, ref.reshape(B, Hq, d), f"splits {n} vs oracle")
        # the splits change only which reference max each probability is rounded against
        compare(o, outs[1].cpu().double().numpy(), f"splits {n} vs 1", max_abs=2e-3, mean_abs=2e-4)


def test_decode_caller_workspace(pa):
    B, Hq, Hkv, Skv, d = 2, 8, 2, 3000, 128
    q = random_bf16((B, Hq, d), 1100).to(DEV)
    k, v = random_bf16((B, Hkv, Skv, d), 1101).to(DEV), random_bf16((B, Hkv, Skv, d), 1102).to(DEV)
    for n in (0, 7):
        need = pa.decode_workspace_bytes(B, Hq, Hkv, Skv, d, n)
        announce(f"attn_decode_ex caller workspace n={n} bytes={need}")
        assert need > 0
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        a = pa.attn_decode(q, k, v, n_splits=n)
        b = pa.attn_decode(q, k, v, n_splits=n, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(a.cpu(), b.cpu()), "caller workspace changes the result"
        small = torch.empty(need - 16, dtype=torch.uint8, device=DEV)
        with pytest.raises(pa.AttnError) as e:
            pa.attn_decode(q, k, v, n_splits=n, workspace=small)
        assert e.value.code == pa.ATTN_EINVAL


# ---------------------------------------------------------------- key splits
class forced_split_plan(forced_plan):
    def __init__(self, bn: int, waves: int, pipe: int, splits: int):
        super().__init__(bn, waves, pipe)
        self.value += f",splits={splits}"


SPLIT_VARIANTS = [(32, 4, 0, 3), (32, 8, 3, 5), (64, 4, 1, 2), (64, 8, 3, 4), (64, 8, 1, 6),
                  (128, 8, 1, 3), (128, 4, 0, 2)]


@pytest.mark.parametrize("variant", SPLIT_VARIANTS, ids=[str(v) for v in SPLIT_VARIANTS])
def test_fwd_key_splits_every_schedule(pa, variant):
    # ragged query tail, key count that leaves a short last split, grouped heads
    B, Hq, Hkv, Sq, Skv = 2, 4, 2, 77, 1000
    for d in (64, 128):
        q, k, v = _qkv(B, Hq, Hkv, Sq, Skv, d, 1200 + d)
        sc = float(np.float32(1.0 / math.sqrt(d)))
        announce(f"attn_fwd_ex key splits {variant} d={d}")
        with forced_split_plan(*variant):
            o, lse = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, return_lse=True)
            o16 = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc,
                              out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        ref, ref_lse = oracle.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, sc, False)
        compare(o, ref, f"splits {variant} d={d}")
        compare(o16.float(), ref, f"splits {variant} d={d} bf16")
        assert torch.equal(o16.cpu(), o.cpu().to(torch.bfloat16))
        compare(lse, ref_lse, f"splits {variant} d={d} lse", max_abs=LSE_MAX_ABS,
                mean_abs=LSE_MEAN_ABS)


def test_fwd_key_splits_one_key_in_last_split(pa):
    # Skv = 2*64 + 1 with 3 splits of 64 keys: the last split holds one key
    B, H, Sq, Skv, d = 1, 3, 130, 129, 128
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 1300)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    announce("attn_fwd_ex key splits, one-key split")
    with forced_split_plan(64, 8, 1, 3):
        o = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc)
    torch.cuda.synchronize()
    compare(o, oracle.attn(q, k, v, B, H, Sq, Skv, d, sc, False), "one-key split")


@pytest.mark.parametrize("variant", [(64, 8, 3, 256), (128, 4, 1, 96), (32, 8, 1, 192)],
                         ids=["64x8x3_256", "128x4x1_96", "32x8x1_192"])
def test_fwd_many_key_splits(pa, variant):
    # more splits than the 32 the combine saw before: one q-tile of a few
    # queries against a long key range, the last split short
    bn, waves, pipe, n = variant
    B, H, Sq, d = 1, 2, 40, 128
    Skv = n * 2 * bn - bn // 2  # chunk 2*bn, every split non-empty, the last half full
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 1350 + n)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    announce(f"attn_fwd_ex many key splits {variant} Skv={Skv}")
    with forced_split_plan(bn, waves, pipe, n):
        o, lse = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, return_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.attn_gqa(q, k, v, B, H, H, Sq, Skv, d, sc, False)
    compare(o, ref, f"{n} splits", rel_fro=1e-2)
    compare(lse, ref_lse, f"{n} splits lse", max_abs=LSE_MAX_ABS, mean_abs=LSE_MEAN_ABS)


def test_fwd_key_splits_chosen_by_the_planner(pa):
    # few heads and queries against many keys: the planner splits the keys
    B, H, Sq, Skv, d = 1, 2, 256, 12000, 128
    plan = pa.parse_plan(pa.get_plan(pa.KIND_FWD, B, H, Sq, Skv, d, False))
    announce(f"attn_fwd planner split {plan}")
    assert plan["KV_SPLITS"] > 1, plan
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 1400)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    o, lse = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, return_lse=True)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.attn_gqa(q, k, v, B, H, H, Sq, Skv, d, sc, False)
    compare(o, ref, "planner split")
    compare(lse, ref_lse, "planner split lse", max_abs=LSE_MAX_ABS, mean_abs=LSE_MEAN_ABS)


def test_fwd_key_splits_after_decode_share_the_workspace(pa):
    # decode and split prefill on one stream reuse the per-stream workspace
    B, H, Sq, Skv, d = 1, 2, 64, 5000, 64
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 1500)
    qd = random_bf16((B, H, d), 1501)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    announce("split prefill interleaved with decode")
    kd, vd = k.to(DEV), v.to(DEV)
    with forced_split_plan(64, 4, 1, 6):
        outs = []
        for _ in range(3):
            outs.append(pa.attn_fwd(q.to(DEV), kd, vd, scale=sc))
            dec = pa.attn_decode(qd.to(DEV), kd, vd)
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.cpu(), outs[0].cpu())
    compare(outs[0], oracle.attn(q, k, v, B, H, Sq, Skv, d, sc, False), "split prefill")
    ref_d = oracle.attn(qd.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc, False)
    compare(dec, ref_d.reshape(B, H, d), "decode between")


def test_two_streams_keep_separate_workspaces(pa):
    # decode on one stream and split-key prefill on another, issued alternately
    # so that both are in flight together: each stream's partials live in its
    # own workspace, so neither result is disturbed by the other
    B, H, Sq, Skv, d = 2, 4, 96, 3000, 128
    q, k, v = _qkv(B, H, H, Sq, Skv, d, 1600)
    qd = random_bf16((B, H, d), 1603)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    qg, kg, vg, qdg = q.to(DEV), k.to(DEV), v.to(DEV), qd.to(DEV)
    torch.cuda.synchronize()
    s_dec, s_fwd = torch.cuda.Stream(), torch.cuda.Stream()
    announce("decode and split prefill on two streams")
    decs, fwds = [], []
    with forced_split_plan(64, 4, 1, 8):
        for _ in range(4):
            with torch.cuda.stream(s_dec):
                decs.append(pa.attn_decode(qdg, kg, vg, n_splits=12))
            with torch.cuda.stream(s_fwd):
                fwds.append(pa.attn_fwd(qg, kg, vg, scale=sc))
    torch.cuda.synchronize()
    for o in decs[1:]:
        assert torch.equal(o.cpu(), decs[0].cpu())
    for o in fwds[1:]:
        assert torch.equal(o.cpu(), fwds[0].cpu())
    compare(fwds[0], oracle.attn(q, k, v, B, H, Sq, Skv, d, sc, False), "split prefill stream")
    ref_d = oracle.attn(qd.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc, False)
    compare(decs[0], ref_d.reshape(B, H, d), "decode stream")


def test_fwd_key_splits_rejected_for_causal(pa):
    q = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16, device=DEV)
    with forced_split_plan(64, 8, 1, 2):
        with pytest.raises(pa.AttnError) as e:
            pa.attn_fwd(q, q, q, causal=True)
    assert e.value.code == pa.ATTN_EINVAL

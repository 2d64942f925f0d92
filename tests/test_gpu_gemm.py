"""GPU parity of the GEMM (C = A B, through the C ABI) against the fp64 oracle.

Tolerance from the arithmetic: bf16 x bf16 products are exact in fp32, and
the MFMA path sums them in fp32 in blocks (16 products per 32x32x16 MFMA,
then one accumulator update per 16 values of k; the 16x16x32 MFMA of the
hand-scheduled kernel gave bit-identical sums at 8192^3, consistent with the
same 16-product blocks), so each output is within
gamma * sum_k |a_mk b_kn| of the exact sum, gamma = (K/16 + 16) * 2^-24
(the usual n*u bound for n = K/16 + 16 rounded additions), taken twice
for margin; bf16 output adds one rounding, 2^-8 |c|.  The oracle returns
sum_k |a_mk b_kn| next to C.
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest
import torch

import oracle
from attn_inputs import random_bf16
from tests.gpu_common import announce

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


class forced_gemm:
    def __init__(self, bm, bn, bk, wm, wn, pipe):
        self.value = f"bm={bm},bn={bn},bk={bk},wm={wm},wn={wn},pipe={pipe}"

    def __enter__(self):
        import os
        self.old = os.environ.get("ATTN_FORCE_GEMM")
        os.environ["ATTN_FORCE_GEMM"] = self.value
        return self

    def __exit__(self, *exc):
        import os
        if self.old is None:
            os.environ.pop("ATTN_FORCE_GEMM", None)
        else:
            os.environ["ATTN_FORCE_GEMM"] = self.old


def _inputs(M, N, K, b_nk, seed):
    a = random_bf16((M, K), seed)
    b = random_bf16((N, K) if b_nk else (K, N), seed + 1)
    return a, b


def _check(got, want, absc, K, what, bf16_out=False):
    g = got.detach().cpu().double().numpy()
    assert g.shape == want.shape, f"{what}: shape {g.shape} vs {want.shape}"
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    tol = 2.0 * (K / 16 + 16) * 2.0 ** -24 * absc + 1e-30
    if bf16_out:
        tol = tol + 2.0 ** -8 * np.abs(want)
    err = np.abs(g - want)
    worst = np.unravel_index(np.argmax(err - tol), err.shape)
    assert np.all(err <= tol), (f"{what}: err {err[worst]:.3g} > tol {tol[worst]:.3g} at {worst}"
                                f" (max err {err.max():.3g})")


SHAPES = [(1, 8, 8), (37, 40, 72), (130, 264, 200), (300, 520, 1000), (513, 136, 4104)]


@pytest.mark.parametrize("b_nk", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_gemm_small(pa, shape, b_nk):
    M, N, K = shape
    a, b = _inputs(M, N, K, b_nk, 4000 + M + N)
    announce(f"attn_gemm {shape} b_nk={b_nk} plan {pa.gemm_plan(M, N, K, b_nk)}")
    c = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
    c16 = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    want, absc = oracle.gemm(a, b, M, N, K, b_nk=b_nk, with_abs=True)
    _check(c, want, absc, K, f"gemm {shape} b_nk={b_nk}")
    _check(c16.float(), want, absc, K, f"gemm {shape} bf16", bf16_out=True)
    assert torch.equal(c16.cpu(), c.cpu().to(torch.bfloat16)), "bf16 output is not RNE of fp32"


VARIANTS = [(64, 64, 64, 2, 2), (128, 128, 32, 2, 2), (128, 128, 64, 2, 2), (256, 128, 32, 2, 2),
            (256, 128, 64, 2, 2), (128, 256, 32, 2, 2), (128, 256, 64, 2, 2),
            (256, 256, 32, 2, 4), (256, 256, 64, 2, 4), (256, 256, 32, 2, 2), (256, 256, 64, 2, 2)]
# the hand-scheduled 256 x 256 kernel on four waves runs with two to four LDS slots
HAND_SCHEDULED = {(256, 256, 32, 2, 2), (256, 256, 64, 2, 2)}


def _fits(variant, pipe, b_nk):
    lo, hi = (1, 3) if variant in HAND_SCHEDULED else (0, 2)
    if not lo <= pipe <= hi:
        return False
    bm, bn, bk = variant[:3]
    lds = bm * (bk + 8) + (bn * (bk + 8) if b_nk else bk * (bn + 32))
    return (pipe + 1) * lds * 2 <= 160 * 1024


@pytest.mark.parametrize("pipe", [0, 1, 2, 3])
@pytest.mark.parametrize("variant", VARIANTS, ids=[str(v) for v in VARIANTS])
def test_gemm_every_variant(pa, variant, pipe):
    # ragged in every dimension against every tile (K not a multiple of BK),
    # and K spanning 1, 2, 3 and many k-tiles (pipeline prologue and tail);
    # the hand-scheduled kernel takes K in whole k-tiles (1, 2, 4, 6 and 12
    # of them, fewer than its slots included)
    shapes = ((290, 328, 384), (70, 24, 64), (33, 8, 128)) if variant in HAND_SCHEDULED else \
        ((290, 328, 360), (70, 24, 40), (33, 8, 104))
    for (M, N, K), b_nk in itertools.product(shapes, (False, True)):
        if not _fits(variant, pipe, b_nk):
            continue
        a, b = _inputs(M, N, K, b_nk, 4100 + pipe)
        announce(f"attn_gemm variant {variant} pipe={pipe} b_nk={b_nk}")
        with forced_gemm(*variant, pipe):
            c = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
            c16 = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        want, absc = oracle.gemm(a, b, M, N, K, b_nk=b_nk, with_abs=True)
        _check(c, want, absc, K, f"variant {variant} pipe={pipe} b_nk={b_nk}")
        # the bf16 epilogue (one or two 32-column blocks per staged piece) is
        # the round-to-nearest-even of the fp32 one
        assert torch.equal(c16.cpu(), c.cpu().to(torch.bfloat16)), f"bf16 {variant} pipe={pipe}" 


@pytest.mark.parametrize("variant", sorted(HAND_SCHEDULED), ids=[str(v) for v in sorted(HAND_SCHEDULED)])
def test_gemm_hand_scheduled_needs_whole_k_tiles(pa, variant):
    # K = 40 is not a whole number of 32- or 64-k tiles: forcing the tile is
    # refused before any launch (the planner never picks it there: checked
    # over seeded shapes by the host planner test)
    a = torch.zeros((64, 40), dtype=torch.bfloat16, device=DEV)
    b = torch.zeros((40, 64), dtype=torch.bfloat16, device=DEV)
    announce(f"attn_gemm {variant} with K = 40 refused")
    with forced_gemm(*variant, 1):
        with pytest.raises(pa.AttnError) as e:
            pa.gemm(a, b)
    assert e.value.code == pa.ATTN_EINVAL


class forced_gemm_split(forced_gemm):
    def __init__(self, bm, bn, bk, wm, wn, pipe, splits):
        self.value = f"bm={bm},bn={bn},bk={bk},wm={wm},wn={wn},pipe={pipe},splits={splits}"


@pytest.mark.parametrize("splits", [2, 3, 4, 8])
@pytest.mark.parametrize("variant", [((256, 256, 64, 2, 2), 1), ((256, 256, 32, 2, 2), 3)],
                         ids=["bk64-pipe1", "bk32-pipe3"])
def test_gemm_k_splits(pa, variant, splits):
    # K split into chunks of whole k-tiles, the last one shorter (23 or 46
    # k-tiles over 2, 3, 4 or 8 splits), ragged M and N, both B layouts and
    # both outputs; the partials are summed in split order, so repeated calls
    # agree bit for bit
    tile, pipe = variant
    M, N, K = 290, 328, 1472
    for b_nk in (False, True):
        a, b = _inputs(M, N, K, b_nk, 4500 + splits)
        announce(f"attn_gemm {tile} pipe={pipe} splits={splits} b_nk={b_nk}")
        with forced_gemm_split(*tile, pipe, splits):
            c = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
            c2 = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
            c16 = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk, out_dtype=torch.bfloat16)
        torch.cuda.synchronize()
        want, absc = oracle.gemm(a, b, M, N, K, b_nk=b_nk, with_abs=True)
        _check(c, want, absc, K, f"split {tile} pipe={pipe} splits={splits} b_nk={b_nk}")
        assert torch.equal(c, c2), "split GEMM not deterministic"
        assert torch.equal(c16.cpu(), c.cpu().to(torch.bfloat16)), "bf16 split output"


def test_gemm_k_split_refused_when_a_split_would_be_empty(pa):
    # 2 k-tiles of 64 cannot be split 3 ways (one split would be empty), and
    # the eight-wave tile has no split form
    a = torch.zeros((64, 128), dtype=torch.bfloat16, device=DEV)
    b = torch.zeros((128, 64), dtype=torch.bfloat16, device=DEV)
    announce("attn_gemm K split refusals")
    for tile, pipe, splits in (((256, 256, 64, 2, 2), 1, 3), ((256, 256, 64, 2, 4), 1, 2)):
        with forced_gemm_split(*tile, pipe, splits):
            with pytest.raises(pa.AttnError) as e:
                pa.gemm(a, b)
        assert e.value.code == pa.ATTN_EINVAL


def test_gemm_special_values(pa):
    # identity: C = A exactly; zeros: C = 0; a NaN in A spreads only to its row
    M, K = 200, 256
    a = random_bf16((M, K), 4200)
    eye = torch.eye(K, dtype=torch.bfloat16)
    announce("attn_gemm identity / zeros / NaN row")
    c = pa.gemm(a.to(DEV), eye.to(DEV))
    z = pa.gemm(a.to(DEV), torch.zeros((K, 72), dtype=torch.bfloat16, device=DEV))
    an = a.clone()
    an[7, 3] = float("nan")
    cn = pa.gemm(an.to(DEV), eye.to(DEV), b_nk=True)
    torch.cuda.synchronize()
    assert torch.equal(c.cpu(), a.float()), "A I != A"
    assert torch.count_nonzero(z).item() == 0
    cn = cn.cpu()
    assert torch.isnan(cn[7]).all() and not torch.isnan(cn[:7]).any() and not torch.isnan(cn[8:]).any()


def test_gemm_deterministic_and_stream_ordered(pa):
    M, N, K = 1000, 1024, 1536
    a, b = _inputs(M, N, K, False, 4300)
    ad, bd = a.to(DEV), b.to(DEV)
    announce("attn_gemm determinism")
    outs = [pa.gemm(ad, bd) for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])


LARGE = [(4096, 4096, 4096, False), (16384, 256, 2048, True), (256, 256, 16384, False),
         (2048, 8192, 1024, True), (2048, 2048, 16384, False), (16384, 256, 16384, True)]


@pytest.mark.parametrize("shape", LARGE, ids=[str(s) for s in LARGE])
def test_gemm_large_sampled_rows(pa, shape):
    # the shapes of the paper's GEMM sweep; rows sampled by the oracle
    M, N, K, b_nk = shape
    a, b = _inputs(M, N, K, b_nk, 4400 + M)
    announce(f"attn_gemm large {shape} plan {pa.gemm_plan(M, N, K, b_nk)}")
    c = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
    torch.cuda.synchronize()
    g = np.random.default_rng(M + N + K)
    rows = np.unique(np.concatenate([[0, M - 1], g.integers(0, M, 10)]))
    want, absc = oracle.gemm(a, b, M, N, K, b_nk=b_nk, rows=rows, with_abs=True)
    _check(c.cpu()[torch.from_numpy(rows)], want, absc, K, f"large {shape}")


@pytest.mark.timeout(900)
def test_gemm_bench_shape_every_element(pa):
    # the benchmark's GEMM (8192^3, B stored [K][N], fp32 C, the same seeded
    # operands and the planner's tile), every output element against the
    # oracle, on an output filled with NaN first.  The oracle reads B^T
    # through its [N][K] path (the same sums; its inner loop then runs along
    # contiguous rows).
    M = N = K = 8192
    a, b = random_bf16((M, K), 31), random_bf16((K, N), 32)
    announce(f"attn_gemm {M}x{N}x{K} every element, plan {pa.gemm_plan(M, N, K)}")
    c = torch.full((M, N), float("nan"), dtype=torch.float32, device=DEV)
    pa.gemm(a.to(DEV), b.to(DEV), c)
    torch.cuda.synchronize()
    got = c.cpu()
    del c
    announce(f"oracle GEMM {M}x{N}x{K} in fp64 on {oracle.num_threads()} threads")
    want, absc = oracle.gemm(a, b.t().contiguous(), M, N, K, b_nk=True, with_abs=True)
    _check(got, want, absc, K, "gemm 8192^3")
    err = np.abs(got.double().numpy() - want)
    print(f"[full-size parity] gemm_m8192_n8192_k8192: max_abs={err.max():.3e} "
          f"mean_abs={err.mean():.3e} max_err_over_bound="
          f"{float(np.max(err / (2.0 * (K / 16 + 16) * 2.0 ** -24 * absc + 1e-30))):.3f}",
          flush=True)


def test_gemm_rejects_before_launch(pa):
    a = torch.zeros((16, 12), dtype=torch.bfloat16, device=DEV)
    b = torch.zeros((12, 16), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:
        pa.gemm(a, b)  # K = 12 is not a multiple of 8
    assert e.value.code == pa.ATTN_EUNSUPPORTED
    c = torch.zeros((16, 16), dtype=torch.float32, device=DEV)
    rc = pa.lib.attn_gemm(a.data_ptr(), b.data_ptr(), c.data_ptr(), 16, 16, 16, 8)
    assert rc == pa.ATTN_EINVAL  # unknown flag


def _sweep_shapes(n, seed=20261204):
    """Seeded random shapes: M any size, N and K multiples of 8, log-uniform
    (so every tile edge and sizes below one tile occur), at most 2^31
    multiply-adds each for the oracle."""
    g = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        M = int(round(np.exp(g.uniform(0, np.log(4000)))))
        N = 8 * int(round(np.exp(g.uniform(0, np.log(500)))))
        K = 8 * int(round(np.exp(g.uniform(0, np.log(800)))))
        if M * N * K <= 1 << 31:
            out.append((len(out), M, N, K, bool(g.integers(0, 2))))
    return out


SWEEP = _sweep_shapes(24)


@pytest.mark.parametrize("case", SWEEP, ids=[f"{c[0]}-M{c[1]}-N{c[2]}-K{c[3]}-nk{int(c[4])}"
                                              for c in SWEEP])
def test_gemm_sweep(pa, case):
    i, M, N, K, b_nk = case
    a, b = _inputs(M, N, K, b_nk, 5000 + 2 * i)
    announce(f"sweep attn_gemm {case}")
    c = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk)
    c16 = pa.gemm(a.to(DEV), b.to(DEV), b_nk=b_nk, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    want, absc = oracle.gemm(a, b, M, N, K, b_nk=b_nk, with_abs=True)
    _check(c, want, absc, K, f"sweep gemm {case}")
    assert torch.equal(c16.cpu(), c.cpu().to(torch.bfloat16)), f"bf16 sweep {case}"

"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

All inputs are seeded and synthetic (attn_inputs).  Every test compares
every output element with the oracle, the five workloads included (at full
size, in the launch configuration the benchmark times, on NaN-filled
outputs); only the largest key range a head may have (8M keys) compares
sampled rows.  Tolerances: max-abs 2e-2 and mean-abs 2e-3 over all output
elements (bf16 inputs, fp32 accumulation); special cases with exact answers
are checked much tighter.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from attn_inputs import CONFIGS, make_inputs, random_bf16
from tests.gpu_common import announce, compare, forced_plan

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


def _rand4(B, H, S, d, seed, scale=1.0):
    return random_bf16((B, H, S, d), seed, scale)


def _fwd_case(pa, B, H, Sq, Skv, d, causal, seed, scale=None, **tol):
    q, k, v = _rand4(B, H, Sq, d, seed), _rand4(B, H, Skv, d, seed + 1), _rand4(B, H, Skv, d, seed + 2)
    sc = float(np.float32(1.0 / math.sqrt(d))) if scale is None else scale
    announce(f"attn_fwd B={B} H={H} Sq={Sq} Skv={Skv} d={d} causal={causal} seed={seed}")
    o = pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), scale=sc, causal=causal)
    torch.cuda.synchronize()
    ref = oracle.attn(q, k, v, B, H, Sq, Skv, d, sc, causal)
    return compare(o, ref, f"fwd {B,H,Sq,Skv,d,causal}", **tol)


def _report(name, stats):
    print(f"[full-size parity] {name}: max_abs={stats['max_abs']:.3e} "
          f"mean_abs={stats['mean_abs']:.3e} rel_fro={stats['rel_fro']:.3e}", flush=True)


# ------------------------------------------------------------ small shapes
def test_config_single_head(pa):
    w = CONFIGS[0]
    q, k, v = make_inputs(w)
    announce(f"attn_fwd {w.name}")
    o = torch.full((w.B, w.H, w.Sq, w.d), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), o=o, scale=w.scale, causal=w.causal)
    torch.cuda.synchronize()
    ref = oracle.attn(q, k, v, w.B, w.H, w.Sq, w.Skv, w.d, w.scale, w.causal)
    _report(w.name, compare(o, ref, w.name, rel_fro=1e-2))


SMALL = [  # B, H, Sq, Skv, d, causal
    (1, 1, 1, 1, 64, False),
    (1, 1, 1, 1, 128, True),
    (2, 3, 37, 53, 64, False),
    (2, 3, 37, 53, 128, True),
    (1, 2, 130, 130, 128, True),
    (1, 2, 300, 300, 64, True),
    (1, 1, 257, 1000, 128, False),
    (1, 1, 100, 1000, 128, True),
    (3, 1, 1, 777, 128, False),
    (1, 2, 513, 129, 64, False),
]


@pytest.mark.parametrize("shape", SMALL, ids=[str(s) for s in SMALL])
def test_fwd_small_planned(pa, shape):
    _fwd_case(pa, *shape, seed=10 + sum(shape[:5]))


VARIANTS = [(bn, w, pp) for bn in (32, 64, 128) for w in (4, 8) for pp in (0, 1, 2, 3)
            if (pp != 2 or w == 8) and (pp != 3 or bn <= 64)]


@pytest.mark.parametrize("variant", VARIANTS, ids=[f"bn{a}_w{b}_pipe{c}" for a, b, c in VARIANTS])
@pytest.mark.parametrize("d", [64, 128])
def test_fwd_every_kernel_variant(pa, variant, d):
    bn, waves, pipe = variant
    with forced_plan(bn, waves, pipe):
        for causal, (Sq, Skv) in ((False, (301, 459)), (True, (290, 290)), (True, (77, 333))):
            _fwd_case(pa, 2, 2, Sq, Skv, d, causal, seed=100 + bn + waves + d)


def test_fwd_negative_and_zero_scale(pa):
    _fwd_case(pa, 1, 2, 65, 97, 128, False, seed=300, scale=-0.0625)
    _fwd_case(pa, 1, 2, 65, 97, 64, True, seed=303, scale=0.0)


# ------------------------------------------------------ exact special cases
def test_fwd_special_cases(pa):
    B, H, S, d = 1, 2, 200, 128
    k, v = _rand4(B, H, S, d, 400), _rand4(B, H, S, d, 401)
    vn = v.double().numpy()
    announce("special cases: Q = 0")
    q0 = torch.zeros((B, H, S, d), dtype=torch.bfloat16)
    o = pa.attn_fwd(q0.to(DEV), k.to(DEV), v.to(DEV), causal=False).cpu().double().numpy()
    np.testing.assert_allclose(o, np.broadcast_to(vn.mean(axis=2, keepdims=True), o.shape),
                               atol=2e-6, rtol=0)
    o = pa.attn_fwd(q0.to(DEV), k.to(DEV), v.to(DEV), causal=True).cpu().double().numpy()
    prefix = np.cumsum(vn, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    np.testing.assert_allclose(o, prefix, atol=2e-6, rtol=0)

    announce("special cases: identical V rows, ones column, causal row 0")
    q = _rand4(B, H, S, d, 402)
    row = random_bf16((d,), 403)
    vrow = row.expand(B, H, S, d).contiguous()
    for causal in (False, True):
        o = pa.attn_fwd(q.to(DEV), k.to(DEV), vrow.to(DEV), causal=causal).cpu().double().numpy()
        np.testing.assert_allclose(o, np.broadcast_to(row.double().numpy(), o.shape), atol=2e-6,
                                   rtol=1e-6)
    v1 = v.clone()
    v1[..., 5] = 1.0
    o = pa.attn_fwd(q.to(DEV), k.to(DEV), v1.to(DEV), causal=True).cpu().double().numpy()
    np.testing.assert_allclose(o[..., 5], 1.0, atol=1e-6, rtol=0)
    np.testing.assert_allclose(o[:, :, 0], v1.double().numpy()[:, :, 0], atol=1e-6, rtol=0)

    announce("special cases: Skv = 1")
    o = pa.attn_fwd(q.to(DEV), k[:, :, :1].contiguous().to(DEV), v[:, :, :1].contiguous().to(DEV))
    np.testing.assert_allclose(o.cpu().double().numpy(),
                               np.broadcast_to(vn[:, :, :1], (B, H, S, d)), atol=1e-6, rtol=0)

    announce("special cases: planted dominant key")
    kp = _rand4(B, H, S, d, 404, 0.01)
    star = 123
    kp[0, 1, star] = (q[0, 1, 17].float() * 64).to(torch.bfloat16)
    o = pa.attn_fwd(q.to(DEV), kp.to(DEV), v.to(DEV), scale=2.0).cpu().double().numpy()
    np.testing.assert_allclose(o[0, 1, 17], vn[0, 1, star], atol=1e-5, rtol=0)


@pytest.mark.parametrize("variant", VARIANTS, ids=[f"bn{a}_w{b}_pipe{c}" for a, b, c in VARIANTS])
@pytest.mark.parametrize("d", [64, 128])
def test_fwd_exact_normaliser_every_kernel_variant(pa, variant, d):
    """The weights applied to V sum to the normaliser (both are sums of the
    same bf16-rounded probabilities), so identical V rows come back exactly and
    a column of ones stays 1, in every kernel variant: those whose row sums run
    on the matrix core and those that keep them on the VALU.  Ragged key and
    query counts, causal and not."""
    bn, waves, pipe = variant
    B, H, Sq, Skv = 1, 2, 137, 203
    q = _rand4(B, H, Sq, d, 500 + d)
    k = _rand4(B, H, Skv, d, 501 + d)
    row = random_bf16((d,), 502 + d)
    vrow = row.expand(B, H, Skv, d).contiguous()
    v1 = _rand4(B, H, Skv, d, 503 + d)
    v1[..., 3] = 1.0
    with forced_plan(bn, waves, pipe):
        for causal in (False, True):
            o = pa.attn_fwd(q.to(DEV), k.to(DEV), vrow.to(DEV), causal=causal)
            o = o.cpu().double().numpy()
            np.testing.assert_allclose(o, np.broadcast_to(row.double().numpy(), o.shape),
                                       atol=2e-6, rtol=1e-6)
            o = pa.attn_fwd(q.to(DEV), k.to(DEV), v1.to(DEV), causal=causal).cpu().double().numpy()
            np.testing.assert_allclose(o[..., 3], 1.0, atol=1e-6, rtol=0)


def test_fwd_nan_poisoned_output_fully_written(pa):
    B, H, Sq, Skv, d = 2, 3, 333, 200, 128
    q, k, v = _rand4(B, H, Sq, d, 500), _rand4(B, H, Skv, d, 501), _rand4(B, H, Skv, d, 502)
    o = torch.full((B, H, Sq, d), float("nan"), device=DEV)
    announce("nan-poisoned output")
    pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), o=o, causal=False)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()


def test_fwd_deterministic(pa):
    B, H, S, d = 2, 4, 1000, 128
    q, k, v = (_rand4(B, H, S, d, 600 + i).to(DEV) for i in range(3))
    announce("determinism")
    a = pa.attn_fwd(q, k, v, causal=True)
    b = pa.attn_fwd(q, k, v, causal=True)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_abi_rejects_before_launch(pa):
    q = torch.zeros((1, 1, 4, 64), dtype=torch.bfloat16, device=DEV)
    o = torch.full((1, 1, 4, 64), 7.0, device=DEV)
    rc = pa.lib.attn_fwd(q.data_ptr(), q.data_ptr(), q.data_ptr(), o.data_ptr(), 1, 1, 4, 2, 64,
                         1.0, 1)
    assert rc == pa.ATTN_EUNSUPPORTED
    rc = pa.lib.attn_fwd(q.data_ptr() + 2, q.data_ptr(), q.data_ptr(), o.data_ptr(), 1, 1, 4, 4,
                         64, 1.0, 0)
    assert rc == pa.ATTN_EINVAL
    torch.cuda.synchronize()
    assert (o == 7.0).all()


@pytest.mark.parametrize("shape", [(0, 2, 8, 8), (1, 0, 8, 8), (1, 2, 0, 8), (1, 2, 8, 0)],
                         ids=["B0", "H0", "Sq0", "Skv0"])
def test_empty_inputs_rejected_through_the_binding(pa, shape):
    # a zero-size batch, head set or sequence is an argument error (EINVAL),
    # raised before any launch; decode likewise for B = 0, H = 0 or Skv = 0
    B, H, Sq, Skv = shape
    q = torch.zeros((B, H, Sq, 64), dtype=torch.bfloat16, device=DEV)
    kv = torch.zeros((B, H, Skv, 64), dtype=torch.bfloat16, device=DEV)
    announce(f"empty input {shape}")
    with pytest.raises(pa.AttnError) as e:
        pa.attn_fwd(q, kv, kv)
    assert e.value.code == pa.ATTN_EINVAL
    if Sq:
        with pytest.raises(pa.AttnError) as e:
            pa.attn_decode(q[:, :, 0].contiguous(), kv, kv)
        assert e.value.code == pa.ATTN_EINVAL
    torch.cuda.synchronize()


# -------------------------------------------------------------------- decode
def test_decode_small_and_split_invariance(pa):
    B, H, Skv, d = 2, 3, 1537, 128
    q = random_bf16((B, H, d), 700)
    k, v = _rand4(B, H, Skv, d, 701), _rand4(B, H, Skv, d, 702)
    sc = float(np.float32(1.0 / math.sqrt(d)))
    ref = oracle.attn(q.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc, False)
    ref = ref.reshape(B, H, d)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    outs = {}
    for n in (0, 1, 2, 3, 7, 12, 64, Skv):
        announce(f"attn_decode B={B} H={H} Skv={Skv} d={d} n_splits={n}")
        outs[n] = pa.attn_decode(qd, kd, vd, n_splits=n)
        torch.cuda.synchronize()
        compare(outs[n], ref, f"decode n={n}")
    for n, o in outs.items():
        assert torch.allclose(o, outs[1], atol=1e-5, rtol=0), f"split {n} differs from unsplit"
    announce("attn_decode vs attn_fwd(Sq=1)")
    f = pa.attn_fwd(qd.reshape(B, H, 1, d).contiguous(), kd, vd, scale=sc).reshape(B, H, d)
    torch.cuda.synchronize()
    assert torch.allclose(f, outs[1], atol=2e-3, rtol=0)


@pytest.mark.parametrize("d", [64, 128])
def test_decode_ragged(pa, d):
    for (B, H, Skv, n) in ((1, 1, 1, 0), (1, 2, 5, 3), (3, 2, 130, 0), (2, 1, 4099, 5)):
        q = random_bf16((B, H, d), 800 + Skv)
        k, v = _rand4(B, H, Skv, d, 801 + Skv), _rand4(B, H, Skv, d, 802 + Skv)
        sc = float(np.float32(1.0 / math.sqrt(d)))
        announce(f"attn_decode B={B} H={H} Skv={Skv} d={d} n_splits={n}")
        o = pa.attn_decode(q.to(DEV), k.to(DEV), v.to(DEV), n_splits=n)
        torch.cuda.synchronize()
        ref = oracle.attn(q.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc, False)
        compare(o, ref.reshape(B, H, d), f"decode {B,H,Skv,d,n}")


def test_decode_special_cases(pa):
    B, H, Skv, d = 1, 4, 3000, 128
    k, v = _rand4(B, H, Skv, d, 900), _rand4(B, H, Skv, d, 901)
    q0 = torch.zeros((B, H, d), dtype=torch.bfloat16)
    announce("decode Q = 0")
    o = pa.attn_decode(q0.to(DEV), k.to(DEV), v.to(DEV), n_splits=5).cpu().double().numpy()
    np.testing.assert_allclose(o, v.double().numpy().mean(axis=2), atol=2e-6, rtol=0)


def test_fwd_largest_key_range(pa):
    # The largest K/V slab one head may have: the tile loads address a head's
    # keys with 31-bit buffer offsets, so Skv * d * 2 bytes must stay below
    # 2^31 (one key more is rejected on the host).  Ragged against every tile
    # width; few queries, so the non-causal launch splits the key range; the
    # causal one (bottom-right aligned) runs unsplit.  The outputs are small
    # (softmax over 8M keys), so the relative error carries the check.
    d = 128
    Skv = 0x7FFFFFFF // (2 * d)  # 8,388,607 keys, 2^31 - 256 bytes per tensor
    B, H, Sq = 1, 1, 40
    q = random_bf16((B, H, Sq, d), 990)
    k = random_bf16((B, H, Skv, d), 991)
    v = random_bf16((B, H, Skv, d), 992)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    rows = [0, 1, 17, Sq - 1]
    scale = float(np.float32(1 / math.sqrt(d)))
    for causal in (False, True):
        announce(f"attn_fwd largest key range Skv={Skv} causal={causal} "
                 f"plan {pa.get_plan(0, B, H, Sq, Skv, d, causal)}")
        o = pa.attn_fwd(qd, kd, vd, scale=scale, causal=causal)
        torch.cuda.synchronize()
        flat = o.reshape(-1, d)
        assert torch.isfinite(flat).all()
        ref = oracle.attn_rows(q, k, v, rows, B, H, Sq, Skv, d, scale, causal)
        compare(flat[rows], ref, f"Skv={Skv} causal={causal}", rel_fro=1e-2)


# -------------------------------------------------- full-size workloads
# Every output element of the four full-size workloads against the fp64
# oracle, in the launch configuration the benchmark times (the planner's
# choice), on outputs filled with NaN first, so an element the kernels never
# write fails.  Max-abs and mean-abs are taken over all B*H*Sq*d elements.
@pytest.mark.timeout(900)
@pytest.mark.parametrize("idx", [1, 2], ids=[CONFIGS[1].name, CONFIGS[2].name])
def test_fwd_full_size_every_element(pa, idx):
    w = CONFIGS[idx]
    q, k, v = make_inputs(w)
    announce(f"attn_fwd full size {w.name} plan "
             f"{pa.get_plan(pa.KIND_FWD, w.B, w.H, w.Sq, w.Skv, w.d, w.causal)}")
    o = torch.full((w.B, w.H, w.Sq, w.d), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), o=o, scale=w.scale, causal=w.causal)
    torch.cuda.synchronize()
    got = o.cpu()
    del o
    announce(f"oracle {w.name} ({w.flops() / 1e9:.0f} GFLOP in fp64 on "
             f"{oracle.num_threads()} threads)")
    ref = oracle.attn(q, k, v, w.B, w.H, w.Sq, w.Skv, w.d, w.scale, w.causal)
    _report(w.name, compare(got, ref, w.name, rel_fro=1e-2))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("idx", [3, 4], ids=[CONFIGS[3].name, CONFIGS[4].name])
def test_decode_full_size_every_element(pa, idx):
    w = CONFIGS[idx]
    q, k, v = make_inputs(w)
    announce(f"attn_decode full size {w.name} plan "
             f"{pa.get_plan(pa.KIND_DECODE, w.B, w.H, 1, w.Skv, w.d)}")
    o = torch.full((w.B, w.H, w.d), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_decode(q.to(DEV), k.to(DEV), v.to(DEV), o=o, n_splits=0)
    torch.cuda.synchronize()
    got = o.cpu()
    announce(f"oracle {w.name}")
    ref = oracle.attn(q.reshape(w.B, w.H, 1, w.d), k, v, w.B, w.H, 1, w.Skv, w.d, w.scale,
                      False)
    _report(w.name, compare(got, ref.reshape(w.B, w.H, w.d), w.name, rel_fro=1e-2))

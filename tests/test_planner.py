"""CPU tests of the analytic planner (HEG composition + constrained argmin).

The composition rules are the paper's latency-modelling equations: a
sequential composition adds, a for node multiplies by its trip count, and a
pipe node with load/body/store stages takes a sum or a max according to its
two-bit knob (Eq. heg-seq, heg-for, heg-pipe).  The rest checks properties
of the constrained argmin over the candidate domain (Eq. heg-optimization,
global-candidate-selection) on synthetic device descriptions.
"""
import ctypes
import itertools

import pytest

import paper_2609_29219_amd as pa

heg_pipe = pa.lib.attn__heg_pipe
heg_pipe.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_int, ctypes.c_int]
heg_pipe.restype = ctypes.c_double
heg_for = pa.lib.attn__heg_for
heg_for.argtypes = [ctypes.c_double, ctypes.c_double]
heg_for.restype = ctypes.c_double


@pytest.mark.parametrize("l,m,s", [(3.0, 5.0, 2.0), (7.0, 1.0, 1.0), (1.0, 1.0, 9.0), (0.0, 4.0, 0.0)])
def test_heg_pipe_knob_cases(l, m, s):
    assert heg_pipe(l, m, s, 0, 0) == l + m + s          # both boundaries closed: one serial stage
    assert heg_pipe(l, m, s, 0, 1) == max(l + m, s)      # body/store open
    assert heg_pipe(l, m, s, 1, 0) == max(l, m + s)      # load/body open
    assert heg_pipe(l, m, s, 1, 1) == max(l, m, s)       # fully pipelined


def test_heg_pipe_open_boundaries_never_slower():
    for l, m, s in itertools.product((0.5, 2.0, 7.0), repeat=3):
        closed = heg_pipe(l, m, s, 0, 0)
        for b in ((0, 1), (1, 0), (1, 1)):
            assert heg_pipe(l, m, s, *b) <= closed
        assert heg_pipe(l, m, s, 1, 1) <= min(heg_pipe(l, m, s, 0, 1), heg_pipe(l, m, s, 1, 0))


def test_heg_for_multiplies():
    assert heg_for(7, 3.5) == 24.5
    assert heg_for(0, 9.0) == 0.0


def spec():
    d = pa.DeviceDesc()
    pa.lib.attn_query_device(ctypes.byref(d))
    d.arch = b"gfx950"
    return d


def plan(desc, kind, B, H, Sq, Skv, d, causal=False, n=0):
    return pa.parse_plan(pa.get_plan(kind, B, H, Sq, Skv, d, causal, n, desc=desc))


WORKLOADS = [(pa.KIND_FWD, 1, 1, 256, 256, 64, False), (pa.KIND_FWD, 4, 16, 2048, 2048, 128, True),
             (pa.KIND_FWD, 1, 32, 8192, 8192, 128, False), (pa.KIND_DECODE, 16, 32, 1, 8192, 128, False),
             (pa.KIND_DECODE, 1, 32, 1, 131072, 128, False)]


@pytest.mark.parametrize("w", WORKLOADS)
def test_plan_is_deterministic_and_named(w):
    a = pa.get_plan(*w, desc=spec())
    b = pa.get_plan(*w, desc=spec())
    assert a == b
    p = pa.parse_plan(a)
    assert p["modeled_us"] > 0 and p["bound"]
    if w[0] == pa.KIND_FWD:
        assert p["BLOCK_N"] in (32, 64, 128) and p["WAVES"] in (4, 8) and p["PIPE"] in (0, 1, 2, 3)
        assert p["PIPE"] != 2 or p["WAVES"] == 8
        assert p["PIPE"] != 3 or p["BLOCK_N"] <= 64
        assert p["BLOCK_M"] == 32 * p["WAVES"]
        assert p["lds_bytes"] <= 160 * 1024
    else:
        assert 1 <= p["N_SPLITS"] <= w[4]
        assert (w[4] + p["CHUNK"] - 1) // p["CHUNK"] == p["N_SPLITS"]  # every split non-empty


def test_lds_capacity_constrains_the_tile():
    d = spec()
    for cap in (160 * 1024, 72 * 1024, 40 * 1024, 20 * 1024):
        d.lds_bytes_per_cu = cap
        p = plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)
        assert p["lds_bytes"] <= cap
    d.lds_bytes_per_cu = 8 * 1024  # nothing fits
    with pytest.raises(pa.AttnError) as e:
        plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)
    assert e.value.code == pa.ATTN_EUNSUPPORTED


def test_register_file_constrains_the_tile():
    d = spec()
    d.vgprs_per_simd_lane = 200
    p = plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)
    assert p["vgprs"] <= 200


def test_causal_models_about_half_the_work():
    d = spec()
    nc = plan(d, pa.KIND_FWD, 4, 16, 2048, 2048, 128, False)["modeled_us"]
    c = plan(d, pa.KIND_FWD, 4, 16, 2048, 2048, 128, True)["modeled_us"]
    assert 0.35 * nc < c < 0.8 * nc


def test_causal_residency_follows_the_grid():
    """A causal grid of one workgroup per CU runs each workgroup alone on its
    CU, whatever the kernel's footprint would allow: doubling it while it
    still fits one round of that footprint doubles the work resident on
    each CU and must cost time (the model used to charge both grids at the
    footprint's residency, the same time)."""
    d = spec()
    cands = lambda B: {(c["BLOCK_N"], c["WAVES"], c["PIPE"]): c
                       for c in pa.fwd_candidates(B, 16, 4096, 4096, 64, True, desc=d)
                       if c["KV_SPLITS"] == 1}
    one, two = cands(2), cands(4)
    checked = 0
    for key, c in one.items():
        if key not in two or c["wg_per_cu"] < 2 or c["grid"] > d.num_cus:
            continue
        if two[key]["grid"] > d.num_cus * c["wg_per_cu"]:
            continue
        assert two[key]["modeled_us"] > 1.4 * c["modeled_us"], key
        checked += 1
    assert checked > 0


def test_modeled_time_grows_with_work():
    d = spec()
    t = [plan(d, pa.KIND_FWD, 1, h, 4096, 4096, 128)["modeled_us"] for h in (8, 32, 128)]
    assert t[0] < t[1] < t[2]


def test_decode_splits_follow_compute_units():
    d = spec()
    last = 0
    for cus in (16, 64, 256, 1024):
        d.num_cus = cus
        n = plan(d, pa.KIND_DECODE, 1, 32, 1, 131072, 128)["N_SPLITS"]
        assert n >= last
        last = n
    assert last > 1  # one head per workgroup cannot fill 1024 CUs


def test_decode_explicit_splits_are_clamped():
    d = spec()
    assert plan(d, pa.KIND_DECODE, 1, 1, 1, 100, 128, n=7)["N_SPLITS"] == 7
    assert plan(d, pa.KIND_DECODE, 1, 1, 1, 100, 128, n=1000)["N_SPLITS"] == 100
    assert plan(d, pa.KIND_DECODE, 1, 1, 1, 10, 128, n=3)["CHUNK"] == 4


def test_decode_split_count_is_bounded_by_keys():
    d = spec()
    for skv in (1, 5, 127, 128, 4096):
        p = plan(d, pa.KIND_DECODE, 1, 1, 1, skv, 64)
        assert 1 <= p["N_SPLITS"] <= skv


def test_bad_descriptions_rejected():
    d = spec()
    d.num_cus = 0
    with pytest.raises(pa.AttnError) as e:
        plan(d, pa.KIND_FWD, 1, 1, 64, 64, 64)
    assert e.value.code == pa.ATTN_EINVAL


@pytest.mark.parametrize("w", [w for w in WORKLOADS if w[0] == pa.KIND_FWD])
def test_plan_is_the_argmin_of_the_candidates(w):
    d = spec()
    cands = pa.fwd_candidates(*w[1:], desc=d)
    assert cands, "no feasible candidate"
    best = min(cands, key=lambda c: c["modeled_us"])
    p = plan(d, *w)
    assert p["modeled_us"] == pytest.approx(best["modeled_us"])
    assert (p["BLOCK_N"], p["WAVES"], p["PIPE"]) in {(c["BLOCK_N"], c["WAVES"], c["PIPE"]) for c in cands}


def test_calibrated_fields_shape_the_model():
    d = spec()
    base = plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)["modeled_us"]
    d.issue_cycles_per_score *= 2
    assert plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)["modeled_us"] > base
    d = spec()
    d.valu_mfma_overlap = 0.0
    assert plan(d, pa.KIND_FWD, 1, 32, 8192, 8192, 128)["modeled_us"] > base
    d = spec()
    d.tile_sync_cycles *= 4
    slow = pa.fwd_candidates(1, 32, 8192, 8192, 128, False, desc=d)
    fast = pa.fwd_candidates(1, 32, 8192, 8192, 128, False, desc=spec())
    # synchronisation costs weigh more on narrow tiles (more tiles per row)
    def ratio(cs, bn):
        return min(c["modeled_us"] for c in cs if c["BLOCK_N"] == bn)
    assert ratio(slow, 32) / ratio(fast, 32) > ratio(slow, 128) / ratio(fast, 128)


@pytest.mark.parametrize("field,value", [("valu_mfma_overlap", 1.0), ("valu_mfma_overlap", -0.1),
                                         ("issue_cycles_per_score", -1.0),
                                         ("tile_sync_cycles", -5.0), ("tile_latency_cycles", -1.0)])
def test_calibrated_fields_out_of_range_rejected(field, value):
    d = spec()
    setattr(d, field, value)
    with pytest.raises(pa.AttnError) as e:
        plan(d, pa.KIND_FWD, 1, 1, 64, 64, 64)
    assert e.value.code == pa.ATTN_EINVAL


# ---------------------------------------------------------------- key splits
SPLIT_SHAPES = [(1, 1, 256, 256, 64, False), (1, 2, 8192, 8192, 128, False),
                (1, 32, 256, 32768, 128, False), (2, 4, 1000, 3001, 64, False),
                (1, 32, 8192, 8192, 128, False), (4, 16, 2048, 2048, 128, True)]


@pytest.mark.parametrize("shape", SPLIT_SHAPES)
def test_key_split_candidates_are_consistent(shape):
    B, H, Sq, Skv, d, causal = shape
    cands = pa.fwd_candidates(B, H, Sq, Skv, d, causal, desc=spec())
    assert cands
    for c in cands:
        n, chunk = c["KV_SPLITS"], c["KV_CHUNK"]
        if causal or c["PIPE"] == 2:
            assert n == 1
        if n == 1:
            assert chunk == Skv
            continue
        # whole tiles, every split non-empty
        assert chunk % c["BLOCK_N"] == 0
        assert (n - 1) * chunk < Skv <= n * chunk
        assert c["grid"] == B * H * c["n_qtiles"] * n
    # every (tile, split count) pair appears once
    keys = [(c["BLOCK_N"], c["WAVES"], c["PIPE"], c["KV_SPLITS"]) for c in cands]
    assert len(keys) == len(set(keys))


def test_key_splits_fill_the_device_only_when_it_is_underfilled():
    desc = spec()
    few = plan(desc, pa.KIND_FWD, 1, 2, 8192, 8192, 128)
    assert few["KV_SPLITS"] > 1  # 2 heads x 32 q-tiles cannot fill 256 CUs
    long_keys = plan(desc, pa.KIND_FWD, 1, 32, 256, 32768, 128)
    assert long_keys["KV_SPLITS"] > 1
    full = plan(desc, pa.KIND_FWD, 1, 32, 8192, 8192, 128)
    assert full["KV_SPLITS"] == 1  # 1024 workgroups already fill it


def test_key_split_model_charges_the_combine():
    # with splits the model adds the partials' traffic and a second launch:
    # on a shape that already fills the device a split can only cost time
    desc = spec()
    cands = pa.fwd_candidates(1, 32, 8192, 8192, 128, False, desc=desc)
    by_tile = {}
    for c in cands:
        by_tile.setdefault((c["BLOCK_N"], c["WAVES"], c["PIPE"]), {})[c["KV_SPLITS"]] = c["modeled_us"]
    for tile, times in by_tile.items():
        if 2 in times:
            assert times[2] > times[1] - 1e-9, tile


# --------------------------------------------------------------------- GEMM
GEMM_SHAPES = [(256, 256, 256), (1024, 1024, 1024), (4096, 4096, 4096), (16384, 256, 2048),
               (256, 256, 16384), (8192, 8192, 8192), (300, 520, 1000)]


@pytest.mark.parametrize("shape", GEMM_SHAPES)
@pytest.mark.parametrize("b_nk", [False, True])
def test_gemm_plan_is_the_argmin_of_its_candidates(shape, b_nk):
    desc = spec()
    M, N, K = shape
    cands = pa.gemm_candidates(M, N, K, b_nk, desc=desc)
    assert cands
    best = min(c["modeled_us"] for c in cands)
    p = pa.parse_plan(pa.gemm_plan(M, N, K, b_nk, desc=desc))
    assert abs(p["modeled_us"] - best) <= 1e-3 * best
    for c in cands:
        assert c["lds_bytes"] <= desc.lds_bytes_per_cu
        splits = c["K_SPLITS"]
        assert c["grid"] == -(-M // c["BLOCK_M"]) * -(-N // c["BLOCK_N"]) * splits
        assert c["b_nk"] == int(b_nk)
        if splits > 1:
            # hand-scheduled tiles only, whole k-tiles per split, none empty
            assert (c["BLOCK_M"], c["BLOCK_N"], c["WAVES_M"], c["WAVES_N"]) == (256, 256, 2, 2)
            assert c["k_chunk"] % c["BLOCK_K"] == 0
            assert (splits - 1) * c["k_chunk"] < K <= splits * c["k_chunk"]
        else:
            assert c["k_chunk"] == K


def test_gemm_k_split_model():
    # a K split pays partial traffic and a reduction: the planner never splits
    # a GEMM that already fills the CUs, and does split one with few output
    # tiles and a long K, whose split candidates it then ranks above the
    # unsplit one of the same tile
    desc = spec()
    big = pa.parse_plan(pa.gemm_plan(8192, 8192, 8192, desc=desc))
    assert big["K_SPLITS"] == 1
    thin = pa.parse_plan(pa.gemm_plan(2048, 2048, 16384, desc=desc))
    assert thin["K_SPLITS"] > 1
    same_tile = [c for c in pa.gemm_candidates(2048, 2048, 16384, desc=desc)
                 if (c["BLOCK_M"], c["BLOCK_N"], c["BLOCK_K"], c["WAVES_M"], c["WAVES_N"],
                     c["PIPE"]) == (thin["BLOCK_M"], thin["BLOCK_N"], thin["BLOCK_K"],
                                    thin["WAVES_M"], thin["WAVES_N"], thin["PIPE"])]
    unsplit = [c for c in same_tile if c["K_SPLITS"] == 1]
    assert unsplit and unsplit[0]["modeled_us"] > thin["modeled_us"]


def test_gemm_double_buffer_trade_off():
    # pipe 1 doubles the LDS footprint: never cheaper in LDS, never slower in
    # the analytic model when occupancy is unchanged (load latency hidden);
    # the measured per-kernel costs may rank a compiled pipe-1 kernel lower
    desc = spec()
    cands = pa.gemm_candidates(8192, 8192, 8192, False, desc=desc, analytic_only=True)
    by_tile = {}
    for c in cands:
        if c["K_SPLITS"] == 1:
            by_tile.setdefault((c["BLOCK_M"], c["BLOCK_N"], c["BLOCK_K"], c["WAVES_M"],
                                c["WAVES_N"]), {})[c["PIPE"]] = c
    for tile, pair in by_tile.items():
        if 0 in pair and 1 in pair:
            assert pair[1]["lds_bytes"] == 2 * pair[0]["lds_bytes"]
            if pair[1]["wg_per_cu"] == pair[0]["wg_per_cu"]:
                assert pair[1]["modeled_us"] <= pair[0]["modeled_us"] + 1e-9


def test_gemm_big_tiles_for_big_shapes_small_tiles_for_small():
    desc = spec()
    big = pa.parse_plan(pa.gemm_plan(8192, 8192, 8192, desc=desc))
    small = pa.parse_plan(pa.gemm_plan(256, 256, 256, desc=desc))
    assert big["BLOCK_M"] * big["BLOCK_N"] > small["BLOCK_M"] * small["BLOCK_N"]
    assert small["grid"] >= 4  # spread a small product over several CUs


def test_gemm_model_bounds():
    # never faster than the MFMA peak or the HBM traffic of A, B and C
    desc = spec()
    for M, N, K in GEMM_SHAPES:
        for c in pa.gemm_candidates(M, N, K, False, desc=desc):
            t = c["modeled_us"] * 1e-6
            peak = desc.mfma_bf16_flops_per_clk_cu * desc.num_cus * desc.clock_ghz * 1e9
            assert 2.0 * M * N * K / t <= peak * 1.0001
            assert (2.0 * (M * K + K * N) + 4.0 * M * N) / t <= desc.hbm_bytes_per_s * 1.0001


def test_measured_primitive_costs_only_rescale():
    # the per-kernel cost factors change modelled times, never the candidate
    # set or the tile symbols
    desc = spec()
    for args in ((4, 16, 2048, 2048, 128, True), (1, 32, 8192, 8192, 64, False)):
        a = pa.fwd_candidates(*args, desc=desc, analytic_only=True)
        b = pa.fwd_candidates(*args, desc=desc)
        key = lambda c: (c["BLOCK_N"], c["WAVES"], c["PIPE"], c["KV_SPLITS"])
        assert [key(c) for c in a] == [key(c) for c in b]
        assert any(abs(x["modeled_us"] - y["modeled_us"]) > 1e-6 for x, y in zip(a, b))
    g1 = pa.gemm_candidates(4096, 4096, 4096, desc=desc, analytic_only=True)
    g2 = pa.gemm_candidates(4096, 4096, 4096, desc=desc)
    assert [c["BLOCK_M"] for c in g1] == [c["BLOCK_M"] for c in g2]

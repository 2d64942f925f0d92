"""CPU tests of the fp64 attention oracle against its pins.

Every pin in ``oracle_pins`` runs on the oracle as built.  Then each planted
mistake (a one-line mutation of ``oracle/oracle_attn.c``, compiled to a
separate library in a temp dir) must make at least one pin fail: the pins
are strong enough to catch a dropped term, a wrong sign, an off-by-one
mask, a transposed/misindexed operand, a missing normalisation, a missing
scale or a wrong combine weight.
"""
import json
import os

import numpy as np
import pytest

import oracle
from attn_inputs import CONFIGS, make_inputs
from tests import oracle_pins

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.default())


# (name, original text, mutated text) -- each applied to one occurrence
MUTANTS = [
    ("drop_last_key", "last_key(i, Sq, Skv, causal), Skv, d, sc,\n",
     "last_key(i, Sq, Skv, causal) - 1, Skv, d, sc,\n"),
    ("exp_sign", "s[j] = exp(s[j] - m);", "s[j] = exp(m - s[j]);"),
    ("no_max_subtraction", "s[j] = exp(s[j] - m);", "s[j] = exp(s[j]);"),
    ("causal_off_by_one", "int64_t lim = i + (Skv - Sq);", "int64_t lim = i + (Skv - Sq) - 1;"),
    ("causal_top_left", "int64_t lim = i + (Skv - Sq);", "int64_t lim = i;"),
    ("reversed_k_dims", "widen_bf16(qrow[c]) * widen_bf16(kslab[j * d + c]);\n        s[j]",
     "widen_bf16(qrow[c]) * widen_bf16(kslab[j * d + (d - 1 - c)]);\n        s[j]"),
    ("values_from_k", "acc[c] += w * widen_bf16(vslab[j * d + c]);",
     "acc[c] += w * widen_bf16(kslab[j * d + c]);"),
    ("no_normalisation", "o_row[c] = acc[c] / l;", "o_row[c] = acc[c];"),
    ("no_scale", "s[j] = scale * dot;", "s[j] = dot;"),
    ("combine_sum_unweighted", "L += exp(m[t] - M) * l[t];", "L += l[t];"),
    ("combine_values_unweighted", "num += exp(m[t] - M) * u[t * d + c];", "num += u[t * d + c];"),
    ("split_drops_last_key", "const int64_t j1 = (j0 + chunk < Skv) ? j0 + chunk : Skv;",
     "const int64_t j1 = (j0 + chunk < Skv) ? j0 + chunk : Skv - 1;"),
    ("split_skips_boundary_key", "const int64_t j0 = t * chunk;",
     "const int64_t j0 = t * chunk + (t > 0);"),
    ("gqa_head_mapping", "const int64_t kvh = b * Hkv + h / group;",
     "const int64_t kvh = b * Hkv + h % Hkv;"),
    ("lse_without_stabiliser", "if (lse) *lse = m + log(l);", "if (lse) *lse = log(l);"),
    ("lse_base_two", "if (lse) *lse = m + log(l);", "if (lse) *lse = m + log2(l);"),
    ("gemm_b_layouts_swapped", "b_nk ? b[(int64_t)n * K + k] : b[(int64_t)k * N + n]",
     "b_nk ? b[(int64_t)k * N + n] : b[(int64_t)n * K + k]"),
    ("gemm_drops_last_k", "for (int k = 0; k < K; ++k) {\n                const uint16_t bk",
     "for (int k = 0; k < K - 1; ++k) {\n                const uint16_t bk"),
    ("gemm_a_row_stride", "const uint16_t* arow = a + m * (int64_t)K;",
     "const uint16_t* arow = a + m * (int64_t)N;"),
    ("gemm_signed_magnitude", "mag += fabs(p);", "mag += p;"),
    ("gemm_rows_ignored", "const int64_t m = rows ? rows[i] : i;", "const int64_t m = i;"),
    ("gemm_first_k_skipped", "double sum = 0.0, mag = 0.0;\n            for (int k = 0;",
     "double sum = 0.0, mag = 0.0;\n            for (int k = 1;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle_attn.c")).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    mutated = src.replace(old, new, 1)
    path = tmp_path / "oracle_attn.c"
    path.write_text(mutated)
    lib = oracle.build(force=True, src=str(path), out=str(tmp_path / f"lib_{name}.so"))
    orc = oracle.Oracle(lib)
    failures = []
    for pin in oracle_pins.ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(orc)
        except (AssertionError, ValueError) as e:
            failures.append((pin.__name__, str(e)[:80]))
    assert failures, f"no pin caught the planted mistake {name}"


def test_golden_regression():
    """Oracle outputs on small seeded inputs, stored by tests/golden/make_golden.py.

    This file is written only by a script that calls the oracle; it guards the
    oracle's arithmetic against unreviewed change (any change to it must name
    the passage or reading that justifies it).
    """
    with open(os.path.join(HERE, "golden", "oracle_small.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        w = CONFIGS[case["config"]].with_(B=case["B"], H=case["H"], Sq=case["Sq"],
                                          Skv=case["Skv"], seed=case["seed"])
        q, k, v = make_inputs(w)
        if w.kind == "decode":
            o = oracle.attn(q.reshape(w.B, w.H, 1, w.d), k, v, w.B, w.H, 1, w.Skv, w.d,
                            w.scale, False)
        else:
            o = oracle.attn(q, k, v, w.B, w.H, w.Sq, w.Skv, w.d, w.scale, w.causal)
        flat = o.reshape(-1)
        idx = np.asarray(case["index"])
        np.testing.assert_allclose(flat[idx], np.asarray(case["value"]), rtol=0, atol=1e-13)
        assert abs(float(np.abs(o).sum()) - case["abs_sum"]) <= 1e-9


def test_num_threads_positive():
    assert oracle.num_threads() >= 1

"""Pins for the attention oracle: checks against things other than itself.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises ``AssertionError`` when the
oracle disagrees with what mathematics or an independent library fixes:

* library routines: PyTorch's ``scaled_dot_product_attention`` and
  scipy's ``softmax`` + numpy ``matmul`` in fp64 (different code, same value);
* closed forms / special cases: Q = 0 gives the (prefix) column mean of V,
  identical V rows give that row, one key gives its value, causal row 0,
  two keys give logistic weights, a dominant planted key wins, a ones column
  of V gives ones;
* invariants: probability rows sum to one and vanish outside the mask,
  O = P V, joint permutation of keys, translation of all keys, linearity in
  V, causal rows ignore future keys, bottom-right causal alignment equals
  the tail of a longer query set, outputs are convex combinations of V;
* the exact value: 50-digit mpmath evaluation on tiny inputs;
* decode: the split-KV combine equals the unsplit result for every split
  count, and one key per split gives closed-form partials;
* grouped-query heads equal full heads with every key/value head repeated
  (and PyTorch's attention on them); the row log-sum-exp equals
  ``torch.logsumexp`` of independently computed scores, exp(s - lse) are the
  probabilities, and Q = 0 or one key give closed forms;
* GEMM: integer matrices give numpy's exact int64 product, tiny inputs the
  exact rational sum, A I = A, ones A gives B's column sums, a rank-one
  product its closed form, both B layouts agree and C^T = B^T A^T, numpy's
  fp64 matmul agrees, row subsets are rows of the full product, and the
  magnitude output is |A| |B|.

``tests/test_oracle.py`` runs every pin on the real oracle and on mutated
copies of it (each with one planted mistake), and requires every mutant to
fail at least one pin.
"""
from __future__ import annotations

import math

import numpy as np
import torch
from scipy.special import softmax as sp_softmax

from attn_inputs import bf16_bits, from_float, random_bf16

ATOL = 1e-12


def _f64(t: torch.Tensor) -> torch.Tensor:
    return t.to(torch.float64)


def _sdpa(q, k, v, scale, mask=None, is_causal=False):
    return torch.nn.functional.scaled_dot_product_attention(
        _f64(q), _f64(k), _f64(v), attn_mask=mask, is_causal=is_causal, scale=scale
    ).numpy()


def _close(a, b, atol=ATOL, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    assert np.all(np.isfinite(a)), f"{what}: non-finite values"
    err = float(np.max(np.abs(a - b))) if a.size else 0.0
    assert err <= atol, f"{what}: max abs err {err:.3e} > {atol:.1e}"


def _rand(shape, seed, scale=1.0):
    return random_bf16(shape, seed, scale)


def _scale(d):
    return float(np.float32(1.0 / math.sqrt(d)))


SHAPES = [  # (B, H, Sq, Skv, d)
    (1, 1, 1, 1, 1),
    (2, 3, 5, 7, 8),
    (1, 2, 17, 17, 16),
    (2, 1, 3, 40, 64),
    (1, 1, 33, 65, 128),
    (1, 1, 70, 70, 64),
]


# --------------------------------------------------------------- libraries
def pin_sdpa_noncausal(orc):
    for n, (B, H, Sq, Skv, d) in enumerate(SHAPES):
        q, k, v = (_rand((B, H, S, d), 100 + 3 * n + t) for t, S in enumerate((Sq, Skv, Skv)))
        sc = _scale(d)
        _close(orc.attn(q, k, v, B, H, Sq, Skv, d, sc, False), _sdpa(q, k, v, sc),
               what=f"sdpa non-causal {B,H,Sq,Skv,d}")


def pin_sdpa_causal(orc):
    for n, (B, H, Sq, Skv, d) in enumerate(SHAPES):
        q, k, v = (_rand((B, H, S, d), 200 + 3 * n + t) for t, S in enumerate((Sq, Skv, Skv)))
        sc = _scale(d)
        # bottom-right aligned mask: key j allowed for row i iff j <= i + Skv - Sq
        mask = torch.ones(Sq, Skv, dtype=torch.bool).tril(diagonal=Skv - Sq)
        _close(orc.attn(q, k, v, B, H, Sq, Skv, d, sc, True), _sdpa(q, k, v, sc, mask=mask),
               what=f"sdpa causal {B,H,Sq,Skv,d}")
        if Sq == Skv:  # library's own causal flag (top-left == bottom-right here)
            _close(orc.attn(q, k, v, B, H, Sq, Skv, d, sc, True),
                   _sdpa(q, k, v, sc, is_causal=True), what="sdpa is_causal")


def pin_scipy_softmax(orc):
    B, H, Sq, Skv, d = 2, 2, 9, 13, 32
    q, k, v = _rand((B, H, Sq, d), 300), _rand((B, H, Skv, d), 301), _rand((B, H, Skv, d), 302)
    sc = 0.37
    qn, kn, vn = (_f64(t).numpy() for t in (q, k, v))
    s = float(np.float32(sc)) * np.matmul(qn, np.swapaxes(kn, -1, -2))
    ref = np.matmul(sp_softmax(s, axis=-1), vn)
    _close(orc.attn(q, k, v, B, H, Sq, Skv, d, sc, False), ref, what="scipy softmax")


# ------------------------------------------------------------ closed forms
def pin_q_zero_mean(orc):
    B, H, S, d = 1, 2, 11, 8
    q = torch.zeros((B, H, S, d), dtype=torch.bfloat16)
    k, v = _rand((B, H, S, d), 400), _rand((B, H, S, d), 401)
    vn = _f64(v).numpy()
    _close(orc.attn(q, k, v, B, H, S, S, d, 0.5, False),
           np.broadcast_to(vn.mean(axis=2, keepdims=True), (B, H, S, d)), what="Q=0 mean")
    prefix = np.cumsum(vn, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    _close(orc.attn(q, k, v, B, H, S, S, d, 0.5, True), prefix, what="Q=0 causal prefix mean")
    # scale = 0 is the same special case with nonzero Q
    q2 = _rand((B, H, S, d), 402)
    _close(orc.attn(q2, k, v, B, H, S, S, d, 0.0, False),
           np.broadcast_to(vn.mean(axis=2, keepdims=True), (B, H, S, d)), what="scale=0 mean")


def pin_identical_v_rows(orc):
    B, H, Sq, Skv, d = 1, 1, 6, 9, 16
    q, k = _rand((B, H, Sq, d), 500), _rand((B, H, Skv, d), 501)
    row = _rand((d,), 502)
    v = row.expand(B, H, Skv, d).contiguous()
    want = np.broadcast_to(_f64(row).numpy(), (B, H, Sq, d))
    for causal in (False, True):
        _close(orc.attn(q, k, v, B, H, Sq, Skv, d, 0.25, causal), want, atol=1e-14,
               what="identical V rows")


def pin_skv_one(orc):
    B, H, Sq, d = 2, 1, 5, 4
    q, k, v = _rand((B, H, Sq, d), 600), _rand((B, H, 1, d), 601), _rand((B, H, 1, d), 602)
    _close(orc.attn(q, k, v, B, H, Sq, 1, d, 1.0, False),
           np.broadcast_to(_f64(v).numpy(), (B, H, Sq, d)), atol=0.0, what="Skv=1")


def pin_causal_row0(orc):
    B, H, S, d = 1, 3, 10, 8
    q, k, v = _rand((B, H, S, d), 700), _rand((B, H, S, d), 701), _rand((B, H, S, d), 702)
    o = orc.attn(q, k, v, B, H, S, S, d, 0.3, True)
    _close(o[:, :, 0], _f64(v).numpy()[:, :, 0], atol=0.0, what="causal row 0")


def pin_two_key_logistic(orc):
    # d = 1, scores s0 = q*k0*scale, s1 = q*k1*scale; weight of key 1 is the
    # logistic function of (s1 - s0).
    q = from_float([[[[1.5]]]])
    k = from_float([[[[0.25], [-0.75]]]])
    v = from_float([[[[2.0], [-3.0]]]])
    sc = 0.5
    s0, s1 = 1.5 * 0.25 * sc, 1.5 * -0.75 * sc
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    want = (1.0 - w1) * 2.0 + w1 * -3.0
    _close(orc.attn(q, k, v, 1, 1, 1, 2, 1, sc, False), [[[[want]]]], what="two-key logistic")


def pin_planted_key(orc):
    # One key equal to a large multiple of the query dominates: the output
    # is that key's value row.  Scores reach ~2e3, so an oracle that skips
    # the max subtraction overflows exp() and fails here.
    B, H, Sq, Skv, d = 1, 1, 4, 12, 16
    q = _rand((B, H, Sq, d), 800)
    k = _rand((B, H, Skv, d), 801, scale=0.01)
    v = _rand((B, H, Skv, d), 802)
    star = 7
    k[0, 0, star] = (q[0, 0, 2].float() * 64.0).to(torch.bfloat16)
    o = orc.attn(q, k, v, B, H, Sq, Skv, d, 2.0, False)
    _close(o[0, 0, 2], _f64(v).numpy()[0, 0, star], atol=1e-12, what="planted key")


def pin_ones_column(orc):
    B, H, Sq, Skv, d = 1, 2, 7, 19, 8
    q, k, v = _rand((B, H, Sq, d), 900), _rand((B, H, Skv, d), 901), _rand((B, H, Skv, d), 902)
    v[..., 3] = 1.0
    for causal in (False, True):
        o = orc.attn(q, k, v, B, H, Sq, Skv, d, 0.7, causal)
        _close(o[..., 3], np.ones((B, H, Sq)), atol=1e-14, what="ones column")


# -------------------------------------------------------------- invariants
def pin_probs(orc):
    B, H, Sq, Skv, d = 2, 1, 9, 14, 8
    q, k, v = _rand((B, H, Sq, d), 1000), _rand((B, H, Skv, d), 1001), _rand((B, H, Skv, d), 1002)
    for causal in (False, True):
        o, p = orc.attn_probs(q, k, v, B, H, Sq, Skv, d, 0.9, causal)
        _close(p.sum(axis=-1), np.ones((B, H, Sq)), atol=1e-14, what="P rows sum to 1")
        assert np.all(p >= 0.0), "negative probability"
        if causal:
            allowed = np.tril(np.ones((Sq, Skv), dtype=bool), k=Skv - Sq)
            assert np.all(p[..., ~allowed] == 0.0), "probability outside the mask"
            assert np.all(p[..., allowed] > 0.0), "zero probability inside the mask"
        _close(o, np.matmul(p, _f64(v).numpy()), atol=1e-13, what="O = P V")


def pin_permutation(orc):
    B, H, Sq, Skv, d = 1, 2, 6, 23, 16
    q, k, v = _rand((B, H, Sq, d), 1100), _rand((B, H, Skv, d), 1101), _rand((B, H, Skv, d), 1102)
    perm = torch.randperm(Skv, generator=torch.Generator().manual_seed(1103))
    a = orc.attn(q, k, v, B, H, Sq, Skv, d, 0.4, False)
    b = orc.attn(q, k[:, :, perm].contiguous(), v[:, :, perm].contiguous(), B, H, Sq, Skv, d,
                 0.4, False)
    _close(a, b, atol=1e-13, what="joint key/value permutation")


def _grid(shape, seed, lo=-16, hi=16, denom=8.0):
    """Values m/denom with small integer m: sums stay exact in bf16."""
    g = np.random.default_rng(seed)
    return from_float(g.integers(lo, hi + 1, size=shape) / denom)


def pin_translation(orc):
    # k_j -> k_j + u for every j adds q.u to every score of row i: no change.
    B, H, Sq, Skv, d = 1, 1, 5, 9, 8
    q, k, v = _grid((B, H, Sq, d), 1200), _grid((B, H, Skv, d), 1201), _grid((B, H, Skv, d), 1202)
    u = _grid((d,), 1203)
    k2 = (k.float() + u.float()).to(torch.bfloat16)
    assert torch.equal(k2.float(), k.float() + u.float()), "translation not exact in bf16"
    for causal in (False, True):
        _close(orc.attn(q, k, v, B, H, Sq, Skv, d, 0.5, causal),
               orc.attn(q, k2, v, B, H, Sq, Skv, d, 0.5, causal), atol=1e-13,
               what="key translation")


def pin_linearity(orc):
    B, H, Sq, Skv, d = 1, 2, 4, 10, 8
    q, k = _grid((B, H, Sq, d), 1300), _grid((B, H, Skv, d), 1301)
    v1, v2 = _grid((B, H, Skv, d), 1302), _grid((B, H, Skv, d), 1303)
    v12 = (v1.float() + v2.float()).to(torch.bfloat16)
    assert torch.equal(v12.float(), v1.float() + v2.float())
    for causal in (False, True):
        a = orc.attn(q, k, v1, B, H, Sq, Skv, d, 0.5, causal)
        b = orc.attn(q, k, v2, B, H, Sq, Skv, d, 0.5, causal)
        c = orc.attn(q, k, v12, B, H, Sq, Skv, d, 0.5, causal)
        _close(c, a + b, atol=1e-13, what="linearity in V")


def pin_causal_future(orc):
    # Row i (causal) must not see keys/values beyond i + Skv - Sq.
    B, H, Sq, Skv, d = 1, 1, 8, 12, 8
    q, k, v = _rand((B, H, Sq, d), 1400), _rand((B, H, Skv, d), 1401), _rand((B, H, Skv, d), 1402)
    a = orc.attn(q, k, v, B, H, Sq, Skv, d, 0.6, True)
    for i in range(Sq):
        lim = i + Skv - Sq
        k2, v2 = k.clone(), v.clone()
        k2[:, :, lim + 1:] = _rand(k2[:, :, lim + 1:].shape, 1500 + i)
        v2[:, :, lim + 1:] = _rand(v2[:, :, lim + 1:].shape, 1600 + i)
        b = orc.attn(q, k2, v2, B, H, Sq, Skv, d, 0.6, True)
        _close(a[:, :, i], b[:, :, i], atol=0.0, what=f"causal row {i} ignores future keys")
        if lim + 1 < Skv:  # and it does see key lim (the last allowed one)
            k3 = k.clone()
            k3[:, :, lim] = _rand(k3[:, :, lim].shape, 1700 + i)
            c = orc.attn(q, k3, v, B, H, Sq, Skv, d, 0.6, True)
            assert np.max(np.abs(c[:, :, i] - a[:, :, i])) > 1e-6, "last allowed key ignored"


def pin_bottom_right(orc):
    # Causal with Sq < Skv equals the last Sq rows of causal attention over a
    # query set padded at the front to Skv rows.
    B, H, Sq, Skv, d = 1, 2, 5, 13, 8
    q, k, v = _rand((B, H, Sq, d), 1800), _rand((B, H, Skv, d), 1801), _rand((B, H, Skv, d), 1802)
    pad = _rand((B, H, Skv - Sq, d), 1803)
    qfull = torch.cat([pad, q], dim=2).contiguous()
    a = orc.attn(q, k, v, B, H, Sq, Skv, d, 0.5, True)
    b = orc.attn(qfull, k, v, B, H, Skv, Skv, d, 0.5, True)
    _close(a, b[:, :, Skv - Sq:], atol=0.0, what="bottom-right causal alignment")


def pin_convexity(orc):
    B, H, Sq, Skv, d = 2, 2, 8, 16, 8
    q, k, v = _rand((B, H, Sq, d), 1900, 3.0), _rand((B, H, Skv, d), 1901, 3.0), \
        _rand((B, H, Skv, d), 1902)
    o = orc.attn(q, k, v, B, H, Sq, Skv, d, 1.0, False)
    vn = _f64(v).numpy()
    lo, hi = vn.min(axis=2, keepdims=True), vn.max(axis=2, keepdims=True)
    assert np.all(o >= lo - 1e-14) and np.all(o <= hi + 1e-14), "output outside hull of V"


# --------------------------------------------------------------- exactness
def pin_mpmath_exact(orc):
    import mpmath
    mpmath.mp.dps = 50
    cases = [(1, 1, 3, 5, 4, False), (1, 2, 4, 4, 3, True), (2, 1, 2, 6, 8, True)]
    for n, (B, H, Sq, Skv, d, causal) in enumerate(cases):
        q, k, v = _rand((B, H, Sq, d), 2000 + n), _rand((B, H, Skv, d), 2010 + n), \
            _rand((B, H, Skv, d), 2020 + n)
        sc = 0.75
        got = orc.attn(q, k, v, B, H, Sq, Skv, d, sc, causal)
        got_lse = orc.attn_gqa(q, k, v, B, H, H, Sq, Skv, d, sc, causal)[1]
        qf, kf, vf = (t.double().numpy() for t in (q, k, v))
        for b in range(B):
            for h in range(H):
                for i in range(Sq):
                    keys = range(Skv) if not causal else range(min(Skv, i + Skv - Sq + 1))
                    logits = [mpmath.mpf(sc) * mpmath.fsum(mpmath.mpf(qf[b, h, i, c]) *
                                                           mpmath.mpf(kf[b, h, j, c])
                                                           for c in range(d)) for j in keys]
                    lse = mpmath.log(mpmath.fsum(mpmath.exp(x) for x in logits))
                    assert abs(float(lse) - got_lse[b, h, i]) <= 1e-14, "mpmath exact lse"
                    for c in range(d):
                        exact = mpmath.fsum(mpmath.exp(x - lse) * mpmath.mpf(vf[b, h, j, c])
                                            for x, j in zip(logits, keys))
                        assert abs(float(exact) - got[b, h, i, c]) <= 1e-14, "mpmath exact"


# ------------------------------------------------------------------ decode
def pin_decode_split_equals_unsplit(orc):
    B, H, Skv, d = 2, 3, 37, 16
    q, k, v = _rand((B, H, d), 2100), _rand((B, H, Skv, d), 2101), _rand((B, H, Skv, d), 2102)
    sc = _scale(d)
    ref = _sdpa(q.reshape(B, H, 1, d), k, v, sc).reshape(B, H, d)
    full = orc.attn(q.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc, False)
    _close(full.reshape(B, H, d), ref, what="decode shape vs sdpa")
    for n in (1, 2, 3, 5, 7, 36, 37, 50):
        _close(orc.decode_split(q, k, v, B, H, Skv, d, sc, n), ref,
               what=f"split combine n={n}")


def pin_decode_split_partials(orc):
    # One key per split: m_t = s_t, l_t = 1, u_t = v_t.
    B, H, Skv, d = 1, 2, 6, 8
    q, k, v = _rand((B, H, d), 2200), _rand((B, H, Skv, d), 2201), _rand((B, H, Skv, d), 2202)
    sc = 0.3
    _, (m, l, u) = orc.decode_split(q, k, v, B, H, Skv, d, sc, Skv, return_partials=True)
    s = float(np.float32(sc)) * np.einsum("bhc,bhjc->bhj", _f64(q).numpy(), _f64(k).numpy())
    _close(m, s, atol=1e-14, what="partial max")
    _close(l, np.ones_like(l), atol=0.0, what="partial sums")
    _close(u, _f64(v).numpy(), atol=0.0, what="partial values")
    # Two splits of 3 keys: partial softmax statistics by hand
    _, (m2, l2, u2) = orc.decode_split(q, k, v, B, H, Skv, d, sc, 2, return_partials=True)
    for t in range(2):
        st = s[:, :, 3 * t:3 * t + 3]
        mt = st.max(axis=-1)
        _close(m2[:, :, t], mt, atol=1e-14, what="2-split max")
        e = np.exp(st - mt[..., None])
        _close(l2[:, :, t], e.sum(-1), atol=1e-14, what="2-split sum")
        _close(u2[:, :, t], np.einsum("bhj,bhjc->bhc", e, _f64(v).numpy()[:, :, 3 * t:3 * t + 3]),
               atol=1e-13, what="2-split values")


def pin_rows_subset(orc):
    B, H, Sq, Skv, d = 2, 2, 9, 9, 8
    q, k, v = _rand((B, H, Sq, d), 2300), _rand((B, H, Skv, d), 2301), _rand((B, H, Skv, d), 2302)
    for causal in (False, True):
        full = orc.attn(q, k, v, B, H, Sq, Skv, d, 0.5, causal).reshape(-1, d)
        rows = [0, 5, 17, 35, 20]
        _close(orc.attn_rows(q, k, v, rows, B, H, Sq, Skv, d, 0.5, causal), full[rows],
               atol=0.0, what="row subset")


# ------------------------------------------ grouped-query heads and lse
def _masked_scores(q, k, sc, causal):
    """fp64 scores scale*q.k (numpy, independent of the oracle), -inf where masked."""
    s = float(np.float32(sc)) * np.matmul(_f64(q).numpy(), np.swapaxes(_f64(k).numpy(), -1, -2))
    if causal:
        Sq, Skv = s.shape[-2], s.shape[-1]
        i = np.arange(Sq)[:, None]
        j = np.arange(Skv)[None, :]
        s = np.where(j <= i + (Skv - Sq), s, -np.inf)
    return s


def pin_gqa_equals_repeated_heads(orc):
    # Query head h reads key/value head h // g: the same as repeating every
    # key/value head g times (the library routine sees full heads).
    B, Hq, Hkv, Sq, Skv, d = 2, 6, 2, 7, 11, 8
    g = Hq // Hkv
    q, k, v = _rand((B, Hq, Sq, d), 2500), _rand((B, Hkv, Skv, d), 2501), \
        _rand((B, Hkv, Skv, d), 2502)
    kr = k.repeat_interleave(g, dim=1).contiguous()
    vr = v.repeat_interleave(g, dim=1).contiguous()
    sc = float(np.float32(0.4))  # the fp32 scale the oracle receives
    for causal in (False, True):
        o, _ = orc.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, sc, causal)
        mask = None
        if causal:
            i = torch.arange(Sq)[:, None]
            j = torch.arange(Skv)[None, :]
            mask = j <= i + (Skv - Sq)
        _close(o, _sdpa(q, kr, vr, sc, mask=mask), atol=1e-13, what=f"gqa vs sdpa causal={causal}")
        _close(o, orc.attn(q, kr, vr, B, Hq, Sq, Skv, d, sc, causal), atol=0.0,
               what="gqa vs repeated-head oracle")
    # one key/value head for every query head (multi-query)
    o, _ = orc.attn_gqa(q, k[:, :1].contiguous(), v[:, :1].contiguous(), B, Hq, 1, Sq, Skv, d,
                        sc, False)
    _close(o, _sdpa(q, k[:, :1].expand(B, Hq, Skv, d).contiguous(),
                    v[:, :1].expand(B, Hq, Skv, d).contiguous(), sc), atol=1e-13, what="mqa")


def pin_lse_logsumexp(orc):
    B, Hq, Hkv, Sq, Skv, d = 1, 4, 2, 9, 13, 16
    q, k, v = _rand((B, Hq, Sq, d), 2600), _rand((B, Hkv, Skv, d), 2601), \
        _rand((B, Hkv, Skv, d), 2602)
    kr = k.repeat_interleave(2, dim=1)
    for causal in (False, True):
        _, lse = orc.attn_gqa(q, k, v, B, Hq, Hkv, Sq, Skv, d, 0.7, causal)
        s = torch.from_numpy(_masked_scores(q, kr, 0.7, causal))
        _close(lse, torch.logsumexp(s, dim=-1).numpy(), atol=1e-13, what=f"lse causal={causal}")
        # the probabilities are exp(s - lse): they sum to one and match attn_probs
        p = np.exp(s.numpy() - lse[..., None])
        _close(p.sum(-1), np.ones_like(lse), atol=1e-13, what="exp(s - lse) sums")
        _, pref = orc.attn_probs(q, kr.contiguous(), v.repeat_interleave(2, dim=1).contiguous(),
                                 B, Hq, Sq, Skv, d, 0.7, causal)
        _close(p, pref, atol=1e-13, what="exp(s - lse) vs probabilities")


def pin_lse_closed_forms(orc):
    # Q = 0: every allowed score is 0, so lse = log(number of allowed keys)
    B, H, Sq, Skv, d = 1, 2, 5, 8, 8
    q0 = from_float(torch.zeros(B, H, Sq, d))
    k, v = _rand((B, H, Skv, d), 2700), _rand((B, H, Skv, d), 2701)
    _, lse = orc.attn_gqa(q0, k, v, B, H, H, Sq, Skv, d, 0.5, False)
    _close(lse, np.full((B, H, Sq), math.log(Skv)), atol=1e-15, what="lse Q=0")
    _, lse = orc.attn_gqa(q0, k, v, B, H, H, Sq, Skv, d, 0.5, True)
    counts = np.arange(Sq) + (Skv - Sq) + 1
    _close(lse, np.broadcast_to(np.log(counts), (B, H, Sq)), atol=1e-15, what="lse Q=0 causal")
    # one key: lse is its score
    q = _rand((B, H, Sq, d), 2702)
    _, lse = orc.attn_gqa(q, k[:, :, :1].contiguous(), v[:, :, :1].contiguous(), B, H, H, Sq, 1,
                          d, 0.5, False)
    s = float(np.float32(0.5)) * np.einsum("bhic,bhc->bhi", _f64(q).numpy(), _f64(k).numpy()[:, :, 0])
    _close(lse, s, atol=1e-14, what="lse one key")


def pin_rejects_bad_args(orc):
    q = _rand((1, 1, 4, 8), 2400)
    k = _rand((1, 1, 3, 8), 2401)
    for args in ((1, 1, 4, 3, 8, 0.5, True),):  # causal with Sq > Skv
        try:
            orc.attn(q, k, k, *args)
        except ValueError:
            pass
        else:
            raise AssertionError("causal Sq > Skv accepted")


# --------------------------------------------------------------------- GEMM
def _int_bf16(shape, seed, lo=-8, hi=8):
    """Small integers (exact in bf16; their products and sums are exact in fp64)."""
    g = np.random.default_rng(seed)
    vals = g.integers(lo, hi + 1, size=shape).astype(np.float32)
    return from_float(torch.from_numpy(vals)), vals.astype(np.int64)


def pin_gemm_integer_exact(orc):
    # integer matrices: the exact product is numpy's int64 matmul
    for (M, N, K), b_nk in (((7, 5, 9), False), ((16, 33, 130), True), ((1, 64, 1000), False)):
        a, ai = _int_bf16((M, K), 3000 + K)
        if b_nk:
            b, bi = _int_bf16((N, K), 3001 + K)
            want = ai @ bi.T
        else:
            b, bi = _int_bf16((K, N), 3001 + K)
            want = ai @ bi
        got = orc.gemm(a, b, M, N, K, b_nk=b_nk)
        assert np.array_equal(got, want.astype(np.float64)), f"gemm integer {M, N, K, b_nk}"


def pin_gemm_brute_force_fractions(orc):
    # tiny random bf16 inputs, the exact rational sum, rounded once
    from fractions import Fraction
    M, N, K = 3, 4, 5
    a, b = _rand((M, K), 3100), _rand((K, N), 3101)
    af, bf = _f64(a).numpy(), _f64(b).numpy()
    got = orc.gemm(a, b, M, N, K)
    for m in range(M):
        for n in range(N):
            exact = sum(Fraction(float(af[m, k])) * Fraction(float(bf[k, n])) for k in range(K))
            assert abs(got[m, n] - float(exact)) <= 4 * K * 2.0 ** -53 * abs(float(exact)) + 1e-300


def pin_gemm_identity(orc):
    M, K = 9, 12
    a = _rand((M, K), 3200)
    eye = from_float(torch.eye(K))
    got = orc.gemm(a, eye, M, K, K)
    assert np.array_equal(got, _f64(a).numpy()), "A I != A"
    got_nk = orc.gemm(a, eye, M, K, K, b_nk=True)
    assert np.array_equal(got_nk, _f64(a).numpy()), "A I != A (b as [N][K])"


def pin_gemm_ones_column_sums(orc):
    # A = ones: every output row is the column sums of B (exact fsum)
    M, N, K = 4, 6, 50
    a = from_float(torch.ones(M, K))
    b = _rand((K, N), 3300)
    bf = _f64(b).numpy()
    got = orc.gemm(a, b, M, N, K)
    sums = np.array([math.fsum(bf[:, n]) for n in range(N)])
    _close(got, np.broadcast_to(sums, (M, N)), atol=1e-12, what="ones @ B")


def pin_gemm_rank_one(orc):
    # a[m][k] = x_m, b[k][n] = y_n (powers of two): c = K x_m y_n exactly
    M, N, K = 5, 7, 24
    x = 2.0 ** np.arange(-2, M - 2)
    y = -(2.0 ** np.arange(-3, N - 3))
    a = from_float(torch.from_numpy(np.repeat(x[:, None], K, 1).astype(np.float32)))
    b = from_float(torch.from_numpy(np.repeat(y[None, :], K, 0).astype(np.float32)))
    got = orc.gemm(a, b, M, N, K)
    assert np.array_equal(got, K * np.outer(x, y)), "rank-one product"


def pin_gemm_layouts_and_transpose(orc):
    # B given as [N][K] equals B given as [K][N]; and C^T = B^T A^T
    M, N, K = 11, 13, 40
    a, b = _rand((M, K), 3400), _rand((K, N), 3401)
    c = orc.gemm(a, b, M, N, K)
    c_nk = orc.gemm(a, b.t().contiguous(), M, N, K, b_nk=True)
    assert np.array_equal(c, c_nk), "b layouts disagree"
    ct = orc.gemm(b.t().contiguous(), a.t().contiguous(), N, M, K)
    _close(ct, c.T, atol=1e-12, what="transpose identity")


def pin_gemm_numpy(orc):
    M, N, K = 40, 24, 700
    a, b = _rand((M, K), 3500), _rand((K, N), 3501)
    want = _f64(a).numpy() @ _f64(b).numpy()
    _close(orc.gemm(a, b, M, N, K), want, atol=1e-10, what="gemm vs numpy")


def pin_gemm_rows_and_abs(orc):
    M, N, K = 30, 8, 64
    a, b = _rand((M, K), 3600), _rand((K, N), 3601)
    full, absc = orc.gemm(a, b, M, N, K, with_abs=True)
    rows = [29, 0, 17, 17]
    assert np.array_equal(orc.gemm(a, b, M, N, K, rows=rows), full[rows]), "row subset"
    want_abs = np.abs(_f64(a).numpy()) @ np.abs(_f64(b).numpy())
    _close(absc, want_abs, atol=1e-10, what="sum of |products|")
    assert np.all(absc >= np.abs(full) - 1e-12)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]

"""Pins for the oracle's routing, permutation and RAC steps.

Routing and permutation are pinned by brute force and closed forms;
RAC by the properties the paper states (Eq. residual-shrink, the
channel-ratio trend of Tab. channel-ratio) and by exact rational arithmetic.
"""

import math
from fractions import Fraction

import numpy as np

from oracle import quant, rac, route


def test_topk_vectorised_equals_brute_force():
    rng = np.random.default_rng(0)
    logits = rng.standard_normal((40, 16)).astype(np.float32)
    logits[3, [2, 7, 9]] = 5.0          # exact ties: lower index first
    logits[4, :] = 0.0
    a = route.topk(logits, 4)
    b = route.topk_fast(logits, 4)
    assert np.array_equal(a, b)
    assert list(a[3][:3]) == [2, 7, 9]
    assert list(a[4]) == [0, 1, 2, 3]


def test_topk_brute_force_by_hand():
    logits = np.array([[0.5, 2.0, -1.0, 2.0, 1.0]], np.float32)
    assert list(route.topk(logits, 3)[0]) == [1, 3, 4]


def test_softmax_weights_closed_form():
    logits = np.array([[0.0, 1.0, 2.0, 3.0]], np.float32)
    ids = np.array([[3, 2]])
    w = route.weights(logits, ids, renorm=True)[0]
    z = math.exp(3) + math.exp(2)
    assert abs(w[0] - math.exp(3) / z) < 1e-15 and abs(w[1] - math.exp(2) / z) < 1e-15
    w0 = route.weights(logits, ids, renorm=False)[0]
    z = sum(math.exp(v) for v in [0, 1, 2, 3])
    assert abs(w0[0] - math.exp(3) / z) < 1e-15
    assert np.allclose(route.weights(logits, np.array([[1]]), True), 1.0)


def test_permutation_canonical():
    rng = np.random.default_rng(1)
    T, E, k = 50, 8, 3
    ids = route.topk_fast(rng.standard_normal((T, E)).astype(np.float32), k)
    p = route.permute(ids, E)
    R = T * k
    assert p["offsets"][0] == 0 and p["offsets"][-1] == R
    assert np.array_equal(np.diff(p["offsets"]), np.bincount(ids.reshape(-1), minlength=E))
    # rows sorted by (expert, token)
    eid = np.searchsorted(p["offsets"], np.arange(R), side="right") - 1
    key = eid.astype(np.int64) * T + p["row_token"]
    assert np.all(np.diff(key) > 0)
    # inverse map
    for t in range(T):
        for s in range(k):
            r = p["inv_row"][t, s]
            assert p["row_token"][r] == t and eid[r] == ids[t, s]


def _acts(seed, T=24, K=128, outliers=(5, 77), scale=20.0):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, K)).astype(np.float32)
    x[:, list(outliers)] *= scale
    return x.astype(np.float32)


def test_scores_match_exact_rational_sum():
    x = _acts(2, T=6, K=32, outliers=(5, 20))
    q = quant.quantize(x)
    r = rac.residual(x, quant.dequantize_f32(q["codes"], q["scales"], q["s_dec"]))
    F = rac.score_shift(q["amax"])
    s = rac.channel_scores(r, q["amax"])
    sq = (r * r).astype(np.float32)
    for j in range(32):
        exact_int = sum(math.floor(Fraction(float(sq[t, j])) * Fraction(2) ** F)
                        for t in range(6))
        assert int(s[j]) == exact_int
    # the ranking agrees with the exact sums of squares away from near-ties
    ex = rac.channel_scores_exact(r)
    for a in range(32):
        for b in range(32):
            if ex[a] > ex[b] * (1 + Fraction(1, 1000)) + Fraction(2) ** (-F + 6):
                assert s[a] >= s[b]


def test_select_brute_force_and_ties():
    scores = np.array([5, 9, 9, 1, 0, 9, 3], dtype=np.uint64)
    assert list(rac.select(scores, 3)) == [1, 2, 5]
    assert list(rac.select(scores, 4)) == [0, 1, 2, 5]
    assert list(rac.select(scores, 0)) == []
    assert list(rac.select(scores, 7)) == list(range(7))


def test_outlier_channels_are_selected():
    # expected behaviour (not a pin of the paper's numbers): the outlier
    # channels' blocks carry the largest residuals
    x = _acts(3)
    out = rac.rac_activation(x, 16)
    sel = set(out["sel"].tolist())
    assert len(sel) == 16
    assert sel <= set(range(0, 16)) | set(range(64, 80))


def test_ks_zero_is_plain_w4a4():
    x = _acts(4)
    out = rac.rac_activation(x, 0)
    assert np.all(out["rq"]["codes"] == 0) and np.all(out["rq"]["scales"] == 0)
    xt = rac.reconstruct(out["xq"], out["rq"])
    xh = quant.dequantize_f64(out["xq"]["codes"], out["xq"]["scales"], out["xq"]["s_dec"])
    assert np.array_equal(xt, xh)


def test_residual_shrink_per_element():
    """Eq. (residual-shrink) with eta = 0, element by element on S."""
    x = _acts(5)
    out = rac.rac_activation(x, 24)
    xq = out["xq"]
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    xt = rac.reconstruct(xq, out["rq"])
    x64 = x.astype(np.float64)
    e0 = np.abs(xh - x64)
    e1 = np.abs(xt - x64)
    assert np.all(e1 <= e0 * (1 + 2 ** -20) + 1e-30)
    sel = out["sel"]
    assert np.linalg.norm(e1[:, sel]) < np.linalg.norm(e0[:, sel])
    assert np.linalg.norm(xt - x64) < np.linalg.norm(xh - x64)


def test_error_non_increasing_in_ks():
    """Tab. channel-ratio: more corrected channels, smaller activation error."""
    x = _acts(6)
    x64 = x.astype(np.float64)
    prev = None
    for Ks in [0, 1, 2, 8, 16, 32, 64, 128]:
        out = rac.rac_activation(x, Ks)
        err = np.linalg.norm(rac.reconstruct(out["xq"], out["rq"]) - x64)
        if prev is not None:
            assert err <= prev * (1 + 1e-12)
        prev = err


def test_masked_residual_structure():
    x = _acts(7)
    out = rac.rac_activation(x, 10)
    rq, sel = out["rq"], out["sel"]
    K = x.shape[1]
    mask = np.zeros(K, bool)
    mask[sel] = True
    assert np.all(rq["codes"][:, ~mask] == 0)
    blocks = mask.reshape(-1, 16).any(axis=1)
    assert np.all(rq["scales"][:, ~blocks] == 0)
    # the residual has its own tensor scale: amax over all channels of r
    assert rq["amax"] == np.max(np.abs(out["r"]))
    full = quant.quantize(out["r"])
    assert np.array_equal(rq["codes"][:, mask], full["codes"][:, mask])
    assert np.array_equal(rq["scales"][:, blocks], full["scales"][:, blocks])

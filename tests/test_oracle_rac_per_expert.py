"""Pins for the per-expert RAC channel sets (reading L7 of Sec. 3.3's
Eq. (channel-score)/(channel-select) computed over each expert's own rows).

Checked against the paper's global definition where the two must agree (one
expert, or every token routed to every expert), against exact rational
scores and a per-(token, slot) evaluation that never builds the
permutation, and against Eq. (residual-shrink) per expert.
"""

from fractions import Fraction

import numpy as np
import torch

from oracle import layer, quant, rac, route


def _bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _case(seed, T=16, H=64, E=4, I=32, outliers=(3, 17, 40)):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H)).astype(np.float32)
    for c in outliers:
        x[:, c] *= 15 + c
    x = _bf16(x)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    w13 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, 2 * I, H)) * 0.05))
    w2 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, H, I)) * 0.05))
    return x, logits, w13, w2


def test_one_expert_equals_global_set():
    x, logits, w13, w2 = _case(1, E=1)
    Ks = 6
    g = layer.moe_layer(x, logits, w13, w2, 1, Ks)
    p = layer.moe_layer(x, logits, w13, w2, 1, Ks, per_expert=True)
    assert np.array_equal(p["act"]["sel_pe"][0], g["act"]["sel"])
    assert np.array_equal(p["act"]["scores_pe"][0], g["act"]["scores"])
    assert np.array_equal(p["gu"], g["gu"])
    assert np.array_equal(p["yb"], g["yb"])


def test_every_token_on_every_expert_equals_global_set():
    E = 4
    x, logits, w13, w2 = _case(2, E=E)
    Ks = 5
    g = layer.moe_layer(x, logits, w13, w2, E, Ks)
    p = layer.moe_layer(x, logits, w13, w2, E, Ks, per_expert=True)
    for e in range(E):
        assert np.array_equal(p["act"]["sel_pe"][e], g["act"]["sel"])
    assert np.array_equal(p["yb"], g["yb"])


def test_brute_force_per_token_slot():
    """S_e from exact rational sums over the tokens that chose e, and every
    (token, slot)'s [g; u] evaluated directly, without the permutation."""
    T, H, E, k, I, Ks = 12, 48, 4, 2, 16, 4
    x, logits, w13, w2 = _case(3, T=T, H=H, E=E, I=I, outliers=(5, 30))
    p = layer.moe_layer(x, logits, w13, w2, k, Ks, per_expert=True)
    ids = route.topk(logits, k)
    xq = quant.quantize(x)
    xhat = quant.dequantize_f32(xq["codes"], xq["scales"], xq["s_dec"])
    r = (xhat - x).astype(np.float32)
    rq = quant.quantize(r)
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    rh = quant.dequantize_f64(rq["codes"], rq["scales"], rq["s_dec"])
    sq = (r * r).astype(np.float32)
    for e in range(E):
        toks = [t for t in range(T) if e in ids[t]]
        exact = [sum((Fraction(float(sq[t, j])) for t in toks), Fraction(0)) for j in range(H)]
        order = sorted(range(H), key=lambda j: (-exact[j], j))
        assert sorted(order[:Ks]) == p["act"]["sel_pe"][e].tolist(), e
    for t in range(T):
        for s in range(k):
            e = int(ids[t, s])
            m = np.zeros(H, dtype=bool)
            m[p["act"]["sel_pe"][e]] = True
            a = xh[t] - np.where(m, rh[t], 0.0)
            W = layer.dequant_bank_f64(w13, e)
            gu = a @ W.T
            row = p["inv_row"][t, s]
            np.testing.assert_allclose(p["gu"][row], gu, rtol=1e-12, atol=1e-14)


def test_per_expert_residual_shrinks_on_its_set():
    """Eq. (residual-shrink) per expert: |x~ - x| <= |x_hat - x| on S_e."""
    T, H, E, k = 20, 64, 4, 2
    x, logits, _, _ = _case(4, T=T, H=H, E=E)
    ids = route.topk_fast(logits, k)
    perm = route.permute(ids, E)
    act = rac.rac_activation_per_expert(x, 8, perm["row_token"], perm["offsets"])
    xh = quant.dequantize_f64(act["xq"]["codes"], act["xq"]["scales"], act["xq"]["s_dec"])
    rh = quant.dequantize_f64(act["rq"]["codes"], act["rq"]["scales"], act["rq"]["s_dec"])
    for e in range(E):
        for t in perm["row_token"][perm["offsets"][e]:perm["offsets"][e + 1]]:
            S = act["sel_pe"][e]
            xt = xh[t, S] - rh[t, S]
            assert np.all(np.abs(xt - x[t, S]) <= np.abs(xh[t, S] - x[t, S]) + 1e-12)


def test_empty_expert_gets_the_first_channels():
    scores = np.zeros((2, 32), dtype=np.uint64)
    scores[1, [3, 9]] = 5
    sel = rac.select_per_expert(scores, 3)
    assert sel[0].tolist() == [0, 1, 2]
    assert sel[1].tolist() == [0, 3, 9]

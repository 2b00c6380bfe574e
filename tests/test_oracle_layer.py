"""Pins for the oracle's contractions and the whole-layer forward.

The grouped GEMM is checked against exact rational arithmetic; the layer is
checked against a brute-force per-(token, expert) evaluation that never
builds the permutation; the residual term against linearity (R6).
"""

import math
from fractions import Fraction

import numpy as np
import torch

from oracle import formats, fp8, layer, quant, rac, route


def _bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _case(seed, T=12, H=64, E=4, k=2, I=32):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H)).astype(np.float32)
    x[:, 3] *= 20
    x = _bf16(x)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    w13 = _bf16(rng.standard_normal((E, 2 * I, H)) * 0.05)
    w2 = _bf16(rng.standard_normal((E, H, I)) * 0.05)
    return x, logits, quant.quantize_weight_bank(w13), quant.quantize_weight_bank(w2)


def test_grouped_gemm_exact_rational():
    x, logits, w13, _ = _case(0, T=5, H=32, E=2, k=1, I=16)
    ids = route.topk_fast(logits, 1)
    perm = route.permute(ids, 2)
    xq = quant.quantize(x)
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    out, _ = layer.grouped_gemm(xh, perm["row_token"], perm["offsets"], w13)
    for r in range(5):
        t = perm["row_token"][r]
        e = layer.expert_of_rows(perm["offsets"], [r])[0]
        W = layer.dequant_bank_f64(w13, int(e))
        for n in range(16):
            exact = sum(Fraction(float(xh[t, kk])) * Fraction(float(W[n, kk]))
                        for kk in range(32))
            assert abs(Fraction(float(out[r, n])) - exact) <= abs(exact) * Fraction(1, 2 ** 45) + Fraction(1, 2 ** 80)


def test_swiglu_closed_form():
    gu = np.array([[0.0, 1.0, 2.0, -3.0, 5.0, 7.0, 1.5, 2.0]])
    h = layer.swiglu(gu, 4)
    ref = [0.0, 1.0 / (1 + math.exp(-1.0)) * 7.0, 2.0 / (1 + math.exp(-2.0)) * 1.5,
           -3.0 / (1 + math.exp(3.0)) * 2.0]
    assert np.array_equal(h[0], formats.bf16_round_f64(np.array(ref)))


def test_combine_single_slot_is_gather():
    z = np.arange(12, dtype=np.float64).reshape(4, 3)
    inv = np.array([[2], [0], [3], [1]])
    y, _ = layer.combine(z, inv, np.ones((4, 1)))
    assert np.array_equal(y, z[[2, 0, 3, 1]])


def test_residual_linearity():
    """R6: W13 stage with RAC = plain W4A4 minus the residual product."""
    x, logits, w13, _ = _case(1)
    ids = route.topk_fast(logits, 2)
    perm = route.permute(ids, 4)
    act = rac.rac_activation(x, 6)
    with_rac, _ = layer.w13_stage(act["xq"], act["rq"], perm["row_token"], perm["offsets"], w13)
    plain, _ = layer.w13_stage(act["xq"], None, perm["row_token"], perm["offsets"], w13)
    rh = quant.dequantize_f64(act["rq"]["codes"], act["rq"]["scales"], act["rq"]["s_dec"])
    res, _ = layer.grouped_gemm(rh, perm["row_token"], perm["offsets"], w13)
    assert np.allclose(with_rac, plain - res, rtol=1e-12, atol=1e-14)
    assert np.any(res != 0)


def test_layer_against_brute_force():
    """Whole layer without the permutation: loop over (token, slot)."""
    T, H, E, k, I, Ks = 10, 64, 4, 2, 32, 6
    x, logits, w13, w2 = _case(2, T, H, E, k, I)
    out = layer.moe_layer(x, logits, w13, w2, k, Ks)
    act = rac.rac_activation(x, Ks)
    xt = rac.reconstruct(act["xq"], act["rq"])
    ids = route.topk(logits, k)
    w = route.weights(logits, ids, True)
    hs = {}
    for t in range(T):
        for s in range(k):
            e = ids[t, s]
            gu = layer.dequant_bank_f64(w13, e) @ xt[t]
            g, u = gu[:I], gu[I:]
            hs[(t, s)] = formats.bf16_round_f64(g / (1 + np.exp(-g)) * u)
    amax_h = max(np.max(np.abs(v)) for v in hs.values())
    y = np.zeros((T, H))
    for t in range(T):
        for s in range(k):
            e = ids[t, s]
            hq = quant.quantize(hs[(t, s)][None, :].astype(np.float32), amax=np.float32(amax_h))
            hh = quant.dequantize_f64(hq["codes"], hq["scales"], hq["s_dec"])[0]
            z = formats.bf16_round_f64(layer.dequant_bank_f64(w2, e) @ hh)
            y[t] += w[t, s] * z
    assert np.array_equal(out["ids"], ids)
    assert np.allclose(out["y"], y, rtol=1e-12, atol=1e-15)


def test_layer_w2_site_rac_brute_force():
    """L6: RAC at the W2 input, checked per (token, slot) without the
    permutation.  The statistics of h (amax, channel scores, the residual's
    amax) are taken over all T*k rows, in any order, so the rows are stacked
    in (token, slot) order here; each row's W2 input is then its own
    reconstruction h_hat - r_S, and the residual must lower the error of z
    against the unquantised h."""
    T, H, E, k, I, Ks, Ks2 = 10, 64, 4, 2, 32, 6, 8
    x, logits, w13, w2 = _case(4, T, H, E, k, I)
    out = layer.moe_layer(x, logits, w13, w2, k, Ks, Ks2=Ks2)
    plain = layer.moe_layer(x, logits, w13, w2, k, Ks)
    act = rac.rac_activation(x, Ks)
    xt = rac.reconstruct(act["xq"], act["rq"])
    ids = route.topk(logits, k)
    w = route.weights(logits, ids, True)
    hrows = []
    for t in range(T):
        for s in range(k):
            gu = layer.dequant_bank_f64(w13, ids[t, s]) @ xt[t]
            g, u = gu[:I], gu[I:]
            hrows.append(formats.bf16_round_f64(g / (1 + np.exp(-g)) * u))
    hm = np.array(hrows)
    act2 = rac.rac_activation(hm.astype(np.float32), Ks2)
    assert np.array_equal(out["act2"]["sel"], act2["sel"])
    ht = rac.reconstruct(act2["xq"], act2["rq"])
    y = np.zeros((T, H))
    err_rac = err_plain = 0.0
    for t in range(T):
        for s in range(k):
            W = layer.dequant_bank_f64(w2, ids[t, s])
            z = formats.bf16_round_f64(W @ ht[t * k + s])
            y[t] += w[t, s] * z
    assert np.allclose(out["y"], y, rtol=1e-12, atol=1e-15)
    # z with the W2-site residual sits closer to h W2_hat^T than plain W4A4 z
    exact = np.zeros_like(out["z"])
    for r in range(T * k):
        e = int(np.searchsorted(out["offsets"], r, side="right") - 1)
        exact[r] = layer.dequant_bank_f64(w2, e) @ out["h"][r]
    err_rac = np.linalg.norm(out["z"] - exact)
    # the plain layer's h equals this one's (RAC at W2 changes nothing upstream)
    assert np.array_equal(plain["h"], out["h"])
    err_plain = np.linalg.norm(plain["z"] - exact)
    assert err_rac < err_plain


def test_fp8_rows_and_gemm():
    rng = np.random.default_rng(3)
    x = _bf16(rng.standard_normal((6, 32)) * 3)
    x[2] = 0.0
    codes, dec = fp8.quantize_rows(x)
    vals = formats.e4m3_decode(codes & 0x7F)
    # the row amax maps to the E4M3 maximum
    for r in [0, 1, 3]:
        j = np.argmax(np.abs(x[r]))
        assert vals[r, j] == 448.0
    assert np.all(codes[2] == 0) and dec[2] == 1.0
    assert np.array_equal((codes >> 7) & 1, np.signbit(x).astype(np.uint8))
    # a library cast gives the same magnitudes
    m = np.max(np.abs(x), axis=1)
    enc = np.where(m > 0, np.float32(448) / np.where(m > 0, m, 1), 1).astype(np.float32)
    v = np.minimum(np.abs(x * enc[:, None]).astype(np.float32), 448).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes & 0x7F, ref)
    # GEMM against exact rationals
    w = _bf16(rng.standard_normal((1, 4, 32)) * 0.1)
    bank = fp8.quantize_bank(w)
    out, _ = fp8.grouped_gemm(codes, dec, None, np.array([0, 6]), bank)
    A = fp8.dequantize_rows_f64(codes, dec)
    B = fp8.dequantize_rows_f64(bank["codes"][0], bank["dec"][0])
    for r in range(6):
        for n in range(4):
            exact = sum(Fraction(float(A[r, j])) * Fraction(float(B[n, j])) for j in range(32))
            assert abs(Fraction(float(out[r, n])) - exact) <= abs(exact) * Fraction(1, 2 ** 45) + Fraction(1, 2 ** 80)

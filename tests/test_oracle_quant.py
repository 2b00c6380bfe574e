"""Pins for the oracle's NVFP4 quantiser (Q1-Q8).

The paper fixes the format (E2M1 values, 16-element blocks, E4M3 scales,
FP32 tensor scale; Sec. 2.2) but not the scale recipe, so the recipe is
pinned by hand-derived special cases (each expected code below is worked out
in the comments from the definitions, not produced by the oracle) and by
invariants that any correct implementation of the recipe satisfies.
"""

import numpy as np
import torch

from oracle import formats, quant


def bf16(v):
    return float(torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).to(torch.float32))


def _worked_row():
    blocks = [
        # A: block amax 6 = tensor amax -> s_enc = 2688/6 = 448, t = 448,
        # sb = 448 = 0x7E, enc = 1, v = x; midpoints go to the even code.
        [6, -6, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5, -0.0, 0.0, -0.25, -2.5, 4.5, 5.5, -1],
        # B: block amax 1.5 -> t = 1.5/6*448 = 112 = 1.75*2^6 (exact E4M3,
        # code 0x6E); enc = 448/112 = 4, v = 4x.
        [1.5, .1875, .3125, .4375, .625, .875, 1.25, .0625, -.0625, -1.5, .25, .5, .75, 1,
         -.875, .125],
        # C: all zeros (8 positive, 8 negative) -> sb = 0, codes keep signs.
        [0.0] * 8 + [-0.0] * 8,
        # D: all equal bf16(0.7) = 0.69921875 -> t = 52.208..., nearest E4M3 is
        # 52 = 1.625*2^5 (0x65); enc = 448/52, v = 6.02... -> code 7.
        [0.69921875] * 16,
        # E: tiny block -> t = bf16(1e-4)/6*448 = 0.00747 = 3.82 * 2^-9 ->
        # subnormal E4M3 4*2^-9 = 2^-7 (0x04); enc = 448*2^7 = 57344.
        [bf16(1e-4), bf16(5e-5), bf16(-1e-4), bf16(2e-5)] + [0.0] * 12,
        # F: t = 2^-20/6*448 = 7.1e-5 < 2^-10 -> scale 0 (underflow).
        [2.0 ** -20] * 16,
    ]
    return np.array([sum(blocks, [])], dtype=np.float32)


def test_worked_example_scales_and_codes():
    x = _worked_row()
    q = quant.quantize(x)
    assert q["amax"] == 6.0
    assert q["s_enc"] == np.float32(448.0)
    assert q["s_dec"] == np.float32(1.0) / np.float32(448.0)
    assert list(q["scales"][0]) == [0x7E, 0x6E, 0x00, 0x65, 0x04, 0x00]
    codes = q["codes"][0]
    # A: 6->7, -6->F, .25->0 (tie to 0), .75->2 (tie to 1.0), 1.25->2,
    # 1.75->4, 2.5->4, 3.5->6, 5->6, -0->8, 0->0, -.25->8, -2.5->C,
    # 4.5->6 (nearest 4), 5.5->7, -1->A
    assert list(codes[0:16]) == [7, 15, 0, 2, 2, 4, 4, 6, 6, 8, 0, 8, 12, 6, 7, 10]
    # B: v = 6, .75, 1.25, 1.75, 2.5, 3.5, 5, .25, -.25, -6, 1, 2, 3, 4, -3.5, .5
    assert list(codes[16:32]) == [7, 2, 2, 4, 4, 6, 6, 0, 8, 15, 2, 4, 5, 6, 14, 1]
    assert list(codes[32:48]) == [0] * 8 + [8] * 8
    assert list(codes[48:64]) == [7] * 16
    # E: v = 5.735 -> 6, 2.867 -> 3, -5.735 -> -6, 1.147 -> 1
    assert list(codes[64:68]) == [7, 5, 15, 2]
    assert list(codes[68:80]) == [0] * 12
    assert list(codes[80:96]) == [0] * 16
    # packing: element 2j in the low nibble
    assert list(q["packed"][0][:8]) == [0xF7, 0x20, 0x42, 0x64, 0x86, 0x80, 0x6C, 0xA7]


def test_worked_example_dequant():
    x = _worked_row()
    q = quant.quantize(x)
    xh = quant.dequantize_f32(q["codes"], q["scales"], q["s_dec"])
    # block A: x_hat = e2m1 * 448 * fl(1/448)
    sdec = np.float32(1.0) / np.float32(448.0)
    assert xh[0, 0] == np.float32(np.float32(6 * 448) * sdec)
    assert np.all(xh[0, 80:96] == 0)
    assert np.array_equal(np.signbit(xh[0, 40:48]), np.ones(8, bool))


def _random_tensor(seed, rows=64, K=512):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((rows, K)).astype(np.float32)
    x[:, rng.choice(K, 5, replace=False)] *= 25
    x[3, 16:32] = 0.0
    x[5, 32:48] = np.float32(-1.25)
    x[7, 48:64] *= 1e-6
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()


def test_invariants_random():
    x = _random_tensor(0)
    q = quant.quantize(x)
    codes, sb = q["codes"], q["scales"]
    rows, K = x.shape
    xb = x.reshape(rows, K // 16, 16)
    cb = codes.reshape(rows, K // 16, 16)
    # (i) the tensor-amax element gets the largest scale and code +-6
    r, c = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert sb[r, c // 16] == 0x7E and (codes[r, c] & 7) == 7
    # (ii) every block with a normal scale has a +-6 code at its amax element
    normal = sb >= 0x08
    amax_pos = np.argmax(np.abs(xb), axis=2)
    top = np.take_along_axis(cb, amax_pos[:, :, None], axis=2)[:, :, 0] & 7
    assert np.all(top[normal] == 7)
    # (iii) the all-equal block gives all -6 codes
    assert np.all(cb[5, 2] == 15)
    # (iv) the zero block has scale 0 and zero codes
    assert sb[3, 1] == 0 and np.all(cb[3, 1] & 7 == 0)
    # signs are kept
    assert np.array_equal((codes >> 3) & 1, np.signbit(x).astype(np.uint8))


def test_error_bound():
    """(v) |x - x_hat| <= half the E2M1 spacing at v, times sbf*s_dec."""
    x = _random_tensor(1)
    q = quant.quantize(x)
    xh = quant.dequantize_f64(q["codes"], q["scales"], q["s_dec"])
    rows, K = x.shape
    sbf = formats.e4m3_decode(q["scales"])
    unit = np.repeat(sbf * np.float64(q["s_dec"]), 16, axis=1)
    v = np.abs(x.astype(np.float64)) / np.where(unit > 0, unit, 1)
    half_gap = np.where(v < 2, 0.25, np.where(v < 4, 0.5, 1.0))
    err = np.abs(x.astype(np.float64) - xh)
    ok = np.where(unit > 0, err <= half_gap * unit * (1 + 2 ** -20), True)
    assert ok.all()


def test_external_amax_gives_static_scale():
    x = _random_tensor(2)
    q1 = quant.quantize(x, amax=np.float32(100.0))
    assert q1["s_enc"] == np.float32(2688.0) / np.float32(100.0)
    q2 = quant.quantize(x)
    assert q2["amax"] == np.max(np.abs(x))


def test_zero_tensor_guard():
    x = np.zeros((2, 32), np.float32)
    x[1, :16] = -0.0
    q = quant.quantize(x)
    assert q["s_enc"] == 1 and q["s_dec"] == 1
    assert np.all(q["scales"] == 0)
    assert list(q["codes"][1, :16]) == [8] * 16
    tiny = np.full((1, 16), 2.0 ** -110, np.float32)
    q = quant.quantize(tiny)
    assert q["s_enc"] == 1 and np.all(q["scales"] == 0) and np.all(q["codes"] == 0)


def test_pack_unpack_roundtrip():
    rng = np.random.default_rng(3)
    c = rng.integers(0, 16, (5, 64)).astype(np.uint8)
    assert np.array_equal(quant.unpack(quant.pack(c)), c)
    assert quant.pack(np.array([[1, 2]], np.uint8))[0, 0] == 0x21


def test_weight_bank_per_expert_scale():
    rng = np.random.default_rng(4)
    w = (rng.standard_normal((3, 32, 64)) * [[[0.02]], [[1.0]], [[5.0]]]).astype(np.float32)
    bank = quant.quantize_weight_bank(w)
    for e in range(3):
        q = quant.quantize(w[e])
        assert np.array_equal(bank["codes"][e], q["codes"])
        assert np.array_equal(bank["scales"][e], q["scales"])
        assert bank["gscale"][e, 0] == q["s_enc"] and bank["gscale"][e, 1] == q["s_dec"]
    fq = quant.fake_quant_weight(w)
    fu = quant.fake_quant_weight(w, unscaled=True)
    for e in range(3):
        assert np.array_equal(fq[e], (fu[e] * bank["gscale"][e, 1]).astype(np.float32))


def test_dequant_f64_is_exact():
    x = _random_tensor(5)
    q = quant.quantize(x)
    d32 = quant.dequantize_f32(q["codes"], q["scales"], q["s_dec"])
    d64 = quant.dequantize_f64(q["codes"], q["scales"], q["s_dec"])
    # the float32 path rounds once (the s_dec product): within half an ulp
    assert np.all(np.abs(d32 - d64) <= np.abs(d64) * 2.0 ** -24)
    # the unscaled product is exactly representable in bfloat16
    u = quant.dequantize_unscaled_f64(q["codes"], q["scales"])
    assert np.array_equal(formats.bf16_round_f64(u), u)

"""Pins for the MXFP4 comparison oracle (oracle/mxfp4.py, rules M1-M5).

The paper does not define MX.  The conversion rule of the OCP Microscaling
(MX) v1.0 specification is pinned three ways.  First, hand-derived blocks:
every expected scale byte and code below is worked out in a comment from
the rule, not produced by the oracle.  Second, invariants that any correct
implementation of the rule satisfies: the error bound, scale invariance
under powers of two, and sign symmetry.  Third, the GEMM against an explicit
triple loop on tiny shapes.
"""

import numpy as np
import pytest

from oracle import mxfp4 as M


def _row(blocks):
    return np.array([v for b in blocks for v in b], dtype=np.float32)[None, :]


def _codes4(codes):
    return M.unpack_codes(codes)[0]


def test_scale_rule_hand_cases():
    # block amax -> floor(log2 amax) - 2 -> byte = s + 127
    cases = [
        (6.0, 127),        # log2 6 = 2.58 -> 2 - 2 = 0
        (1.0, 125),        # 0 - 2
        (7.99, 127),       # floor(log2 7.99) = 2
        (8.0, 128),        # 3 - 2
        (0.3, 123),        # log2 0.3 = -1.74 -> -2 - 2 = -4
        (2.0 ** 127, 252),  # 127 - 2 = 125
        (2.0 ** -130, 0),  # -130 - 2 = -132, clamped to -127 (a subnormal float32)
        (0.0, 0),          # all-zero block: s = -127
    ]
    for amax, byte in cases:
        x = np.zeros((1, 32), np.float32)
        x[0, 5] = np.float32(amax)
        x[0, 9] = -np.float32(amax) / 4
        _, scales = M.quantize_rows(x)
        assert int(scales[0, 0]) == byte, (amax, int(scales[0, 0]), byte)


def test_element_rounding_ties_to_even():
    # amax 6 -> X = 1: the codes are E2M1_RNE of the values themselves.
    # ties: 0.25 -> 0 (code 0, even) | 0.75 -> 1.0 (code 2) | 1.25 -> 1.0
    # (code 2) | 1.75 -> 2.0 (code 4) | 2.5 -> 2.0 (code 4) | 3.5 -> 4.0
    # (code 6) | 5.0 -> 4.0 (code 6); 7.0 saturates to 6 (code 7);
    # near ties: 0.2501 -> 0.5 (1), 2.4999 -> 2.0 (4), 5.0001 -> 6 (7)
    vals = [6.0, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.2501, 2.4999, 5.0001,
            -0.25, -0.75, -2.5, -5.0, 0.0, -0.0, 1.0, -6.0, 0.5, 3.0, 4.0, -1.5, 0.1,
            0.3, 0.7, 1.1, 1.9, 2.7, 3.2, 4.9, 5.9]
    want = [7, 0, 2, 2, 4, 4, 6, 6, 1, 4, 7,
            8, 10, 12, 14, 0, 8, 2, 15, 1, 5, 6, 11, 0,
            1, 1, 2, 4, 5, 5, 6, 7]
    codes, scales = M.quantize_rows(np.array([vals], np.float32))
    assert int(scales[0, 0]) == 127
    assert _codes4(codes).tolist() == want


def test_saturation_block():
    # amax 7.5 -> floor(log2 7.5) = 2 -> X = 1: 7.5 and 6.5 saturate to 6,
    # the rest round normally; a second block with amax 0.09375 (= 1.5 * 2^-4)
    # -> s = -4 - 2 = -6, X = 2^-6: 0.09375 / X = 6 (code 7), 0.0234375 / X
    # = 1.5 (code 3), 0.005 / X = 0.32 -> 0.5 (code 1)
    b0 = [7.5, -6.5, 1.0] + [0.0] * 29
    b1 = [0.09375, 0.0234375, -0.005] + [0.0] * 29
    codes, scales = M.quantize_rows(_row([b0, b1]))
    assert scales[0].tolist() == [127, 121]
    c = _codes4(codes)
    assert c[:3].tolist() == [7, 15, 2]
    assert c[32:35].tolist() == [7, 3, 9]


def test_packing_low_nibble_first():
    x = np.zeros((1, 32), np.float32)
    x[0, 0], x[0, 1], x[0, 2] = 6.0, 0.5, -1.0     # codes 7, 1, 10
    codes, _ = M.quantize_rows(x)
    assert codes[0, 0] == 7 | (1 << 4)
    assert codes[0, 1] == 10


def test_error_bound_and_invariants():
    rng = np.random.default_rng(3)
    x = (rng.standard_t(3, size=(40, 256)) * np.exp(rng.normal(0, 2, size=(40, 1)))).astype(np.float32)
    x[5] = 0.0
    codes, scales = M.quantize_rows(x)
    d = M.dequantize_f64(codes, scales)
    X = np.repeat(np.ldexp(1.0, scales.astype(np.int64) - 127), 32, axis=1)
    err = np.abs(d - x)
    # values up to 6X round to a neighbour at most X apart (the widest gap,
    # 4..6, is 2X); above 6X saturation costs at most 8X - 6X = 2X
    assert np.all(err <= 2 * X)
    small = np.abs(x) <= 6 * X
    assert np.all(err[small] <= X[small])
    # scaling a row by a power of two moves its scale bytes, not its codes
    c2, s2 = M.quantize_rows(x * np.float32(8.0))
    assert np.array_equal(c2, codes)
    assert np.array_equal(s2[np.arange(40) != 5], scales[np.arange(40) != 5] + 3)
    # negation flips sign bits only
    c3, s3 = M.quantize_rows(-x)
    c4 = M.unpack_codes(c3)
    nz = M.unpack_codes(codes)
    assert np.array_equal(s3, scales)
    assert np.array_equal(c4 ^ 8, nz)


def test_grouped_gemm_brute_force():
    rng = np.random.default_rng(9)
    T, K, E, N = 6, 64, 2, 5
    x = rng.standard_normal((T, K)).astype(np.float32)
    w = (rng.standard_normal((E, N, K)) * 0.05).astype(np.float32)
    xc, xs = M.quantize_rows(x)
    bank = M.quantize_bank(w)
    offsets = np.array([0, 4, 9])
    row_token = np.array([0, 2, 3, 5, 1, 1, 2, 4, 0])
    out, _ = M.grouped_gemm(xc, xs, row_token, offsets, bank)
    A = M.dequantize_f64(xc, xs)
    for r in range(9):
        e = 0 if r < 4 else 1
        W = M.dequantize_f64(bank["codes"][e], bank["scales"][e])
        for n in range(N):
            ref = 0.0
            for kk in range(K):
                ref += A[row_token[r], kk] * W[n, kk]
            assert out[r, n] == pytest.approx(ref, rel=1e-12, abs=1e-300)

"""MXFP4 W4A4 MoE layer: a comparison layer on the native FP4 format (no RAC).

Test infrastructure only: imported by tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline, never by the library.

This is not part of the paper's method.  The paper's format is NVFP4
(Sec. 2.2, "FP4" paragraph): E2M1 elements, one E4M3 scale per 16 elements
and an FP32 tensor scale.  MXFP4 is the OCP Microscaling format that CDNA4's
scaled MFMA reads natively.  It differs in two places: one power-of-two
scale (E8M0, no mantissa) per 32 elements, and no tensor scale.  Running
both layers on the same routing and shapes shows what exact NVFP4 semantics
cost on this hardware.

Conversion rule, as the OCP Microscaling Formats (MX) v1.0 specification
states it (the paper does not define MX, so this is a reading):

  M1  Per block of 32 consecutive elements of a row, with amax m = max |v|:
      shared exponent s = floor(log2 m) - 2, where 2 is the exponent of
      E2M1's largest value (6 = 1.5 * 2^2).  s is clamped to [-127, 127],
      and m == 0 gives s = -127.  The scale byte is s + 127 (E8M0); X = 2^s.
  M2  Element code = E2M1_RNE(|v| / X) with ties to even, saturating at 6,
      and the sign in bit 3.  The division by a power of two is exact.
  M3  Value = e2m1(code) * X.
  M4  out[r, n] = sum_k a[r, k] * w[e, n, k], computed in float64 here.
  M5  The layer uses the same routing, permutation, SwiGLU and combine as
      the NVFP4 layer (L1-L5), with MXFP4 activations (per token row) and
      weights (per output-channel row), and no residual.  h and z are held
      as bf16, and y = bf16_RNE of the combine.

Packing: codes u8 [rows][K/2] with element 2i in bits 3:0 and 2i+1 in bits
7:4; scales u8 [rows][K/32].

Parity is pinned in tests/test_oracle_mxfp4.py: the scale rule on chosen
blocks, the E2M1 rounding at every tie, the error bound, and a brute-force
GEMM.
"""

import numpy as np

from .formats import E2M1_MAG, e2m1_encode_mag, e2m1_decode, bf16_round_f64
from . import layer as _layer, route

BLOCK = 32
EMAX_ELEM = 2          # floor(log2(6))


def shared_exponent(m):
    """M1: float32 block maxima (>= 0) -> int64 shared exponents s."""
    m = np.asarray(m, dtype=np.float32).astype(np.float64)
    s = np.full(m.shape, -127, dtype=np.int64)
    nz = m > 0
    # frexp: m = f * 2^e, f in [0.5, 1), so floor(log2 m) = e - 1, exactly,
    # for normal and subnormal float32 values alike
    _, e = np.frexp(m[nz])
    s[nz] = np.clip(e.astype(np.int64) - 1 - EMAX_ELEM, -127, 127)
    return s


def quantize_rows(x):
    """M1-M2.  x float32 [rows][K], K % 32 == 0 -> (codes u8 [rows][K/2],
    scales u8 [rows][K/32])."""
    x = np.asarray(x, dtype=np.float32)
    R, K = x.shape
    assert K % BLOCK == 0
    blk = x.reshape(R, K // BLOCK, BLOCK)
    s = shared_exponent(np.max(np.abs(blk), axis=2) if K else np.zeros((R, 0), np.float32))
    scales = (s + 127).astype(np.uint8)
    # |v| / 2^s is exact in float64, and below 8 in magnitude
    q = np.abs(blk.astype(np.float64)) * np.ldexp(1.0, -s)[:, :, None]
    mag = e2m1_encode_mag(q.astype(np.float32))
    c4 = (mag | (np.signbit(blk).astype(np.uint8) << 3)).astype(np.uint8).reshape(R, K)
    codes = (c4[:, 0::2] | (c4[:, 1::2] << 4)).astype(np.uint8)
    return codes, scales


def unpack_codes(codes):
    """u8 [rows][K/2] -> 4-bit codes u8 [rows][K]."""
    codes = np.asarray(codes, dtype=np.uint8)
    out = np.empty(codes.shape[:-1] + (codes.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = codes & 15
    out[..., 1::2] = codes >> 4
    return out


def dequantize_f64(codes, scales):
    """M3: the exact values, float64 [rows][K]."""
    c4 = unpack_codes(codes)
    X = np.ldexp(1.0, np.asarray(scales, dtype=np.int64) - 127)
    return e2m1_decode(c4) * np.repeat(X, BLOCK, axis=-1)


def quantize_bank(w):
    """Per-output-channel MXFP4 bank: w float32 [E][N][K]."""
    E, N, K = w.shape
    codes = np.empty((E, N, K // 2), dtype=np.uint8)
    scales = np.empty((E, N, K // BLOCK), dtype=np.uint8)
    for e in range(E):
        codes[e], scales[e] = quantize_rows(w[e])
    return dict(codes=codes, scales=scales)


def grouped_gemm(a_codes, a_scales, row_token, offsets, bank, rows=None):
    """M4 for the permuted rows; returns (out, abssum) in float64."""
    offsets = np.asarray(offsets, dtype=np.int64)
    R = int(offsets[-1])
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    src = rows if row_token is None else np.asarray(row_token, dtype=np.int64)[rows]
    N = bank["codes"].shape[1]
    out = np.zeros((rows.size, N))
    mag = np.zeros((rows.size, N))
    eid = _layer.expert_of_rows(offsets, rows)
    for e in np.unique(eid):
        pick = np.nonzero(eid == e)[0]
        W = dequantize_f64(bank["codes"][e], bank["scales"][e])
        A = dequantize_f64(a_codes[src[pick]], a_scales[src[pick]])
        out[pick] = A @ W.T
        mag[pick] = np.abs(A) @ np.abs(W).T
    return out, mag


def moe_layer(x, logits, w13, w2, k, renorm=True):
    """M5: the free-running MXFP4 W4A4 layer."""
    x = np.asarray(x, dtype=np.float32)
    E = logits.shape[1]
    I = w13["codes"].shape[1] // 2
    ids = route.topk_fast(logits, k)
    wts = route.weights(logits, ids, renorm)
    perm = route.permute(ids, E)
    xc, xs = quantize_rows(x)
    gu, _ = grouped_gemm(xc, xs, perm["row_token"], perm["offsets"], w13)
    h = _layer.swiglu(gu, I)
    hc, hs = quantize_rows(h.astype(np.float32))
    z, _ = grouped_gemm(hc, hs, None, perm["offsets"], w2)
    zb = bf16_round_f64(z)
    y, _ = _layer.combine(zb, perm["inv_row"], wts)
    return dict(ids=ids, w=wts, **perm, xc=xc, xs=xs, gu=gu, h=h, hc=hc, hs=hs,
                z=z, zb=zb, y=y, yb=bf16_round_f64(y))


__all__ = ["BLOCK", "shared_exponent", "quantize_rows", "unpack_codes", "dequantize_f64",
           "quantize_bank", "grouped_gemm", "moe_layer", "E2M1_MAG"]

"""NVFP4 quantise / dequantise (the QDQ operators Q_W and Q_A).

Paper: Sec. 2.2 ("FP4" paragraph) fixes the format: E2M1 codes, one E4M3
scale per sixteen consecutive elements, an FP32 tensor scale.  Sec. 3.1
Eq. (weight-error-def) and Eq. (act-error-def) use the same QDQ operator for
weights and activations; Sec. 3.2 Eq. (w4a16-qat-forward) requires the
trainer's weight fake-quant to share it bit for bit with the rollout kernel.

The paper gives no scale recipe.  Reading used here (parity unpinned by the
paper; pinned by closed-form special cases and invariants in the tests):

  Q1  x: [rows][K] float32 (bf16-valued or float32), K % 16 == 0; blocks are
      16 consecutive elements along K (the contraction axis).
  Q2  amax = max |x| over the whole tensor (a caller may supply it).
  Q3  s_enc = fl(2688 / amax) (2688 = 6 * 448); s_dec = fl(1 / s_enc).
      If amax < 2^-100 the tensor is treated as zero: s_enc = s_dec = 1 and
      every block scale is 0 (this keeps s_enc / sbf finite for every
      non-zero E4M3 scale).
  Q4  per block b: a_b = max |x_i|; t = fl(fl(a_b / 6) * s_enc);
      sb = E4M3_RNE(min(t, 448)); sbf = value(sb).
  Q5  enc_b = 0 if sbf == 0 else fl(s_enc / sbf).
  Q6  v_i = fl(x_i * enc_b); code_i = sign(x_i) << 3 | E2M1_RNE_SAT(|v_i|)
      (negative zero and negatives that round to 0 keep the sign bit).
  Q7  byte j of a row = code_{2j} | code_{2j+1} << 4.
  Q8  x_hat_i = fl(fl(e2m1(code_i) * sbf) * s_dec); the first product is
      exact.  Contractions use the same numbers in float64 (exact).

fl(.) is one IEEE float32 operation with round-to-nearest-even; numpy
float32 scalar/array arithmetic is exactly that.
"""

import numpy as np

from .formats import (E2M1_MAG, e2m1_encode_mag, e4m3_decode, e4m3_encode_pos,
                      E4M3_MAX)

BLOCK = 16
ZERO_AMAX = np.float32(2.0 ** -100)


def tensor_scale(amax):
    """Q3: (s_enc, s_dec) as float32 from the tensor amax."""
    amax = np.float32(amax)
    if not amax >= ZERO_AMAX:
        return np.float32(1.0), np.float32(1.0)
    s_enc = np.float32(2688.0) / amax
    s_dec = np.float32(1.0) / s_enc
    return np.float32(s_enc), np.float32(s_dec)


def amax_of(x):
    """Q2: max |x| over the tensor, float32."""
    x = np.asarray(x, dtype=np.float32)
    return np.float32(np.max(np.abs(x))) if x.size else np.float32(0.0)


def quantize(x, amax=None):
    """Q1-Q7.  x: float32 [rows][K].

    Returns dict(codes=uint8 [rows][K] unpacked 4-bit codes,
                 packed=uint8 [rows][K/2], scales=uint8 [rows][K/16],
                 s_enc=float32, s_dec=float32, amax=float32).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    rows, K = x.shape
    if K % BLOCK:
        raise ValueError("K must be a multiple of 16")
    if amax is None:
        amax = amax_of(x)
    amax = np.float32(amax)
    s_enc, s_dec = tensor_scale(amax)
    zero_tensor = not amax >= ZERO_AMAX

    xb = x.reshape(rows, K // BLOCK, BLOCK)
    a_b = np.max(np.abs(xb), axis=2)                        # float32
    if zero_tensor:
        sb = np.zeros(a_b.shape, dtype=np.uint8)
    else:
        t = (a_b / np.float32(6.0)) * s_enc                  # two fl32 ops
        t = np.minimum(t, np.float32(E4M3_MAX))
        sb = e4m3_encode_pos(t)
    sbf = e4m3_decode(sb).astype(np.float32)                 # exact
    with np.errstate(divide="ignore"):
        enc = np.where(sbf == 0, np.float32(0.0),
                       s_enc / np.where(sbf == 0, np.float32(1.0), sbf))
    enc = enc.astype(np.float32)
    v = xb * enc[:, :, None]                                 # fl32
    mag = e2m1_encode_mag(np.abs(v))
    sign = np.signbit(xb).astype(np.uint8)
    codes = (sign << 3 | mag).reshape(rows, K).astype(np.uint8)
    return dict(codes=codes, packed=pack(codes), scales=sb,
                s_enc=s_enc, s_dec=s_dec, amax=amax)


def pack(codes):
    """Q7: two 4-bit codes per byte, element 2j in the low nibble."""
    codes = np.asarray(codes, dtype=np.uint8)
    return (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)


def unpack(packed):
    """Inverse of Q7."""
    packed = np.asarray(packed, dtype=np.uint8)
    rows, half = packed.shape
    codes = np.empty((rows, half * 2), dtype=np.uint8)
    codes[:, 0::2] = packed & 0xF
    codes[:, 1::2] = packed >> 4
    return codes


def _signed_mag(codes):
    mag = E2M1_MAG[codes & 7]
    return np.where((codes >> 3) & 1, -mag, mag)


def dequantize_f32(codes, scales, s_dec):
    """Q8 in float32: fl(fl(e2m1 * sbf) * s_dec) (first product exact)."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows, K = codes.shape
    e = _signed_mag(codes).astype(np.float32).reshape(rows, K // BLOCK, BLOCK)
    sbf = e4m3_decode(scales).astype(np.float32)
    p = e * sbf[:, :, None]
    return (p * np.float32(s_dec)).reshape(rows, K).astype(np.float32)


def dequantize_unscaled_f64(codes, scales):
    """e2m1(code) * sbf without the tensor scale, float64 (exact)."""
    codes = np.asarray(codes, dtype=np.uint8)
    rows, K = codes.shape
    e = _signed_mag(codes).reshape(rows, K // BLOCK, BLOCK)
    sbf = e4m3_decode(scales)
    return (e * sbf[:, :, None]).reshape(rows, K)


def dequantize_f64(codes, scales, s_dec):
    """Q8 in float64: e2m1 * sbf * s_dec, exact (<= 30 significant bits)."""
    return dequantize_unscaled_f64(codes, scales) * np.float64(np.float32(s_dec))


def quantize_weight_bank(w):
    """Q_W on an expert bank w: float32 [E][N][K] (bf16-valued).

    One tensor scale per expert matrix (Sec. 3.2: the same QDQ path is shared
    with the trainer's fake-quant).  Returns dict with codes [E][N][K],
    packed [E][N][K/2], scales [E][N][K/16], gscale float32 [E][2].
    """
    E, N, K = w.shape
    codes = np.empty((E, N, K), dtype=np.uint8)
    scales = np.empty((E, N, K // BLOCK), dtype=np.uint8)
    gscale = np.empty((E, 2), dtype=np.float32)
    for e in range(E):
        q = quantize(w[e])
        codes[e] = q["codes"]
        scales[e] = q["scales"]
        gscale[e] = (q["s_enc"], q["s_dec"])
    packed = (codes[:, :, 0::2] | (codes[:, :, 1::2] << 4)).astype(np.uint8)
    return dict(codes=codes, packed=packed, scales=scales, gscale=gscale)


def fake_quant_weight(w, unscaled=False):
    """QDQ_W of Eq. (w4a16-qat-forward): the trainer-side fake-quant.

    Returns float32 [E][N][K]: with unscaled=False the Q8 value
    fl(fl(e2m1*sbf)*s_dec); with unscaled=True the exact product e2m1*sbf
    (the tensor scale is then applied by the caller to the GEMM output).
    """
    q = quantize_weight_bank(np.asarray(w, dtype=np.float32))
    E = w.shape[0]
    out = np.empty(w.shape, dtype=np.float32)
    for e in range(E):
        if unscaled:
            out[e] = dequantize_unscaled_f64(q["codes"][e], q["scales"][e]).astype(np.float32)
        else:
            out[e] = dequantize_f32(q["codes"][e], q["scales"][e], q["gscale"][e, 1])
    return out

"""FP8 W8A8 MoE layer: the comparison baseline (no RAC).

The paper's FP8 rollout baseline (Sec. 2.2 "FP8" paragraph; Sec. 4.4.2)
uses E4M3 codes (max 448) with fine-grained scales.  The comparison layer
here uses the simplest scaling that keeps every product exact in float32
(reading; parity unpinned by the paper):

  P1  activations: one scale per row (token); weights: one scale per output
      channel (row n of W[e]).  For a row with amax m > 0:
      enc = fl(448 / m), dec = fl(1 / enc); m == 0 gives enc = dec = 1.
  P2  code = E4M3_RNE(min(|fl(x * enc)|, 448)) with the sign in bit 7.
  P3  out[r, n] = dec_a[r] * dec_w[e, n] * sum_k a_k w_k (float64 here;
      products of two E4M3 values are exact in float32).
  P4  layer: same routing / permutation / SwiGLU / combine as the NVFP4 layer
      (L1-L5) with FP8 in place of NVFP4 and no residual compensation;
      h and z are held as bf16, the layer output is bf16_RNE(y).
"""

import numpy as np

from .formats import e4m3_decode, e4m3_encode_pos, bf16_round_f64
from . import layer as _layer, route


def quantize_rows(x):
    """P1-P2 per row.  x float32 [rows][K] -> (codes uint8, dec float32 [rows])."""
    x = np.asarray(x, dtype=np.float32)
    m = np.max(np.abs(x), axis=1) if x.shape[1] else np.zeros(x.shape[0], np.float32)
    m = m.astype(np.float32)
    zero = ~(m > 0)
    enc = np.where(zero, np.float32(1.0),
                   np.float32(448.0) / np.where(zero, np.float32(1.0), m)).astype(np.float32)
    dec = (np.float32(1.0) / enc).astype(np.float32)
    v = np.abs(x * enc[:, None]).astype(np.float32)
    v = np.minimum(v, np.float32(448.0))
    mag = e4m3_encode_pos(v)
    codes = (mag | (np.signbit(x).astype(np.uint8) << 7)).astype(np.uint8)
    return codes, dec


def dequantize_rows_f64(codes, dec):
    return e4m3_decode(codes) * np.asarray(dec, dtype=np.float64)[:, None]


def quantize_bank(w):
    """Per-output-channel FP8 bank: w float32 [E][N][K]."""
    E, N, K = w.shape
    codes = np.empty((E, N, K), dtype=np.uint8)
    dec = np.empty((E, N), dtype=np.float32)
    for e in range(E):
        codes[e], dec[e] = quantize_rows(w[e])
    return dict(codes=codes, dec=dec)


def grouped_gemm(a_codes, a_dec, row_token, offsets, bank, rows=None):
    """P3 for the permuted rows; returns (out, abssum)."""
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
        W = dequantize_rows_f64(bank["codes"][e], bank["dec"][e])
        A = dequantize_rows_f64(a_codes[src[pick]], a_dec[src[pick]])
        out[pick] = A @ W.T
        mag[pick] = np.abs(A) @ np.abs(W).T
    return out, mag


def moe_layer(x, logits, w13, w2, k, renorm=True):
    """P4: free-running FP8 W8A8 layer."""
    x = np.asarray(x, dtype=np.float32)
    E = logits.shape[1]
    I = w13["codes"].shape[1] // 2
    ids = route.topk_fast(logits, k)
    wts = route.weights(logits, ids, renorm)
    perm = route.permute(ids, E)
    xc, xd = quantize_rows(x)
    gu, _ = grouped_gemm(xc, xd, perm["row_token"], perm["offsets"], w13)
    h = _layer.swiglu(gu, I)
    hc, hd = quantize_rows(h.astype(np.float32))
    z, _ = grouped_gemm(hc, hd, None, perm["offsets"], w2)
    zb = bf16_round_f64(z)
    y, _ = _layer.combine(zb, perm["inv_row"], wts)
    return dict(ids=ids, w=wts, **perm, xc=xc, xd=xd, gu=gu, h=h, hc=hc, hd=hd,
                z=z, zb=zb, y=y, yb=bf16_round_f64(y))

"""Residual Activation Compensation (RAC), Sec. 3.3 of the paper.

  Eq. (residual-def)   dX_q = Q_A(X) - X
  Eq. (residual-recon) X~ = Q_A(X) - M_S (.) Q_A(dX_q)
  Eq. (channel-score)  s_j = || dX_q[:, j] ||_2 over the current token batch
  Eq. (channel-select) S = TopK(s_j)
  Eq. (residual-shrink) ||X~ - X|| < ||Q_A(X) - X||  (property, tested)

Readings used (the paper is silent on these; parity of the exact residual
grouping is unpinned by the paper):

  R1  r = fl32(x_hat - x) for every element, x_hat from Q8.
  R2  ranking score: with amax_x = f * 2^e (frexp, f in [0.5, 1)) the
      tensor amax of X, F = 36 - 2e and
          score_j = sum_t trunc(fl32(r_tj * r_tj) * 2^F)   (uint64).
      Every |r| <= amax_x (x_hat and x share a sign and neither exceeds
      amax_x by more than an ulp), so each term is < 2^37 and the sum over up
      to 2^24 tokens fits in 64 bits.  Integer addition is associative, so
      the score is independent of summation order.  Ranking by sum r^2 is
      ranking by the L2 norm; the fixed point only merges channels whose
      squared norms differ by less than 2^-36 * amax_x^2 per token.
  R3  S = the K_s channels of largest score, ties to the lower index;
      emitted in ascending channel order.  K_s is an explicit count (the
      paper's k% = K_s / d).
  R4  the residual is quantised with Q1-Q7 over all channels (own tensor
      amax and tensor scale), then codes outside S are set to 0 and the
      scales of blocks holding no selected channel to 0 (the mask applied
      to Q_A(dX_q), as Eq. (residual-recon) writes it).
  R5  x~ = x_hat - M_S (.) r_hat  (float64, from the exact dequantised values)
  R6  y = x~ W_hat^T in float64; by linearity this equals the plain W4A4
      product minus the residual product over the selected channels.
  L7  (per-expert channel sets, a variant of R2-R4) each expert e ranks the
      channels by the scores of its own rows alone (the tokens routed to e,
      same fixed point as R2) and keeps its own S_e; the residual is
      quantised once over all channels (R4 without the mask), and the W13
      input of permuted row (t, e) is x_hat[t] - M_{S_e} (.) r_hat[t].
"""

import numpy as np

from . import quant

SCORE_FRAC_BITS = 36


def residual(x, xhat_f32):
    """R1: r = fl32(x_hat - x)."""
    return (np.asarray(xhat_f32, dtype=np.float32)
            - np.asarray(x, dtype=np.float32)).astype(np.float32)


def score_shift(amax_x):
    """R2: F = 36 - 2e with amax_x = f * 2^e, f in [0.5, 1)."""
    _, e = np.frexp(np.float32(amax_x))
    return SCORE_FRAC_BITS - 2 * int(e)


def channel_scores(r, amax_x):
    """R2: uint64 fixed-point sum of squares per channel (column)."""
    r = np.asarray(r, dtype=np.float32)
    F = score_shift(amax_x)
    sq = (r * r).astype(np.float32)                         # fl32(r^2)
    terms = np.trunc(np.ldexp(sq.astype(np.float64), F))     # exact scaling
    return terms.astype(np.uint64).sum(axis=0, dtype=np.uint64)


def channel_scores_exact(r):
    """Exact sum of fl32(r^2) per channel with rational arithmetic.

    Used by the tests to check the fixed-point ranking; slow.
    """
    from fractions import Fraction
    r = np.asarray(r, dtype=np.float32)
    sq = (r * r).astype(np.float32)
    T, K = sq.shape
    return [sum((Fraction(float(sq[t, j])) for t in range(T)), Fraction(0))
            for j in range(K)]


def select(scores, Ks):
    """R3: top-K_s channels by (score desc, index asc), returned ascending."""
    scores = np.asarray(scores, dtype=np.uint64)
    K = scores.shape[0]
    if Ks < 0 or Ks > K:
        raise ValueError("K_s out of range")
    order = sorted(range(K), key=lambda j: (-int(scores[j]), j))
    return np.array(sorted(order[:Ks]), dtype=np.int32)


def masked_residual_quant(r, sel):
    """R4: QDQ of the full residual, then the channel mask M_S."""
    r = np.asarray(r, dtype=np.float32)
    T, K = r.shape
    q = quant.quantize(r)
    mask = np.zeros(K, dtype=bool)
    mask[np.asarray(sel, dtype=np.int64)] = True
    codes = np.where(mask[None, :], q["codes"], 0).astype(np.uint8)
    block_has = mask.reshape(K // quant.BLOCK, quant.BLOCK).any(axis=1)
    scales = np.where(block_has[None, :], q["scales"], 0).astype(np.uint8)
    return dict(codes=codes, packed=quant.pack(codes), scales=scales,
                s_enc=q["s_enc"], s_dec=q["s_dec"], amax=q["amax"], mask=mask)


def reconstruct(xq, rq):
    """R5: x~ = x_hat - M_S (.) r_hat in float64."""
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    rh = quant.dequantize_f64(rq["codes"], rq["scales"], rq["s_dec"])
    return xh - rh          # r_hat is already zero outside S


def channel_scores_per_expert(r, amax_x, row_token, offsets):
    """R2 per expert (reading L7): score_e[j] over the rows routed to expert
    e, i.e. the tokens row_token[off_e .. off_{e+1}), with the fixed point of
    the whole batch (F from amax_x).  uint64 [E][K]."""
    r = np.asarray(r, dtype=np.float32)
    offsets = np.asarray(offsets, dtype=np.int64)
    row_token = np.asarray(row_token, dtype=np.int64)
    E = offsets.size - 1
    out = np.zeros((E, r.shape[1]), dtype=np.uint64)
    for e in range(E):
        toks = row_token[offsets[e]:offsets[e + 1]]
        if toks.size:
            out[e] = channel_scores(r[toks], amax_x)
    return out


def select_per_expert(scores_pe, Ks):
    """R3 per expert: S_e = top-K_s of score_e by (score desc, index asc),
    ascending.  An expert without rows has all-zero scores, so its S_e is
    channels 0 .. K_s - 1 (no row uses it).  int32 [E][K_s]."""
    scores_pe = np.asarray(scores_pe, dtype=np.uint64)
    return np.stack([select(s, Ks) for s in scores_pe]).astype(np.int32).reshape(
        scores_pe.shape[0], Ks)


def residual_quant(r):
    """R4 without the mask: Q1-Q7 of the residual over all channels with its
    own tensor scale (the per-expert variant masks it per expert, L7)."""
    return quant.quantize(np.asarray(r, dtype=np.float32))


def rac_activation_per_expert(x, Ks, row_token, offsets):
    """A3-A5 with one channel set per expert (reading L7): quantise, residual,
    per-expert scores over each expert's rows, per-expert selection, the
    residual quantised once over all channels.  The W13 input of permuted row
    (t, e) is x_hat[t] - M_{S_e} (.) r_hat[t]."""
    x = np.asarray(x, dtype=np.float32)
    xq = quant.quantize(x)
    xhat = quant.dequantize_f32(xq["codes"], xq["scales"], xq["s_dec"])
    r = residual(x, xhat)
    scores_pe = channel_scores_per_expert(r, xq["amax"], row_token, offsets)
    sel_pe = select_per_expert(scores_pe, Ks)
    rq = residual_quant(r)
    return dict(xq=xq, r=r, scores_pe=scores_pe, sel_pe=sel_pe, rq=rq)


def rac_activation(x, Ks):
    """A3-A5 on one activation tensor: quantise, residual, score, select,
    masked residual quantise.  x: float32 [T][K] (bf16-valued)."""
    x = np.asarray(x, dtype=np.float32)
    xq = quant.quantize(x)
    xhat = quant.dequantize_f32(xq["codes"], xq["scales"], xq["s_dec"])
    r = residual(x, xhat)
    scores = channel_scores(r, xq["amax"])
    sel = select(scores, Ks)
    rq = masked_residual_quant(r, sel)
    return dict(xq=xq, r=r, scores=scores, sel=sel, rq=rq)

"""The NVFP4 W4A4 MoE expert layer with RAC at the W13 input (Sec. 3.3).

Layer order (routing, SwiGLU and the weighted combine are not specified by
the paper; readings, parity unpinned by the paper):

  L4  per expert e, rows [off_e, off_{e+1}):  [g; u] = x~[row_token] W13_hat[e]^T
      (float64; W13[e] is [2I][H], gate rows [0, I), up rows [I, 2I));
      h = bf16_RNE(silu(g) * u), silu(g) = g / (1 + exp(-g)).
  L5  h_hat = Q_A(h) (plain NVFP4; the paper profiles RAC at the W13
      activation site only, Sec. 3.3);
      z = bf16_RNE(h_hat W2_hat[e]^T) (float64 product, W2[e] is [H][I]; the
      expert outputs are held as bf16 between the down projection and the
      combine);
      y[t] = sum_s w[t, s] * z[inv_row[t, s]] (float64), s = 0..k-1; the
      layer output is bf16_RNE(y).
  L6  Optional RAC at the W2 input as well (K_s2 > 0; an extension the
      paper's method admits at any activation site, Sec. 3.3): h goes
      through the same steps A3-A5 as X, with the R = T*k permuted rows of h
      as the batch (one channel set shared by all experts), and
      z = bf16_RNE((h_hat - M_S (.) Q_A(dh_q)) W2_hat[e]^T) as in
      Eq. (residual-recon).
  L7  Optional per-expert channel sets at the W13 input (per_expert=True):
      each expert selects S_e from the scores of its own rows (oracle.rac,
      reading L7) and its rows subtract M_{S_e} (.) r_hat.

Stage functions take the previous stage's values explicitly so the tests can
teacher-force them with the GPU's own intermediates (bf16 h, z), and return
the sum of absolute products next to each contraction: the magnitude of the
terms a float32 accumulator adds, used for the tolerance floor.
"""

import numpy as np

from . import quant, rac, route
from .formats import bf16_round_f64


def dequant_bank_f64(bank, e):
    """Exact float64 W_hat[e] from a quantised bank (Q8)."""
    return quant.dequantize_f64(bank["codes"][e], bank["scales"][e],
                                bank["gscale"][e, 1])


def expert_of_rows(offsets, rows):
    offsets = np.asarray(offsets, dtype=np.int64)
    return np.searchsorted(offsets, np.asarray(rows, dtype=np.int64), side="right") - 1


def grouped_gemm(a_src, row_token, offsets, bank, rows=None, a_abs_src=None):
    """Per-expert float64 GEMM: out[r] = a_src[src(r)] W_hat[e(r)]^T.

    a_src: float64 [*][K] dequantised operand rows; row r of the grouped
    problem reads a_src[row_token[r]] (or a_src[r] when row_token is None).
    rows: optional subset of row indices to evaluate (default all).
    a_abs_src: optional magnitudes used for the abs-sum (default |a_src|).
    Returns (out [len(rows)][N], abssum [len(rows)][N]).
    """
    offsets = np.asarray(offsets, dtype=np.int64)
    R = int(offsets[-1])
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    src = rows if row_token is None else np.asarray(row_token, dtype=np.int64)[rows]
    N = bank["codes"].shape[1]
    out = np.zeros((rows.size, N), dtype=np.float64)
    mag = np.zeros((rows.size, N), dtype=np.float64)
    eid = expert_of_rows(offsets, rows)
    for e in np.unique(eid):
        pick = np.nonzero(eid == e)[0]
        W = dequant_bank_f64(bank, int(e))
        A = a_src[src[pick]]
        out[pick] = A @ W.T
        Aa = np.abs(A) if a_abs_src is None else a_abs_src[src[pick]]
        mag[pick] = Aa @ np.abs(W).T
    return out, mag


def w13_stage(xq, rq, row_token, offsets, w13, rows=None):
    """A6 contraction (before the SwiGLU): [g; u] for the permuted rows.

    The residual enters with its own tensor scale (R5/R6).  The abs-sum
    counts both the main and the residual terms, which a GPU accumulates
    separately.  row_token None means the rows are the tokens themselves
    (a dense GEMM).
    """
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    if rq is not None:
        rh = quant.dequantize_f64(rq["codes"], rq["scales"], rq["s_dec"])
    else:
        rh = np.zeros_like(xh)
    return grouped_gemm(xh - rh, row_token, offsets, w13, rows=rows,
                        a_abs_src=np.abs(xh) + np.abs(rh))


def w13_stage_per_expert(xq, rq, sel_pe, row_token, offsets, w13, rows=None):
    """A6 with per-expert channel sets (L7): permuted row r of expert e
    contracts x_hat[t] - M_{S_e} (.) r_hat[t] (t = row_token[r]) against
    W13_hat[e].  rq: the unmasked residual quantisation.  Returns ([g; u],
    abs-sum) like w13_stage."""
    xh = quant.dequantize_f64(xq["codes"], xq["scales"], xq["s_dec"])
    rh = quant.dequantize_f64(rq["codes"], rq["scales"], rq["s_dec"])
    offsets = np.asarray(offsets, dtype=np.int64)
    row_token = np.asarray(row_token, dtype=np.int64)
    R = int(offsets[-1])
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    H = xh.shape[1]
    # the operand row of every permuted row, masked by its expert's set
    eid = expert_of_rows(offsets, rows)
    a = np.zeros((rows.size, H))
    a_abs = np.zeros((rows.size, H))
    for i, (r, e) in enumerate(zip(rows, eid)):
        t = row_token[r]
        m = np.zeros(H, dtype=bool)
        m[np.asarray(sel_pe[e], dtype=np.int64)] = True
        rr = np.where(m, rh[t], 0.0)
        a[i] = xh[t] - rr
        a_abs[i] = np.abs(xh[t]) + np.abs(rr)
    # rows are evaluated in their own order: a dense product per expert
    N = w13["codes"].shape[1]
    out = np.zeros((rows.size, N))
    mag = np.zeros((rows.size, N))
    for e in np.unique(eid):
        pick = np.nonzero(eid == e)[0]
        W = dequant_bank_f64(w13, int(e))
        out[pick] = a[pick] @ W.T
        mag[pick] = a_abs[pick] @ np.abs(W).T
    return out, mag


def silu(g):
    g = np.asarray(g, dtype=np.float64)
    return g / (1.0 + np.exp(-g))


def swiglu(gu, I):
    """L4 epilogue: h = bf16(silu(g) * u), float64 before the one rounding."""
    g = gu[:, :I]
    u = gu[:, I:2 * I]
    return bf16_round_f64(silu(g) * u)


def w2_stage(hq, offsets, w2, rows=None, rq=None):
    """A8: z = h_hat W2_hat[e]^T for the permuted rows.  rq (L6): the masked
    residual of h, subtracted from h_hat before the contraction; the abs-sum
    then counts both terms."""
    hh = quant.dequantize_f64(hq["codes"], hq["scales"], hq["s_dec"])
    if rq is None:
        return grouped_gemm(hh, None, offsets, w2, rows=rows)
    rh = quant.dequantize_f64(rq["codes"], rq["scales"], rq["s_dec"])
    return grouped_gemm(hh - rh, None, offsets, w2, rows=rows, a_abs_src=np.abs(hh) + np.abs(rh))


def combine(z, inv_row, w, tokens=None):
    """A9: y[t] = sum_s w[t, s] z[inv_row[t, s]] (float64).

    Returns (y, abssum) for the requested tokens (default all)."""
    inv_row = np.asarray(inv_row, dtype=np.int64)
    w = np.asarray(w, dtype=np.float64)
    T, k = inv_row.shape
    tokens = np.arange(T) if tokens is None else np.asarray(tokens, dtype=np.int64)
    z = np.asarray(z, dtype=np.float64)
    y = np.zeros((tokens.size, z.shape[1]), dtype=np.float64)
    mag = np.zeros_like(y)
    for s in range(k):
        zz = z[inv_row[tokens, s]]
        y += w[tokens, s][:, None] * zz
        mag += np.abs(w[tokens, s][:, None] * zz)
    return y, mag


def moe_layer(x, logits, w13, w2, k, Ks, renorm=True, Ks2=0, per_expert=False):
    """Free-running forward of the whole layer (A1-A9).

    x: float32 [T][H] (bf16-valued); logits float32 [T][E];
    w13 / w2: quantised banks from quant.quantize_weight_bank;
    Ks2: channels of h compensated at the W2 input (L6; 0: none);
    per_expert: one channel set per expert at the W13 input (L7).
    Returns a dict of every intermediate.
    """
    x = np.asarray(x, dtype=np.float32)
    T, H = x.shape
    E = logits.shape[1]
    I = w13["codes"].shape[1] // 2
    ids = route.topk_fast(logits, k)
    wts = route.weights(logits, ids, renorm)
    perm = route.permute(ids, E)
    if per_expert:
        act = rac.rac_activation_per_expert(x, Ks, perm["row_token"], perm["offsets"])
        gu, gu_mag = w13_stage_per_expert(act["xq"], act["rq"], act["sel_pe"], perm["row_token"],
                                          perm["offsets"], w13)
    else:
        act = rac.rac_activation(x, Ks)
        gu, gu_mag = w13_stage(act["xq"], act["rq"], perm["row_token"], perm["offsets"], w13)
    h = swiglu(gu, I)
    if Ks2 > 0:
        act2 = rac.rac_activation(h.astype(np.float32), Ks2)
        hq, rq2 = act2["xq"], act2["rq"]
    else:
        act2, hq, rq2 = None, quant.quantize(h.astype(np.float32)), None
    z, z_mag = w2_stage(hq, perm["offsets"], w2, rq=rq2)
    zb = bf16_round_f64(z)
    y, y_mag = combine(zb, perm["inv_row"], wts)
    return dict(ids=ids, w=wts, **perm, act=act, gu=gu, gu_mag=gu_mag, h=h,
                hq=hq, act2=act2, z=z, zb=zb, z_mag=z_mag, y=y, y_mag=y_mag,
                yb=bf16_round_f64(y))

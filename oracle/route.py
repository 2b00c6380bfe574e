"""Top-k expert routing and the token -> expert-row permutation.

The paper names the MoE layer (Sec. 3.3, the "W13" gate/up projection; the
MoE 25B-A2.8B model of Sec. 4.1) but does not specify its router.  Reading
used here (parity unpinned by the paper; pinned by brute force in the tests):

  L1  ids[t] = the k largest logits of token t, ordered by (logit desc,
      expert index asc): ties go to the lower expert index.
  L2  renorm = 1: w[t, s] = exp(l_s - l_max) / sum over the k selected
      (softmax renormalised over the selected experts); renorm = 0: the
      full softmax probability over all E experts.
  L3  rows of the grouped GEMMs are ordered by (expert asc, token asc);
      offsets = exclusive scan of per-expert counts; row_token[row] is the
      token of a row, inv_row[t, s] the row holding (t, ids[t, s]).
"""

import numpy as np


def topk(logits, k):
    """L1 by brute force: a stable sort of every token's logits."""
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    ids = np.empty((T, k), dtype=np.int32)
    for t in range(T):
        # python's sort is stable, so equal logits keep ascending index order
        order = sorted(range(E), key=lambda e: -float(logits[t, e]))
        ids[t] = order[:k]
    return ids


def topk_fast(logits, k):
    """L1 vectorised (lexsort on (index, -logit)); same result as topk()."""
    logits = np.asarray(logits, dtype=np.float32)
    T, E = logits.shape
    idx = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((idx, -logits.astype(np.float64)), axis=1)
    return order[:, :k].astype(np.int32)


def weights(logits, ids, renorm=True):
    """L2 in float64."""
    logits = np.asarray(logits, dtype=np.float64)
    sel = np.take_along_axis(logits, ids.astype(np.int64), axis=1)
    if renorm:
        m = sel.max(axis=1, keepdims=True)
        ex = np.exp(sel - m)
        return ex / ex.sum(axis=1, keepdims=True)
    m = logits.max(axis=1, keepdims=True)
    ex_all = np.exp(logits - m)
    return np.exp(sel - m) / ex_all.sum(axis=1, keepdims=True)


def permute(ids, E):
    """L3: canonical (expert asc, token asc) row order."""
    ids = np.asarray(ids, dtype=np.int64)
    T, k = ids.shape
    counts = np.bincount(ids.reshape(-1), minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    fill = offsets[:-1].copy()
    row_token = np.empty(T * k, dtype=np.int32)
    inv_row = np.empty((T, k), dtype=np.int32)
    for t in range(T):                 # tokens in ascending order
        for s in range(k):
            e = ids[t, s]
            r = fill[e]
            fill[e] += 1
            row_token[r] = t
            inv_row[t, s] = r
    return dict(counts=counts.astype(np.int32), offsets=offsets.astype(np.int32),
                row_token=row_token, inv_row=inv_row)

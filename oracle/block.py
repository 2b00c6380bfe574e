"""The MoE block's input path ahead of the expert layer: RMSNorm and router.

Test infrastructure: only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg use this package; the library never does.

The paper's rollout model (Sec. 4.1, an MoE transformer) feeds each expert
layer the RMS-normalised hidden state, and its router scores the experts from
that same normalised state; the paper defines neither step.  Readings used
here (parity unpinned by the paper; pinned in the tests by closed forms,
invariants and brute force):

  B1  x[t] = bf16_RNE( h[t] / sqrt(mean_j h[t, j]^2 + eps) * gamma ), in
      float64 with one rounding (the standard RMSNorm; h, gamma bf16-valued).
  B2  logits[t, e] = fp32_RNE( sum_j x[t, j] * w_r[e, j] ), the float64
      contraction of the bf16 x with the bf16 router weights w_r [E][H],
      rounded once to float32 (the routing consumes float32 logits).
  B3  the block output is the expert layer (oracle.layer.moe_layer) on x and
      those logits.
"""

import numpy as np

from . import layer
from .formats import bf16_round_f64


def rmsnorm(h, gamma, eps):
    """B1: float64 RMSNorm of each row, rounded once to bf16 (as float64)."""
    h = np.asarray(h, dtype=np.float64)
    g = np.asarray(gamma, dtype=np.float64)
    ms = np.mean(h * h, axis=1, keepdims=True)
    return bf16_round_f64(h / np.sqrt(ms + float(eps)) * g[None, :])


def router_logits(x, w_r):
    """B2: float64 x w_r^T rounded to float32; also the sum of |products|
    behind each logit (the magnitude a float32 accumulator adds)."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w_r, dtype=np.float64)
    return (x @ w.T).astype(np.float32), np.abs(x) @ np.abs(w).T


def moe_block(h, gamma, eps, w_r, w13, w2, k, Ks, renorm=True, Ks2=0):
    """B1-B3 free-running: the layer's dict plus x and logits."""
    x = rmsnorm(h, gamma, eps)
    lg, _ = router_logits(x, w_r)
    out = layer.moe_layer(x.astype(np.float32), lg, w13, w2, k, Ks, renorm=renorm, Ks2=Ks2)
    out["x"] = x
    out["logits"] = lg
    return out

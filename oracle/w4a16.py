"""The trainer-side forward of QUADS: asymmetric W4A16 (Sec. 3.2, Eq.
(w4a16-qat-forward)).

Test infrastructure only: imported by tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline, never by the library.

The trainer keeps bf16 activations and fake-quantises only the weights with
the same QDQ the rollout side applies (Sec. 3.2, Eq. (weight-qdq-align)):

  T1  W_hat = QDQ_W(W): quant.quantize_weight_bank, dequantised exactly
      (layer.dequant_bank_f64, tensor scale included).
  T2  Y = X W_hat^T for the permuted rows of each expert, X the bf16
      activations taken as they are (no activation quantiser), in float64.
  T3  The MoE layer forward on this side: the routing and permutation of
      the rollout layer (L1-L3), [g; u] = X W13_hat^T, h = bf16(silu(g) u),
      z = bf16(h W2_hat^T), y = bf16(combine) (L4-L5 with no activation
      quantisation and no residual).

The backward pass of the same section (the straight-through estimator) is
not a kernel: the gradient passes W_hat's as W's.

Parity is pinned in tests/test_oracle_w4a16.py: on weights that the NVFP4
grid holds exactly, the forward equals X W^T computed from W itself; the
rows against an exact rational sum; the layer against a per-(token, slot)
loop.
"""

import numpy as np

from . import layer as _layer, route
from .formats import bf16_round_f64


def grouped_gemm(x, row_token, offsets, bank, rows=None):
    """T2: x float32 (bf16-valued) [*][K]; returns (out, abssum) float64."""
    xs = np.asarray(x, dtype=np.float32).astype(np.float64)
    return _layer.grouped_gemm(xs, row_token, offsets, bank, rows=rows)


def moe_layer(x, logits, w13, w2, k, renorm=True):
    """T3: the free-running W4A16 layer forward."""
    x = np.asarray(x, dtype=np.float32)
    E = logits.shape[1]
    I = w13["codes"].shape[1] // 2
    ids = route.topk_fast(logits, k)
    wts = route.weights(logits, ids, renorm)
    perm = route.permute(ids, E)
    gu, gu_mag = grouped_gemm(x, perm["row_token"], perm["offsets"], w13)
    h = _layer.swiglu(gu, I)
    z, z_mag = grouped_gemm(h.astype(np.float32), None, perm["offsets"], w2)
    zb = bf16_round_f64(z)
    y, y_mag = _layer.combine(zb, perm["inv_row"], wts)
    return dict(ids=ids, w=wts, **perm, gu=gu, gu_mag=gu_mag, h=h, z=z, zb=zb, z_mag=z_mag,
                y=y, y_mag=y_mag, yb=bf16_round_f64(y))


__all__ = ["grouped_gemm", "moe_layer"]

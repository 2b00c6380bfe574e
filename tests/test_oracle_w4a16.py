"""Pins for the W4A16 trainer-forward oracle (oracle/w4a16.py, T1-T3).

T1-T2 are pinned on weights that the NVFP4 grid holds exactly: every block
is E2M1 values times a power of two, and one block holds 6 * 448, so the
tensor scale is 1 and the QDQ returns W itself.  The forward must then be
X W^T computed from W directly.  The layer (T3) is pinned against a
per-(token, slot) loop that never builds the permutation.
"""

import numpy as np
import torch

from oracle import formats, layer, quant, route, w4a16

E2M1 = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], dtype=np.float64)


def _bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _grid_bank(rng, E, N, K):
    """Weights on the NVFP4 grid with tensor amax 2688 (s_enc = s_dec = 1)."""
    w = np.empty((E, N, K))
    for e in range(E):
        for n in range(N):
            for b in range(K // 16):
                m = int(rng.integers(-9, 6))
                vals = E2M1[rng.integers(0, 8, 16)] * rng.choice([-1.0, 1.0], 16)
                vals[rng.integers(0, 16)] = 6.0 * rng.choice([-1.0, 1.0])   # block amax 6 * 2^m
                w[e, n, 16 * b:16 * b + 16] = vals * 2.0 ** m
        w[e, 0, :16] = E2M1[rng.integers(0, 8, 16)] * 448.0
        w[e, 0, 3] = 6.0 * 448.0
    return w.astype(np.float32)


def test_forward_on_grid_weights_is_x_times_w():
    rng = np.random.default_rng(5)
    E, N, K, T = 3, 8, 64, 11
    w = _grid_bank(rng, E, N, K)
    bank = quant.quantize_weight_bank(w)
    for e in range(E):
        assert np.array_equal(layer.dequant_bank_f64(bank, e), w[e].astype(np.float64))
        assert bank["gscale"][e].tolist() == [1.0, 1.0]
    x = _bf16(rng.standard_normal((T, K)) * 3)
    offsets = np.array([0, 4, 4, 9])          # expert 1 holds no rows
    row_token = np.array([3, 0, 10, 7, 1, 2, 2, 5, 9])
    out, mag = w4a16.grouped_gemm(x, row_token, offsets, bank)
    for r in range(9):
        e = int(np.searchsorted(offsets, r, side="right") - 1)
        ref = w[e].astype(np.float64) @ x[row_token[r]].astype(np.float64)
        np.testing.assert_allclose(out[r], ref, rtol=1e-13, atol=1e-300)
        assert np.all(mag[r] >= np.abs(out[r]) - 1e-9)


def test_layer_against_brute_force():
    rng = np.random.default_rng(8)
    T, H, E, k, I = 9, 64, 4, 2, 32
    x = _bf16(rng.standard_normal((T, H)))
    logits = rng.standard_normal((T, E)).astype(np.float32)
    w13 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, 2 * I, H)) * 0.05))
    w2 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, H, I)) * 0.05))
    out = w4a16.moe_layer(x, logits, w13, w2, k)
    ids = route.topk(logits, k)
    wts = route.weights(logits, ids, True)
    y = np.zeros((T, H))
    for t in range(T):
        for s in range(k):
            e = ids[t, s]
            gu = layer.dequant_bank_f64(w13, e) @ x[t].astype(np.float64)
            g, u = gu[:I], gu[I:]
            h = formats.bf16_round_f64(g / (1 + np.exp(-g)) * u)
            z = formats.bf16_round_f64(layer.dequant_bank_f64(w2, e) @ h)
            y[t] += wts[t, s] * z
    assert np.array_equal(out["ids"], ids)
    np.testing.assert_allclose(out["y"], y, rtol=1e-12, atol=1e-15)

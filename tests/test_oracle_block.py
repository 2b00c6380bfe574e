"""Pins for the block input path (oracle.block, readings B1-B3): RMSNorm by
closed forms, exact power-of-two scale invariance and a per-row brute force
with exactly rounded sums; the router by exact rational sums."""

import math
from fractions import Fraction

import numpy as np
import torch

from oracle import block, quant, route


def _bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).to(torch.float32).numpy()


def _bf16_of_f64(v):
    """One rounding float64 -> bf16 (torch's direct conversion)."""
    return torch.tensor(v, dtype=torch.float64).to(torch.bfloat16).to(torch.float64).numpy()


def test_rmsnorm_closed_forms():
    gamma = np.array([1.0, 0.5, -2.0, 3.0, 0.09375, -0.75, 1.5, 2.0])
    # a constant row c has RMS |c|: x = sign(c) * gamma (eps = 0)
    for c in (1.0, -3.0, 0.0625, 448.0):
        x = block.rmsnorm(np.full((1, 8), c), gamma, 0.0)
        assert np.array_equal(x[0], np.sign(c) * gamma)
    # eps enters under the root: RMS 1 with eps 3 halves the row
    x = block.rmsnorm(np.ones((1, 8)), gamma, 3.0)
    assert np.array_equal(x[0], gamma / 2)
    # [3, 4]: mean square 12.5, x = [3, 4] * sqrt(2) / 5
    x = block.rmsnorm(np.array([[3.0, 4.0]]), np.ones(2), 0.0)
    want = _bf16_of_f64([3 * math.sqrt(2) / 5, 4 * math.sqrt(2) / 5])
    assert np.array_equal(x[0], want)
    assert x[0, 0] != x[0, 1]


def test_rmsnorm_power_of_two_invariance():
    rng = np.random.default_rng(3)
    h = _bf16(rng.standard_normal((6, 48)) * 3)
    g = _bf16(1 + 0.1 * rng.standard_normal(48))
    x0 = block.rmsnorm(h, g, 0.0)
    for j in (-4, -1, 3, 7):
        assert np.array_equal(block.rmsnorm(h * 2.0 ** j, g, 0.0), x0)
    # a dropped mean (sum instead of mean) or a missing root breaks this
    assert not np.array_equal(block.rmsnorm(h * 3.0, g, 1.0), block.rmsnorm(h, g, 1.0))


def test_rmsnorm_unit_rms():
    rng = np.random.default_rng(4)
    h = _bf16(rng.standard_normal((16, 256)) * 5 + 1)
    x = block.rmsnorm(h, np.ones(256), 0.0)
    ms = np.mean(x * x, axis=1)
    assert np.all(np.abs(ms - 1.0) < 2.0 ** -7)


def test_rmsnorm_brute_force():
    rng = np.random.default_rng(5)
    T, H = 5, 24
    h = _bf16(rng.standard_normal((T, H)) * 2)
    g = _bf16(1 + 0.2 * rng.standard_normal(H))
    eps = 1e-5
    x = block.rmsnorm(h, g, eps)
    for t in range(T):
        # exactly rounded sum of squares; then the same float64 root and
        # products, one rounding to bf16
        ms = math.fsum(float(v) * float(v) for v in h[t]) / H
        r = math.sqrt(ms + eps)
        want = _bf16_of_f64([float(h[t, j]) / r * float(g[j]) for j in range(H)])
        assert np.array_equal(x[t], want), t


def test_router_exact_rational():
    rng = np.random.default_rng(6)
    T, H, E = 4, 16, 5
    x = _bf16(rng.standard_normal((T, H)))
    w = _bf16(rng.standard_normal((E, H)) * 0.1)
    lg, mag = block.router_logits(x, w)
    assert lg.dtype == np.float32
    for t in range(T):
        for e in range(E):
            s = sum(Fraction(float(x[t, j])) * Fraction(float(w[e, j])) for j in range(H))
            assert lg[t, e] == np.float32(float(s)), (t, e)
            m = sum(abs(Fraction(float(x[t, j])) * Fraction(float(w[e, j]))) for j in range(H))
            assert mag[t, e] == float(m)


def test_block_routes_on_its_logits():
    rng = np.random.default_rng(7)
    T, H, E, k, I = 9, 32, 4, 2, 16
    h = _bf16(rng.standard_normal((T, H)))
    g = _bf16(1 + 0.1 * rng.standard_normal(H))
    wr = _bf16(rng.standard_normal((E, H)) * 0.2)
    w13 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, 2 * I, H)) * 0.05))
    w2 = quant.quantize_weight_bank(_bf16(rng.standard_normal((E, H, I)) * 0.05))
    out = block.moe_block(h, g, 1e-6, wr, w13, w2, k, Ks=4)
    assert np.array_equal(out["ids"], route.topk(out["logits"], k))
    assert np.array_equal(out["x"], block.rmsnorm(h, g, 1e-6))

"""GPU parity of the block entry point (qd_moe_block_forward): RMSNorm and the
router folded into the layer's first launch (oracle.block, readings B1-B3).

x and the logits are float32 arithmetic on the GPU against the float64
readings: x within one bf16 ulp (nearly all elements equal), the logits
within a float32 accumulation bound.  The routing is checked bit for bit
against the oracle's top-k of the GPU's own logits, and everything after
that against the plain layer (qd_moe_layer_forward) on the GPU's x and
logits, bit for bit; the free-running output against the oracle's block.
"""

import zlib

import numpy as np
import pytest
import torch

from oracle import block as OB, route as ORt
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import np_bf16, oracle_bank

pytestmark = pytest.mark.gpu

DEV = "cuda"
EPS = 1e-6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


def _ulp_diff(a, b):
    """|a - b| in bf16 units of the last place (same-sign values)."""
    ia = a.contiguous().view(torch.int16).to(torch.int32)
    ib = b.contiguous().view(torch.int16).to(torch.int32)
    # map the sign-magnitude bit patterns to a monotone integer line
    fa = torch.where(ia < 0, -(ia & 0x7FFF), ia)
    fb = torch.where(ib < 0, -(ib & 0x7FFF), ib)
    return (fa - fb).abs()


def _check_x_logits(h, gamma, w_r, v, rows=None):
    hf = np_bf16(h if rows is None else h[rows])
    x_or = OB.rmsnorm(hf, np_bf16(gamma), EPS)
    xg = v["x"] if rows is None else v["x"][rows]
    d = _ulp_diff(xg.cpu(), torch.from_numpy(x_or).to(torch.bfloat16))
    assert int(d.max()) <= 1, f"x: {int(d.max())} ulp"
    assert float((d == 0).float().mean()) >= 0.99
    # the logits on the GPU's own x: float32 accumulation of bf16 products
    lg_or, mag = OB.router_logits(np_bf16(xg), np_bf16(w_r))
    lg = v["logits"] if rows is None else v["logits"][rows]
    lgn = lg.cpu().numpy().astype(np.float64)
    err = np.abs(lgn - lg_or.astype(np.float64))
    assert np.all(err <= 2.0 ** -16 * mag + 2.0 ** -40), float((err / (mag + 1e-30)).max())


CASES = [
    # name, T, H, E, k, I, Ks, Ks2, renorm, kwargs
    ("blk_small", 64, 256, 8, 2, 128, 8, 0, True, {}),
    # T not a multiple of the 32-token block, several column chunks
    ("blk_ragged_t", 100, 512, 16, 4, 96, 24, 0, True, {}),
    ("blk_t1", 1, 256, 8, 2, 128, 8, 0, True, {}),
    # fewer experts than one 32-expert MFMA block; H one chunk
    ("blk_e4", 40, 128, 4, 2, 64, 4, 0, True, {}),
    # H = 16 (a partial chunk only), H = 144 (a chunk and a partial one)
    ("blk_h16", 33, 16, 4, 2, 16, 4, 0, True, {}),
    ("blk_h144", 48, 144, 8, 2, 32, 8, 0, True, {}),
    # E = 256 (two expert blocks per wave), E = 160 (uneven blocks) with
    # RAC at the W2 input and the full softmax
    ("blk_e256", 64, 256, 256, 8, 64, 8, 0, True, {}),
    ("blk_e160_w2rac", 70, 256, 160, 6, 64, 16, 8, False, {}),
    # heavy tails, edge values, zero rows (RMS = sqrt(eps))
    ("blk_edges", 48, 256, 16, 4, 64, 16, 0, True,
     dict(acts="student_t3", edge_cases=True, outlier_frac=0.0)),
    # the widest hidden state the block's LDS rows take (8 tokens x 9200)
    ("blk_h9200", 16, 9200, 8, 2, 32, 8, 0, True, {}),
    # many rows per expert: the tile GEMM
    ("blk_tile", 256, 256, 4, 2, 128, 8, 0, True, {}),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_block_small(case):
    name, T, H, E, k, I, Ks, Ks2, renorm, kw = case
    seed = zlib.crc32(name.encode()) % 1000
    inp = synth.small_moe(name, T, H, E, k, I, Ks, seed=seed, **kw)
    gamma, w_r = synth.block_params(H, E, seed=seed)
    h = inp.x.to(DEV)
    if name == "blk_edges":
        h[3] = 0                              # an all-zero row
    gamma, w_r = gamma.to(DEV), w_r.to(DEV)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    blk = ops.MoEBlock(w13, w2, T, k, Ks, gamma, w_r, eps=EPS, renorm=renorm, Ks2=Ks2)
    y = blk(h)
    torch.cuda.synchronize()
    v = blk.views()
    _check_x_logits(h, gamma, w_r, v)
    # routing: the oracle's top-k and weights of the GPU's logits
    lg = v["logits"].cpu().numpy()
    ids = ORt.topk(lg, k) if T <= 64 else ORt.topk_fast(lg, k)
    assert np.array_equal(v["ids"].cpu().numpy(), ids)
    np.testing.assert_allclose(v["w"].cpu().numpy(), ORt.weights(lg, ids, renorm), rtol=2e-6,
                               atol=1e-7)
    # the rest is the plain layer on that x and those logits, bit for bit
    lay = ops.MoELayer(w13, w2, T, k, Ks, renorm=renorm, Ks2=Ks2)
    y2 = lay(v["x"].clone(), v["logits"].clone())
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
    v2 = lay.views()
    for key in ("ids", "w", "offsets", "row_token", "xq_codes", "xq_scales", "xq_gscale", "sel",
                "h", "hq_codes", "z"):
        assert torch.equal(v[key], v2[key]), key
    # free-running: the oracle's block from h
    full = OB.moe_block(np_bf16(h.cpu()), np_bf16(gamma), EPS, np_bf16(w_r), oracle_bank(inp.w13),
                        oracle_bank(inp.w2), k, Ks, renorm=renorm, Ks2=Ks2)
    assert np.array_equal(full["ids"], v["ids"].cpu().numpy())
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= 1e-3, f"free-running rel-L2 {rel:.3e}"


@pytest.mark.parametrize("name", ["moe_decode_t256_h2048", "moe_prefill_t8192_h2048"])
def test_block_full_size(name):
    """The workload's shapes through the block entry point: x and the logits
    against the readings on every row (decode) or 512 sampled rows
    (prefill), the routing against the oracle's top-k of the GPU logits, and
    the output bit for bit against the plain layer on the GPU's x and
    logits."""
    wl = synth.WORKLOADS[name]
    inp = synth.generate(name)
    T, H, E, k, I, Ks = wl.T, wl.H, wl.E, wl.k, wl.I, wl.Ks
    gamma, w_r = synth.block_params(H, E, seed=wl.index)
    h, gamma, w_r = inp.x.to(DEV), gamma.to(DEV), w_r.to(DEV)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    blk = ops.MoEBlock(w13, w2, T, k, Ks, gamma, w_r, eps=EPS)
    y = blk(h)
    torch.cuda.synchronize()
    v = blk.views()
    rows = None
    if T > 512:
        rows = torch.from_numpy(np.random.default_rng(1).choice(T, 512, replace=False)).to(DEV)
    _check_x_logits(h, gamma, w_r, v, rows)
    lg = v["logits"].cpu().numpy()
    ids = ORt.topk_fast(lg, k)
    assert np.array_equal(v["ids"].cpu().numpy(), ids)
    np.testing.assert_allclose(v["w"].cpu().numpy(), ORt.weights(lg, ids, True), rtol=2e-6,
                               atol=1e-7)
    lay = ops.MoELayer(w13, w2, T, k, Ks)
    y2 = lay(v["x"].clone(), v["logits"].clone())
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))

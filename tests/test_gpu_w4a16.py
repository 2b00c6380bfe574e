"""GPU parity of the trainer-side W4A16 forward (moe_w4a16_grouped_gemm,
Sec. 3.2, Eq. (w4a16-qat-forward)) against oracle/w4a16.py.

The weights are the GPU's NVFP4 bank, checked bit for bit against the
oracle's quantisation first.  Products of bf16 activations and exact
e2m1 * e4m3 weights are exact in f32, so the GEMM is held to the tolerance
of every other NVFP4 contraction (helpers.check_close_bf16: rel-L2 <= 1e-3,
2 bf16 ulp plus 2^-20 * sum|products| per element).
"""

import numpy as np
import pytest
import torch

from oracle import layer as OL, route as ORt, w4a16 as OW
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import assert_bank_equal, bf16_tensor, check_close_bf16, np_bf16, oracle_bank

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


CASES = [
    # name, T, H, E, k, I, kwargs
    ("decode", 64, 256, 8, 2, 128, {}),
    ("prefill", 512, 512, 4, 2, 256, {}),
    ("ragged_zipf", 300, 384, 8, 2, 192, dict(routing="zipf", acts="student_t3")),
    ("one_expert_rows", 200, 128, 16, 4, 64, dict(routing="zipf")),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_w4a16_stages_and_layer(case):
    name, T, H, E, k, I, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, 0, seed=31, **kw)
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    lg = inp.logits.numpy()
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    W13, W2 = oracle_bank(inp.w13), oracle_bank(inp.w2)
    assert_bank_equal(w13, W13, range(E))
    assert_bank_equal(w2, W2, range(E))
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    perm = ORt.permute(ORt.topk_fast(lg, k), E)
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    R = T * k
    xf = np_bf16(inp.x)
    # W13 without and with the SwiGLU epilogue
    gu = ops.w4a16_grouped_gemm(x, w13, R, row_token, offs)
    ref_gu, mag_gu = OW.grouped_gemm(xf, perm["row_token"], perm["offsets"], W13)
    check_close_bf16(np_bf16(gu), ref_gu, mag_gu, "W4A16 [g;u]")
    h = ops.w4a16_grouped_gemm(x, w13, R, row_token, offs, Q.QD_EPI_SWIGLU)
    ref_h = OL.silu(ref_gu[:, :I]) * ref_gu[:, I:]
    mag_h = (np.abs(OL.silu(ref_gu[:, :I])) * mag_gu[:, I:] +
             1.1 * np.abs(ref_gu[:, I:]) * mag_gu[:, :I])
    check_close_bf16(np_bf16(h), ref_h, mag_h, "W4A16 h")
    # W2 on the oracle's h (no gather)
    h_or = OL.swiglu(ref_gu, I).astype(np.float32)
    z = ops.w4a16_grouped_gemm(bf16_tensor(h_or), w2, R, None, offs)
    ref_z, mag_z = OW.grouped_gemm(h_or, None, perm["offsets"], W2)
    check_close_bf16(np_bf16(z), ref_z, mag_z, "W4A16 z")
    # the layer forward, free-running
    y = ops.W4A16MoELayer(w13, w2, k)(x, logits)
    full = OW.moe_layer(xf, lg, W13, W2, k)
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= 1e-3, f"W4A16 layer rel-L2 {rel:.3e}"


def test_w4a16_full_size_sampled_rows():
    """The prefill workload's shapes (T=8192, H=2048, E=128, k=8, I=768) with
    three experts carrying real weights; their rows are checked."""
    name = "moe_prefill_t8192_h2048"
    wl = synth.WORKLOADS[name]
    lg = synth.generate(name, with_weights=False).logits.numpy()
    perm = ORt.permute(ORt.topk_fast(lg, wl.k), wl.E)
    counts = np.diff(perm["offsets"])
    nz = np.nonzero(counts)[0]
    S = sorted({int(nz[np.argmax(counts[nz])]), int(nz[np.argmin(counts[nz])]), int(nz[len(nz) // 2])})
    inp = synth.generate(name, experts=S)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    W13 = oracle_bank(inp.w13, S)
    assert_bank_equal(w13, W13, S)
    x = inp.x.to(DEV)
    ids, wts, offs, row_token, inv_row = ops.route_permute(inp.logits.to(DEV), wl.k)
    R = wl.T * wl.k
    h = ops.w4a16_grouped_gemm(x, w13, R, row_token, offs, Q.QD_EPI_SWIGLU)
    rows = np.concatenate([np.arange(perm["offsets"][e], perm["offsets"][e + 1]) for e in S])
    gu, mag = OW.grouped_gemm(np_bf16(inp.x), perm["row_token"], perm["offsets"], W13, rows=rows)
    I = wl.I
    ref_h = OL.silu(gu[:, :I]) * gu[:, I:]
    mag_h = np.abs(OL.silu(gu[:, :I])) * mag[:, I:] + 1.1 * np.abs(gu[:, I:]) * mag[:, :I]
    check_close_bf16(np_bf16(h[torch.from_numpy(rows).to(DEV)]), ref_h, mag_h, "W4A16 h (sampled)")

"""GPU parity of the MXFP4 W4A4 comparison layer against its oracle
(oracle/mxfp4.py).

Codes and E8M0 scale bytes must match bit for bit.  Each GEMM stage is fed
the oracle's own quantised operands and passes helpers.check_close_bf16.
That is 2 bf16 ulp plus FLOOR_MX * sum|products|: the scaled MFMA's
accumulation of E2M1 products stays at float32 level, unlike its E4M3 path.
The whole layer runs free and is held to a relative L2 bound, because h
carries one scale per 32-block; a one-ulp difference in h moves a block's
codes.
"""

import numpy as np
import pytest
import torch

from oracle import mxfp4 as OM, layer as OL, route as ORt
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import bf16_tensor, check_close_bf16, np_bf16

pytestmark = pytest.mark.gpu

DEV = "cuda"
FLOOR_MX = 2.0 ** -18
REL_L2_MX_LAYER = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


def test_mxfp4_quantize_rows_exact():
    rng = np.random.default_rng(21)
    x = (rng.standard_t(3, size=(37, 320)) * np.exp(rng.normal(0, 3, size=(37, 1)))).astype(np.float32)
    x[3] = 0.0                                   # zero blocks: byte 0, codes 0
    x[4, :] = -0.0                               # negative zeros keep their sign
    x[5, :32] = np.float32(6.0)                  # all equal, X = 1
    x[6, 40] = np.float32(3e38)                  # near the float32 top
    x[7, :] *= np.float32(1e-39)                 # subnormal inputs
    x[8, 64:96] = np.array([6, .25, .75, 1.25, 1.75, 2.5, 3.5, 5, 7] + [0] * 23, np.float32)
    for t in (torch.from_numpy(x).to(DEV), torch.from_numpy(x).to(torch.bfloat16).to(DEV)):
        codes, scales = ops.mxfp4_quantize_rows(t)
        rc, rs = OM.quantize_rows(t.float().cpu().numpy())
        assert np.array_equal(scales.cpu().numpy(), rs)
        assert np.array_equal(codes.cpu().numpy(), rc)


CASES = [
    # name, T, H, E, k, I, kwargs: 32-row passes (decode) and 256-row tiles
    ("decode", 64, 256, 8, 2, 256, {}),
    ("decode_zipf", 96, 512, 8, 4, 256, dict(routing="zipf")),
    ("prefill", 512, 256, 4, 2, 256, {}),
    ("prefill_ragged", 300, 512, 4, 2, 384, dict(routing="zipf", acts="student_t3")),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_mxfp4_layer_stagewise(case):
    name, T, H, E, k, I, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, 0, seed=17, **kw)
    lg = inp.logits.numpy()
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    w13c, w13s = ops.mxfp4_quantize_rows(inp.w13.to(DEV))
    w2c, w2s = ops.mxfp4_quantize_rows(inp.w2.to(DEV))
    B13 = OM.quantize_bank(inp.w13.float().numpy())
    B2 = OM.quantize_bank(inp.w2.float().numpy())
    assert np.array_equal(w13c.cpu().numpy(), B13["codes"])
    assert np.array_equal(w13s.cpu().numpy(), B13["scales"])
    assert np.array_equal(w2c.cpu().numpy(), B2["codes"])
    assert np.array_equal(w2s.cpu().numpy(), B2["scales"])
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    perm = ORt.permute(ORt.topk_fast(lg, k), E)
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    R = T * k
    # W13 + SwiGLU on the (identical) activation codes
    xf = np_bf16(inp.x)
    xc, xs = ops.mxfp4_quantize_rows(x)
    rc, rs = OM.quantize_rows(xf)
    assert np.array_equal(xc.cpu().numpy(), rc)
    assert np.array_equal(xs.cpu().numpy(), rs)
    h = ops.mxfp4_grouped_gemm(xc, xs, w13c, w13s, R, row_token, offs, Q.QD_EPI_SWIGLU)
    gu, mag = OM.grouped_gemm(rc, rs, perm["row_token"], perm["offsets"], B13)
    ref_h = OL.silu(gu[:, :I]) * gu[:, I:]
    mag_h = np.abs(OL.silu(gu[:, :I])) * mag[:, I:] + 1.1 * np.abs(gu[:, I:]) * mag[:, :I]
    check_close_bf16(np_bf16(h), ref_h, mag_h, "mxfp4 h", floor=FLOOR_MX)
    # W2 on the oracle's quantised h
    h_or = OL.swiglu(gu, I).astype(np.float32)
    hc_or, hs_or = OM.quantize_rows(h_or)
    z = ops.mxfp4_grouped_gemm(torch.from_numpy(hc_or).to(DEV), torch.from_numpy(hs_or).to(DEV),
                               w2c, w2s, R, None, offs)
    ref_z, mag_z = OM.grouped_gemm(hc_or, hs_or, None, perm["offsets"], B2)
    check_close_bf16(np_bf16(z), ref_z, mag_z, "mxfp4 z", floor=FLOOR_MX)
    # the whole layer, free-running
    lay = ops.MXFP4MoELayer(w13c, w13s, w2c, w2s, T, k)
    y = lay(x, logits)
    full = OM.moe_layer(xf, lg, B13, B2, k)
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= REL_L2_MX_LAYER, f"mxfp4 layer rel-L2 {rel:.3e}"


@pytest.mark.parametrize("name", ["moe_decode_t256_h2048", "moe_zipf_decode_t64_h4096"])
def test_mxfp4_full_size_decode(name):
    """A decode workload at full size (T=256, H=2048, E=128, I=768; and the
    Zipf-routed T=64, H=4096, I=1536 one with heavy tails and edge values)
    through the layer call the benchmark times; three experts carry real
    weights."""
    wl = synth.WORKLOADS[name]
    lg = synth.generate(name, with_weights=False).logits.numpy()
    perm = ORt.permute(ORt.topk_fast(lg, wl.k), wl.E)
    counts = np.diff(perm["offsets"])
    nz = np.nonzero(counts)[0]
    S = sorted({int(nz[np.argmax(counts[nz])]), int(nz[np.argmin(counts[nz])]), int(nz[len(nz) // 2])})
    inp = synth.generate(name, experts=S)
    w13c, w13s = ops.mxfp4_quantize_rows(inp.w13.to(DEV))
    w2c, w2s = ops.mxfp4_quantize_rows(inp.w2.to(DEV))
    lay = ops.MXFP4MoELayer(w13c, w13s, w2c, w2s, wl.T, wl.k)
    y = np_bf16(lay(inp.x.to(DEV), inp.logits.to(DEV)))

    def bank(w):
        E, N, K = w.shape
        zc, zs = OM.quantize_rows(np.zeros((1, K), np.float32))
        out = dict(codes=np.broadcast_to(zc, (E, N, K // 2)).copy(),
                   scales=np.broadcast_to(zs, (E, N, K // 32)).copy())
        for e in S:
            out["codes"][e], out["scales"][e] = OM.quantize_rows(w[e].float().numpy())
        return out

    B13, B2 = bank(inp.w13), bank(inp.w2)
    for e in S:
        assert np.array_equal(w13c[e].cpu().numpy(), B13["codes"][e])
        assert np.array_equal(w13s[e].cpu().numpy(), B13["scales"][e])
    full = OM.moe_layer(np_bf16(inp.x), lg, B13, B2, wl.k)
    yb = full["yb"]
    rel = np.linalg.norm(y - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= REL_L2_MX_LAYER, f"rel-L2 {rel:.3e}"

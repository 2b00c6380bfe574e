"""GPU parity of the FP8 W8A8 comparison layer against the oracle (oracle/fp8.py).

Codes and row scales must match bit for bit; the whole layer is compared
free-running by relative L2.  GEMM outputs pass helpers.check_close_bf16 with
a wider absolute floor than the NVFP4 path: the f8f6f4 MFMA reduces the 64
products of one instruction at less than f32 precision (measured on the
device: +448*448, -448*448 and 62 products of 2^-9 in one 64-element block
give 56 * 2^-9, and the small parity cases show errors up to about
2^-15.5 * sum|products|, where f32 accumulation in any order stays near
2^-18).  The floor here is 2^-13 * sum|products|.
Free-running, h carries one scale per row: a one-ulp difference of a row's
amax (f32 against float64 accumulation) moves every code of that row, so the
layer is held to rel-L2 <= 1e-2 there, the stages to the bars above.
"""

REL_L2_FP8_LAYER = 1e-2

FLOOR_FP8 = 2.0 ** -13

import numpy as np
import pytest
import torch

from oracle import fp8 as OF, layer as OL, route as ORt
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import bf16_tensor, check_close_bf16, np_bf16

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


def test_fp8_quantize_rows_exact():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((37, 320)).astype(np.float32)
    x[3] = 0.0                                   # zero row: dec = 1, codes 0 / 0x80
    x[4, :] = -0.0
    x[5] *= 1e-6                                 # small row: subnormal-range codes after scaling
    x[6, 7] = 3e4                                # one large element: most others subnormal
    x[7] = np.float32(0.5)                       # all equal
    xb = np_bf16(torch.from_numpy(x).to(torch.bfloat16))
    codes, dec = ops.fp8_quantize_rows(bf16_tensor(xb))
    rc, rd = OF.quantize_rows(xb)
    assert np.array_equal(codes.cpu().numpy(), rc)
    assert np.array_equal(dec.cpu().numpy().view(np.uint32), rd.view(np.uint32))
    # f32 input path as well
    codes32, dec32 = ops.fp8_quantize_rows(torch.from_numpy(x).to(DEV))
    rc32, rd32 = OF.quantize_rows(x)
    assert np.array_equal(codes32.cpu().numpy(), rc32)
    assert np.array_equal(dec32.cpu().numpy().view(np.uint32), rd32.view(np.uint32))


FP8_CASES = [
    # name, T, H, E, k, I, kwargs -- few rows per expert (32-row passes) and many
    ("decode", 64, 256, 8, 2, 256, {}),
    ("decode_zipf_passes", 96, 512, 8, 4, 256, dict(routing="zipf")),
    ("prefill", 512, 256, 4, 2, 256, {}),
    ("prefill_ragged", 300, 512, 4, 2, 256, dict(routing="zipf")),
]


@pytest.mark.parametrize("case", FP8_CASES, ids=[c[0] for c in FP8_CASES])
def test_fp8_layer_stagewise(case):
    name, T, H, E, k, I, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, 0, seed=11, **kw)
    lg = inp.logits.numpy()
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    w13c, w13d = ops.fp8_quantize_rows(inp.w13.to(DEV))
    w2c, w2d = ops.fp8_quantize_rows(inp.w2.to(DEV))
    B13 = OF.quantize_bank(inp.w13.float().numpy())
    B2 = OF.quantize_bank(inp.w2.float().numpy())
    assert np.array_equal(w13c.cpu().numpy(), B13["codes"])
    assert np.array_equal(w13d.cpu().numpy().view(np.uint32), B13["dec"].view(np.uint32))
    assert np.array_equal(w2c.cpu().numpy(), B2["codes"])
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    ref_ids = ORt.topk_fast(lg, k)
    perm = ORt.permute(ref_ids, E)
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    R = T * k
    # W13 + SwiGLU on the oracle's (identical) activation codes
    xf = np_bf16(inp.x)
    xc, xd = ops.fp8_quantize_rows(x)
    rc, rd = OF.quantize_rows(xf)
    assert np.array_equal(xc.cpu().numpy(), rc)
    h = ops.fp8_grouped_gemm(xc, xd, w13c, w13d, R, row_token, offs, Q.QD_EPI_SWIGLU)
    gu, mag = OF.grouped_gemm(rc, rd, perm["row_token"], perm["offsets"], B13)
    ref_h = OL.silu(gu[:, :I]) * gu[:, I:]
    mag_h = np.abs(OL.silu(gu[:, :I])) * mag[:, I:] + 1.1 * np.abs(gu[:, I:]) * mag[:, :I]
    check_close_bf16(np_bf16(h), ref_h, mag_h, "fp8 h", floor=FLOOR_FP8)
    # W2 on the oracle's quantised h
    h_or = OL.swiglu(gu, I).astype(np.float32)
    hc_or, hd_or = OF.quantize_rows(h_or)
    z = ops.fp8_grouped_gemm(torch.from_numpy(hc_or).to(DEV), torch.from_numpy(hd_or).to(DEV),
                             w2c, w2d, R, None, offs)
    ref_z, mag_z = OF.grouped_gemm(hc_or, hd_or, None, perm["offsets"], B2)
    check_close_bf16(np_bf16(z), ref_z, mag_z, "fp8 z", floor=FLOOR_FP8)
    # the whole layer, free-running
    lay = ops.FP8MoELayer(w13c, w13d, w2c, w2d, T, k)
    y = lay(x, logits)
    full = OF.moe_layer(xf, lg, B13, B2, k)
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= REL_L2_FP8_LAYER, f"fp8 layer rel-L2 {rel:.3e}"


@pytest.mark.parametrize("name", ["moe_decode_t256_h2048", "moe_zipf_decode_t64_h4096"])
def test_fp8_full_size_decode(name):
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
    w13c, w13d = ops.fp8_quantize_rows(inp.w13.to(DEV))
    w2c, w2d = ops.fp8_quantize_rows(inp.w2.to(DEV))
    lay = ops.FP8MoELayer(w13c, w13d, w2c, w2d, wl.T, wl.k)
    y = np_bf16(lay(inp.x.to(DEV), inp.logits.to(DEV)))

    # the oracle's banks: its quantisation of the sampled experts, and of a
    # zero row for every other one
    def bank(w):
        E, N, K = w.shape
        zc, zd = OF.quantize_rows(np.zeros((1, K), np.float32))
        out = dict(codes=np.broadcast_to(zc, (E, N, K)).copy(),
                   dec=np.broadcast_to(zd, (E, N)).copy())
        for e in S:
            out["codes"][e], out["dec"][e] = OF.quantize_rows(w[e].float().numpy())
        return out

    B13, B2 = bank(inp.w13), bank(inp.w2)
    for e in S + [next(i for i in range(wl.E) if i not in S)]:
        assert np.array_equal(w13c[e].cpu().numpy(), B13["codes"][e])
        assert np.array_equal(w13d[e].cpu().numpy(), B13["dec"][e])
    full = OF.moe_layer(np_bf16(inp.x), lg, B13, B2, wl.k)
    yb = full["yb"]
    rel = np.linalg.norm(y - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= REL_L2_FP8_LAYER, f"rel-L2 {rel:.3e}"

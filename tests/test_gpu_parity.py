"""GPU parity: every step of the HIP path against the CPU oracle.

Codes, scales, tensor scales, routing ids, the permutation and the channel
selection must match bit for bit; contraction outputs must pass the
tolerance of helpers.check_close_bf16 (rel-L2 <= 1e-3 and 2 bf16 ulp per
element plus a 2^-20 * sum|products| floor).  The oracle never consumes a
GPU output: each GPU stage runs either on its own previous stage (and is
compared with the oracle's free-running value) or on the oracle's
intermediate uploaded to the device (so a bit-exact stage sees exactly the
oracle's input).  The whole layer is also compared free-running.
"""

import zlib

import numpy as np
import pytest
import torch

from oracle import layer as OL, quant as OQ, rac as OR, route as ORt
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import (assert_bank_equal, assert_nvfp4_equal, bf16_tensor, check_close_bf16,
                     np_bf16, oracle_bank, upload_nvfp4)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()          # the HIP library must load; there is no fallback
    yield


SMALL = [
    # name, T, H, E, k, I, Ks, kwargs
    ("normal", 64, 256, 8, 2, 128, 8, {}),
    ("ktail", 100, 512, 16, 4, 96, 24, {}),
    ("zipf_t3_edges", 48, 256, 16, 4, 64, 16,
     dict(acts="student_t3", routing="zipf", edge_cases=True, outlier_frac=0.0)),
    ("k1_ragged", 33, 128, 4, 1, 64, 5, {}),
    ("k_eq_E", 20, 128, 4, 4, 32, 128, {}),
    ("ks0", 40, 256, 8, 2, 64, 0, {}),
    ("ks1", 40, 256, 8, 2, 64, 1, {}),
    # the decode kernel's down projection (K = I a multiple of 256), experts
    # needing several 64-row passes, and workgroups running several tiles
    ("skinny_w2", 64, 256, 8, 2, 256, 8, {}),
    ("skinny_passes_zipf", 160, 256, 8, 2, 256, 8, dict(routing="zipf")),
    ("skinny_multitile", 64, 1024, 128, 4, 512, 16, {}),
    # many rows per expert and weight rows a multiple of 256: the 256 x 256
    # tile kernel (several n-tiles, partial m-tiles, skewed routing)
    ("tile", 256, 256, 4, 2, 128, 0, {}),
    ("tile_ragged_zipf", 300, 512, 8, 2, 256, 0, dict(routing="zipf")),
    # the tile kernel with the residual fused in compact form: K_s padded to
    # 16, skewed routing with edge-case activations, and K_s = K
    ("tile_rac", 256, 256, 4, 2, 128, 8, {}),
    ("tile_rac_zipf_edges", 300, 512, 8, 2, 128, 40,
     dict(routing="zipf", acts="student_t3", edge_cases=True, outlier_frac=0.0)),
    ("tile_rac_all", 256, 256, 4, 2, 64, 256, {}),
    # the largest K_s the compact table takes at two workgroups per CU
    ("tile_rac_compact_max", 256, 512, 4, 2, 128, 144, {}),
    # K_s beyond it: the residual as a second pass over K on the masked
    # residual (K_s = 145, K_s = H/2, and a ragged K_s near K with skewed
    # routing and edge values; tile_rac_all above is K_s = K)
    ("tile_rac_dense_145", 256, 512, 4, 2, 128, 145, {}),
    ("tile_rac_dense", 256, 1024, 4, 2, 128, 512, {}),
    ("tile_rac_dense_zipf_edges", 300, 1024, 8, 2, 128, 1000,
     dict(routing="zipf", acts="student_t3", edge_cases=True, outlier_frac=0.0)),
    # N = 2I >= 2048 with the residual in compact form: the layer stages the
    # activations stage-major for the W13 tile GEMM (its h is compared bit for
    # bit with the gathered-row GEMM below)
    ("tile_rac_staged", 256, 256, 4, 2, 1024, 8, {}),
    ("tile_rac_staged_zipf", 300, 512, 8, 2, 1024, 40, dict(routing="zipf")),
    # the dense residual pass after a staged first pass (the second pass reads
    # the masked residual by gathered row)
    ("tile_rac_dense_staged", 256, 256, 4, 2, 1024, 200, {}),
    # K = 384, not a multiple of 256: no A-scale ring (every stage loads its
    # own activation scales) in each tile form
    ("tile_k384", 300, 384, 4, 2, 128, 0, {}),
    ("tile_rac_k384", 300, 384, 4, 2, 128, 12, {}),
    ("tile_rac_dense_k384", 300, 384, 4, 2, 128, 200, {}),
    # H > 4096 at decode shapes: the one-workgroup selection and the separate
    # masked-residual pass instead of the fused selection by rank
    ("wide_h_resq", 16, 5120, 4, 2, 64, 40, {}),
    # many rows per expert: the tiled (prefill) kernel instead of the skinny one
    ("many_rows", 256, 256, 4, 2, 64, 8, {}),
    ("many_rows_ktail", 300, 384, 4, 2, 96, 12, {}),
    # a single token (single-sequence decode), and the narrowest width the
    # format allows (one 16-element block per row: H = I = 16)
    ("t1", 1, 256, 8, 2, 128, 8, {}),
    ("t1_k8_ks0", 1, 512, 16, 8, 64, 0, {}),
    ("h16_i16", 40, 16, 4, 2, 16, 4, {}),
    ("h16_t1", 1, 16, 4, 2, 16, 16, {}),
    ("h16_i48_zipf", 64, 16, 8, 4, 48, 3, dict(routing="zipf", acts="student_t3")),
]


def _run_small(case):
    name, T, H, E, k, I, Ks, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, Ks, seed=zlib.crc32(name.encode()) % 1000, **kw)
    return inp


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_layer_stagewise_small(case):
    name, T, H, E, k, I, Ks, _ = case
    inp = _run_small(case)
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    if name == "k1_ragged":
        logits[:, 2] = -1e4         # expert 2 receives no token
    lg = logits.cpu().numpy()
    # A0: weights (the oracle quantises its own banks)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    W13, W2 = oracle_bank(inp.w13), oracle_bank(inp.w2)
    assert_bank_equal(w13, W13, range(E))
    assert_bank_equal(w2, W2, range(E))
    # A1-A2
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    ref_ids = ORt.topk(lg, k)
    assert np.array_equal(ids.cpu().numpy(), ref_ids)
    perm = ORt.permute(ref_ids, E)
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    assert np.array_equal(row_token.cpu().numpy(), perm["row_token"])
    assert np.array_equal(inv_row.cpu().numpy(), perm["inv_row"])
    ref_w = ORt.weights(lg, ref_ids, True)
    np.testing.assert_allclose(wts.cpu().numpy(), ref_w, rtol=2e-6, atol=1e-7)
    if name == "k1_ragged":
        assert perm["counts"][2] == 0
    # A3-A5
    xf = np_bf16(inp.x)
    xq, scores, ramax = ops.quantize_act(x, rac=True)
    act = OR.rac_activation(xf, Ks)
    assert_nvfp4_equal(xq, act["xq"], "xq")
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores"])
    assert ramax.item() == np.max(np.abs(act["r"]))
    sel, rq, _, _ = ops.select_channels(x, xq, Ks, scores, ramax)
    assert np.array_equal(sel.cpu().numpy(), act["sel"])
    assert_nvfp4_equal(rq, act["rq"], "rq")
    # the compact residual: exact unscaled values at the selected channels
    rq_sel = ops.gather_selected(rq, sel).float().cpu().numpy()
    ref_un = OQ.dequantize_unscaled_f64(act["rq"]["codes"], act["rq"]["scales"])
    assert rq_sel.shape == (T, (Ks + 15) // 16 * 16)
    assert np.array_equal(rq_sel[:, :Ks].astype(np.float64), ref_un[:, act["sel"]])
    assert not rq_sel[:, Ks:].any()
    # the unfused score pass gives the same statistics
    sel2, rq2, sc2, ra2 = ops.select_channels(x, xq, Ks)
    assert np.array_equal(sc2.cpu().numpy(), scores.cpu().numpy())
    assert ra2.item() == ramax.item()
    assert np.array_equal(sel2.cpu().numpy(), sel.cpu().numpy())
    # A6 without the epilogue: [g; u] against the float64 contraction
    R = T * k
    if name.startswith("tile_rac"):
        # the tile kernel's dense residual mode reads the masked residual, the
        # compact one rq_sel
        form = Q.lib().moe_w4a4_grouped_gemm_residual_form(R, 2 * I, H, E, Ks, Q.QD_EPI_SWIGLU)
        dense = name.startswith("tile_rac_dense") or name == "tile_rac_all"
        assert form == (1 if dense else 2)
    gu, _ = ops.grouped_gemm(xq, w13, R, row_token, offs, rq if Ks else None,
                             sel if Ks else None, Q.QD_EPI_NONE)
    ref_gu, mag_gu = OL.w13_stage(act["xq"], act["rq"] if Ks else None, perm["row_token"],
                                  perm["offsets"], W13)
    check_close_bf16(np_bf16(gu), ref_gu, mag_gu, "W13 [g;u]")
    # A6 with SwiGLU against silu(g)*u of the float64 g, u
    h, hamax = ops.grouped_gemm(xq, w13, R, row_token, offs, rq if Ks else None,
                                sel if Ks else None, Q.QD_EPI_SWIGLU, want_amax=True)
    hf = np_bf16(h)
    ref_h = OL.silu(ref_gu[:, :I]) * ref_gu[:, I:]
    mag_h = (np.abs(OL.silu(ref_gu[:, :I])) * mag_gu[:, I:] +
             1.1 * np.abs(ref_gu[:, I:]) * mag_gu[:, :I])
    check_close_bf16(hf, ref_h, mag_h, "h (SwiGLU)")
    assert hamax.max().item() == np.max(np.abs(hf))
    # the GEMM's amax partials give the same quantisation as a fresh amax pass
    hq_gpu, _, _ = ops.quantize_act(h, amax_partials=hamax)
    hq_gpu2, _, _ = ops.quantize_act(h)
    assert torch.equal(hq_gpu.codes, hq_gpu2.codes) and torch.equal(hq_gpu.scales, hq_gpu2.scales)
    # A7 on the oracle's h (bit-exact given the same input)
    h_or = OL.swiglu(ref_gu, I).astype(np.float32)
    ref_hq = OQ.quantize(h_or)
    hq, _, _ = ops.quantize_act(bf16_tensor(h_or))
    assert_nvfp4_equal(hq, ref_hq, "hq")
    # A8 on the oracle's hq
    z, _ = ops.grouped_gemm(upload_nvfp4(ref_hq), w2, R, None, offs)
    ref_z, mag_z = OL.w2_stage(ref_hq, perm["offsets"], W2)
    check_close_bf16(np_bf16(z), ref_z, mag_z, "z")
    # A9 on the oracle's z and routing weights
    from oracle.formats import bf16_round_f64
    zb = bf16_round_f64(ref_z)
    w32 = ref_w.astype(np.float32)
    y = ops.unpermute_combine(bf16_tensor(zb), inv_row, torch.from_numpy(w32).to(DEV))
    ref_y, mag_y = OL.combine(zb, perm["inv_row"], w32)
    check_close_bf16(np_bf16(y), ref_y, mag_y, "y")
    # whole layer in one call: identical to the GPU op-by-op sequence
    lay = ops.MoELayer(w13, w2, T, k, Ks)
    y2 = lay(x, logits)
    torch.cuda.synchronize()
    v = lay.views()
    assert torch.equal(v["h"].view(torch.int16), h.view(torch.int16))
    assert torch.equal(v["hq_codes"], hq_gpu.codes[0])
    zg, _ = ops.grouped_gemm(hq_gpu, w2, R, None, offs)
    yg = ops.unpermute_combine(zg, inv_row, wts)
    assert torch.equal(y2.view(torch.int16), yg.view(torch.int16))
    # free-running: the oracle's own layer end to end
    full = OL.moe_layer(xf, lg, W13, W2, k, Ks)
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y2) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= 1e-3, f"free-running rel-L2 {rel:.3e}"


W2RAC = [
    # name, T, H, E, k, I, Ks, Ks2, kwargs: RAC at the W2 input as well
    # (the decode kernel with K = I = 256, the tile kernel with the compact
    # residual, every channel of h, and skewed routing with edge values)
    ("w2rac_skinny", 64, 256, 8, 2, 256, 8, 16, {}),
    ("w2rac_tile", 256, 256, 4, 2, 128, 8, 24, {}),
    ("w2rac_all_ks0", 64, 256, 8, 2, 64, 0, 64, {}),
    ("w2rac_zipf_edges", 300, 512, 8, 2, 128, 40, 20,
     dict(routing="zipf", acts="student_t3", edge_cases=True, outlier_frac=0.0)),
    # many rows per expert at W2 (the tile kernel with the compact residual)
    ("w2rac_prefill_tile", 512, 256, 2, 2, 256, 8, 24, {}),
    # K_s2 = I/2 at W2 with many rows: the tile kernel's dense residual pass
    ("w2rac_prefill_dense", 512, 256, 2, 2, 1024, 8, 512, {}),
]


@pytest.mark.parametrize("case", W2RAC, ids=[c[0] for c in W2RAC])
def test_layer_w2_site_rac(case):
    name, T, H, E, k, I, Ks, Ks2, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, Ks, seed=zlib.crc32(name.encode()) % 1000, **kw)
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    lg = inp.logits.numpy()
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    W13, W2 = oracle_bank(inp.w13), oracle_bank(inp.w2)
    xf = np_bf16(inp.x)
    full = OL.moe_layer(xf, lg, W13, W2, k, Ks, Ks2=Ks2)
    R = T * k
    offs = torch.from_numpy(full["offsets"].astype(np.int32)).to(DEV)
    # A3-A5 at the W2 site on the oracle's h: bit-exact
    h_or = full["h"].astype(np.float32)
    act2 = full["act2"]
    hq, sc, ra = ops.quantize_act(bf16_tensor(h_or), rac=True)
    assert_nvfp4_equal(hq, act2["xq"], "hq")
    assert np.array_equal(sc.cpu().numpy().view(np.uint64), act2["scores"])
    assert ra.item() == np.max(np.abs(act2["r"]))
    sel, hr, _, _ = ops.select_channels(bf16_tensor(h_or), hq, Ks2, sc, ra)
    assert np.array_equal(sel.cpu().numpy(), act2["sel"])
    assert_nvfp4_equal(hr, act2["rq"], "hr")
    # A8 with the residual on the oracle's operands
    sel_or = torch.from_numpy(act2["sel"].astype(np.int32)).to(DEV)
    z, _ = ops.grouped_gemm(upload_nvfp4(act2["xq"]), w2, R, None, offs,
                            upload_nvfp4(act2["rq"]), sel_or)
    ref_z, mag_z = OL.w2_stage(act2["xq"], full["offsets"], W2, rq=act2["rq"])
    check_close_bf16(np_bf16(z), ref_z, mag_z, "z (W2-site RAC)")
    # the layer call equals the GPU op-by-op sequence from its own h
    lay = ops.MoELayer(w13, w2, T, k, Ks, Ks2=Ks2)
    y = lay(x, logits)
    torch.cuda.synchronize()
    v = lay.views()
    hq_g, sc_g, ra_g = ops.quantize_act(v["h"], rac=True)
    sel_g, hr_g, _, _ = ops.select_channels(v["h"], hq_g, Ks2, sc_g, ra_g)
    assert torch.equal(v["hq_codes"], hq_g.codes[0])
    assert torch.equal(v["h_scores"], sc_g)
    assert torch.equal(v["sel2"], sel_g)
    # the W2 residual: in full, or compacted to S where the tile kernel takes
    # it in that form (many rows per expert, I and H multiples of 128,
    # I >= 256, K_s2 small enough for the compact table)
    tile_w2 = Q.lib().moe_w4a4_grouped_gemm_residual_form(R, H, I, E, Ks2, Q.QD_EPI_NONE) == 2
    assert tile_w2 == (name == "w2rac_prefill_tile")
    if tile_w2:
        assert torch.equal(v["hr_sel"], ops.gather_selected(hr_g, sel_g))
    else:
        assert torch.equal(v["hr_codes"], hr_g.codes[0])
        assert torch.equal(v["hr_scales"], hr_g.scales[0])
    zg, _ = ops.grouped_gemm(hq_g, w2, R, None, v["offsets"], hr_g, sel_g)
    yg = ops.unpermute_combine(zg, v["inv_row"], v["w"])
    assert torch.equal(y.view(torch.int16), yg.view(torch.int16))
    # free-running against the oracle's layer
    yb = full["yb"]
    rel = np.linalg.norm(np_bf16(y) - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= 1e-3, f"free-running rel-L2 {rel:.3e}"
    # and the W2-site residual is live: the output differs from K_s2 = 0
    y0 = ops.MoELayer(w13, w2, T, k, Ks)(x, logits)
    assert not torch.equal(y0, y)


ROUTE_CASES = [
    # T, E, k: one workgroup per token (T < 1024), one wave per token
    # (T >= 1024), and the arg-max rounds for E > 256
    (100, 8, 2), (100, 128, 8), (1500, 128, 8), (1100, 256, 6), (1030, 64, 1), (600, 300, 4),
]


@pytest.mark.parametrize("renorm", [True, False])
@pytest.mark.parametrize("T,E,k", ROUTE_CASES)
def test_route_topk_paths(T, E, k, renorm):
    rng = np.random.default_rng(T * 7 + E + k)
    lg = rng.standard_normal((T, E)).astype(np.float32)
    lg[::7, : E // 2] = np.float32(0.5)            # ties, broken by the lower index
    lg[1::9, 0] = np.float32(-0.0)
    lg[1::9, 1] = np.float32(0.0)
    lg[2::11] = np.round(lg[2::11] * 2) / 2        # many equal values
    ids, wts, offs, row_token, inv_row = ops.route_permute(torch.from_numpy(lg).to(DEV), k,
                                                           renorm=renorm)
    ref_ids = ORt.topk(lg, k)
    assert np.array_equal(ids.cpu().numpy(), ref_ids)
    np.testing.assert_allclose(wts.cpu().numpy(), ORt.weights(lg, ref_ids, renorm), rtol=2e-6,
                               atol=1e-7)
    perm = ORt.permute(ref_ids, E)
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    assert np.array_equal(row_token.cpu().numpy(), perm["row_token"])
    assert np.array_equal(inv_row.cpu().numpy(), perm["inv_row"])


@pytest.mark.parametrize("T,k,H", [(5, 1, 8), (64, 8, 2048), (7, 12, 4104), (3, 32, 136),
                                   (70001, 2, 24)])
def test_combine_slot_counts(T, k, H):
    """A9 on its own: k <= 8 (all loads in flight) and the generic loop
    (k > 8), column blocks past one workgroup's 2048 columns, ragged H, and
    more tokens than the grid's 65535 rows (workgroups loop over tokens)."""
    rng = np.random.default_rng(T + k + H)
    R = T * k
    zb = np_bf16(torch.from_numpy(rng.standard_normal((R, H)).astype(np.float32)).to(torch.bfloat16))
    inv = rng.permutation(R).astype(np.int32).reshape(T, k)
    w = rng.random((T, k)).astype(np.float32)
    y = ops.unpermute_combine(bf16_tensor(zb), torch.from_numpy(inv).to(DEV),
                              torch.from_numpy(w).to(DEV))
    ref, mag = OL.combine(zb, inv, w)
    check_close_bf16(np_bf16(y), ref, mag, "combine")


def test_dense_gemm_with_rac():
    """16 tokens x K=256 x N=128, 4 outlier channels x30, RAC on 8 channels."""
    inp = synth.generate("dense_t16_k256_n128")
    wl = inp.wl
    x = inp.x.to(DEV)
    w = ops.quantize_weight(inp.w13.to(DEV))
    W = oracle_bank(inp.w13)
    assert_bank_equal(w, W, [0])
    xq, scores, ramax = ops.quantize_act(x, rac=True)
    act = OR.rac_activation(np_bf16(inp.x), wl.Ks)
    assert_nvfp4_equal(xq, act["xq"], "xq")
    sel, rq, _, _ = ops.select_channels(x, xq, wl.Ks, scores, ramax)
    assert np.array_equal(sel.cpu().numpy(), act["sel"])
    assert_nvfp4_equal(rq, act["rq"], "rq")
    out, _ = ops.grouped_gemm(xq, w, wl.T, rq=rq, sel=sel)
    ref, mag = OL.w13_stage(act["xq"], act["rq"], None, np.array([0, wl.T]), W)
    check_close_bf16(np_bf16(out), ref, mag, "dense")
    # the standalone residual contraction (f32 output) and linearity
    res = ops.residual_gemm(rq, sel, w, wl.T)
    rh = OQ.dequantize_f64(act["rq"]["codes"], act["rq"]["scales"], act["rq"]["s_dec"])
    ref_r, mag_r = OL.grouped_gemm(rh, None, np.array([0, wl.T]), W)
    err = np.abs(res.cpu().numpy() - ref_r)
    assert np.all(err <= 2.0 ** -20 * mag_r + 1e-30)
    plain, _ = ops.grouped_gemm(xq, w, wl.T)
    ref_p, mag_p = OL.w13_stage(act["xq"], None, None, np.array([0, wl.T]), W)
    check_close_bf16(np_bf16(plain), ref_p, mag_p, "dense plain")
    # the RAC output moves toward the unquantised product (expected, reported)
    xf64 = np_bf16(inp.x).astype(np.float64)
    wf = inp.w13[0].float().numpy().astype(np.float64)
    exact = xf64 @ wf.T
    e_rac = np.linalg.norm(np_bf16(out) - exact)
    e_plain = np.linalg.norm(np_bf16(plain) - exact)
    assert e_rac < e_plain


@pytest.mark.parametrize("K,Ks", [(4096, 128), (4096, 4096), (8192, 200), (20480, 333)])
def test_select_sizes(K, Ks):
    """Channel selection and masked residual across the selection kernels'
    size ranges (sorting network up to 4096 channels, radix select above),
    including K_s = K and ties from duplicated columns."""
    rng = np.random.default_rng(K + Ks)
    T = 6
    xf = rng.standard_normal((T, K)).astype(np.float32)
    xf[:, rng.choice(K, size=max(1, K // 100), replace=False)] *= 20.0
    xf[:, 7] = xf[:, 3]           # equal residual columns: ties broken by index
    x = bf16_tensor(xf)
    xb = np_bf16(x)
    xq, scores, ramax = ops.quantize_act(x.to(DEV), rac=True)
    act = OR.rac_activation(xb, Ks)
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores"])
    sel, rq, _, _ = ops.select_channels(x.to(DEV), xq, Ks, scores, ramax)
    assert np.array_equal(sel.cpu().numpy(), act["sel"])
    assert_nvfp4_equal(rq, act["rq"], "rq")


def test_dequantize_modes():
    rng = np.random.default_rng(5)
    w = bf16_tensor(rng.standard_normal((3, 32, 64)) * 0.05)
    q = ops.quantize_weight(w)
    ref = OQ.fake_quant_weight(w.float().cpu().numpy())
    refu = OQ.fake_quant_weight(w.float().cpu().numpy(), unscaled=True)
    d = ops.dequantize(q).cpu().numpy()
    du = ops.dequantize(q, unscaled=True).cpu().numpy()
    assert np.array_equal(d.view(np.uint32), ref.view(np.uint32))
    assert np.array_equal(du.view(np.uint32), refu.view(np.uint32))
    db = ops.dequantize(q, dtype=torch.bfloat16)
    refb = torch.from_numpy(ref).to(torch.bfloat16)
    assert torch.equal(db.cpu().view(torch.int16), refb.view(torch.int16))


def test_quantize_f32_input_and_static_scale():
    rng = np.random.default_rng(6)
    x = (rng.standard_normal((37, 96)) * 3).astype(np.float32)
    xt = torch.from_numpy(x).to(DEV)
    q, _, _ = ops.quantize_act(xt)
    assert_nvfp4_equal(q, OQ.quantize(x), "f32 input")
    amax = torch.tensor([10.0, 250.0, 3.0], device=DEV)
    q2, _, _ = ops.quantize_act(xt, amax_partials=amax)
    assert_nvfp4_equal(q2, OQ.quantize(x, amax=np.float32(250.0)), "static scale")
    big = torch.rand(1000, device=DEV) * 7.0      # more partials than one pass holds
    q3, _, _ = ops.quantize_act(xt, amax_partials=big)
    assert_nvfp4_equal(q3, OQ.quantize(x, amax=np.float32(big.max().item())), "many partials")


def test_quantize_edge_values():
    """The oracle's hand-checked special cases on the GPU: ties, zeros,
    subnormal and underflowing block scales, tiny and zero tensors."""
    import test_oracle_quant as TQ
    row = TQ._worked_row()
    x = np.concatenate([row, -row, row * 0.5], axis=0)
    xt = bf16_tensor(x)
    q, _, _ = ops.quantize_act(xt)
    assert_nvfp4_equal(q, OQ.quantize(np_bf16(xt)), "worked rows")
    z = torch.zeros((4, 32), dtype=torch.bfloat16, device=DEV)
    z[1, :16] = -0.0
    qz, _, _ = ops.quantize_act(z)
    assert_nvfp4_equal(qz, OQ.quantize(np_bf16(z)), "zero tensor")
    tiny = torch.full((2, 16), 2.0 ** -110, dtype=torch.float32, device=DEV)
    qt, _, _ = ops.quantize_act(tiny)
    assert_nvfp4_equal(qt, OQ.quantize(tiny.cpu().numpy()), "tiny tensor")


@pytest.mark.parametrize("e", [-70, -30, 0, 40])
def test_channel_scores_extreme_scales(e):
    """The fixed-point channel scores (Eq. (channel-score), reading R2) at
    tensor scales 2^e: at 2^-70 the squared residuals are float32 subnormals
    whose terms trunc(r^2 * 2^F) are still large (F = 36 - 2 * exponent of
    the tensor amax), at 2^40 F is negative.  Both the fused score pass of the
    quantiser and the standalone one, bit for bit against the oracle."""
    rng = np.random.default_rng(100 + e)
    x = np_bf16(torch.from_numpy(rng.standard_normal((300, 512)).astype(np.float32) *
                                 np.float32(2.0 ** e)).to(torch.bfloat16))
    act = OR.rac_activation(x, 8)
    if e == -70:
        sq = (act["r"] * act["r"]).astype(np.float32)
        assert np.any((sq > 0) & (sq < np.float32(2.0 ** -126)))   # subnormal squares
    xt = bf16_tensor(x)
    xq, scores, ramax = ops.quantize_act(xt, rac=True)
    assert_nvfp4_equal(xq, act["xq"], "xq")
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores"])
    assert ramax.item() == np.max(np.abs(act["r"]))
    sel, rq, sc2, ra2 = ops.select_channels(xt, xq, 8)
    assert np.array_equal(sc2.cpu().numpy().view(np.uint64), act["scores"])
    assert ra2.item() == ramax.item()
    assert np.array_equal(sel.cpu().numpy(), act["sel"])
    assert_nvfp4_equal(rq, act["rq"], "rq")


def test_determinism():
    inp = synth.small_moe("det", 96, 256, 8, 2, 64, 12, seed=7)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    lay = ops.MoELayer(w13, w2, 96, 2, 12)
    x, lg = inp.x.to(DEV), inp.logits.to(DEV)
    y1 = lay(x, lg).clone()
    v1 = {k: t.clone() for k, t in lay.views().items()}
    y2 = lay(x, lg)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    for k, t in lay.views().items():
        a, b = v1[k], t
        if a.dtype == torch.bfloat16:
            a, b = a.view(torch.int16), b.view(torch.int16)
        assert torch.equal(a, b), k


def test_empty_batch():
    inp = synth.small_moe("empty", 4, 128, 4, 2, 32, 4, seed=8)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    lay = ops.MoELayer(w13, w2, 0, 2, 4)
    x = torch.empty((0, 128), dtype=torch.bfloat16, device=DEV)
    lg = torch.empty((0, 4), dtype=torch.float32, device=DEV)
    y = lay(x, lg)
    torch.cuda.synchronize()
    assert y.shape == (0, 128)


FULL = [
    # workload, token count (None: the workload's), experts with real weights
    # ("all": every expert that receives a row; "sampled": three of them),
    # K_s (None: the workload's)
    ("moe_decode_t256_h2048", None, "all", None),
    ("moe_zipf_decode_t64_h4096", None, "all", None),
    ("moe_prefill_t8192_h2048", None, "sampled", None),
    ("moe_prefill_t4096_h4096", None, "sampled", None),
    # a single token (single-sequence decode) at the decode workloads' sizes
    ("moe_decode_t256_h2048", 1, "all", None),
    ("moe_zipf_decode_t64_h4096", 1, "all", None),
    # K_s = H/2 on the prefill workload (the tile kernel's dense residual pass)
    ("moe_prefill_t8192_h2048", None, "sampled", 1024),
]


def _sampled_experts(counts):
    """The most and least loaded non-empty experts and one in between."""
    nz = np.nonzero(counts)[0]
    order = nz[np.argsort(counts[nz], kind="stable")]
    return sorted({int(order[-1]), int(order[0]), int(order[len(order) // 2])})


@pytest.mark.parametrize("name,T,which,ks", FULL,
                         ids=[f"{n}-T{T or 'full'}-{w}" + (f"-ks{ks}" if ks else "")
                              for n, T, w, ks in FULL])
def test_full_size(name, T, which, ks):
    """A MoE workload at its full size (or a single token at its sizes)
    through the whole-layer call the benchmark times (same shapes, hence the
    same kernels and grids).

    "all": every expert that receives a row carries its real weights, so
    every work unit of every kernel is compared with the oracle.  "sampled"
    (the prefill workloads, whose full oracle takes minutes): three experts
    carry their real weights and the rest are zero; the kernels do the same
    work either way, and the zero experts make every output computable by the
    oracle: their rows of h and z and their shares of y are exactly zero, so
    h's tensor amax comes from the sampled rows alone.  Routing, the
    activation quantisation and the channel selection are compared in full,
    bit for bit, in both modes."""
    wl = synth.WORKLOADS[name]
    lg = synth.generate(name, T=T, with_weights=False).logits.numpy()
    ref_ids = ORt.topk_fast(lg, wl.k)
    perm = ORt.permute(ref_ids, wl.E)
    offs_np = perm["offsets"]
    counts = np.diff(offs_np)
    S = [int(e) for e in np.nonzero(counts)[0]] if which == "all" else _sampled_experts(counts)
    zero_e = next((e for e in range(wl.E) if e not in S), None)
    inp = synth.generate(name, T=T, experts=S)
    T = inp.x.shape[0]
    H, E, k, I, Ks = wl.H, wl.E, wl.k, wl.I, (wl.Ks if ks is None else ks)
    R = T * k
    print(f"{name} T={T}: {len(S)} experts with weights, rows "
          f"{sorted(int(counts[e]) for e in S)[-3:]} (largest)", flush=True)

    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    lay = ops.MoELayer(w13, w2, T, k, Ks)
    y = lay(x, logits)
    torch.cuda.synchronize()
    v = lay.views()

    banked = S + ([zero_e] if zero_e is not None else [])
    W13 = oracle_bank(inp.w13, banked)
    W2 = oracle_bank(inp.w2, banked)
    assert_bank_equal(w13, W13, banked)
    assert_bank_equal(w2, W2, banked)
    # A1-A2
    assert np.array_equal(v["ids"].cpu().numpy(), ref_ids)
    assert np.array_equal(v["offsets"].cpu().numpy(), offs_np)
    assert np.array_equal(v["row_token"].cpu().numpy(), perm["row_token"])
    assert np.array_equal(v["inv_row"].cpu().numpy(), perm["inv_row"])
    ref_w = ORt.weights(lg, ref_ids, True)
    np.testing.assert_allclose(v["w"].cpu().numpy(), ref_w, rtol=2e-6, atol=1e-7)
    # A3-A5 in full
    act = OR.rac_activation(np_bf16(inp.x), Ks)
    assert_nvfp4_equal(dict(packed=v["xq_codes"].cpu().numpy(), scales=v["xq_scales"].cpu().numpy(),
                            gscale=v["xq_gscale"].cpu().numpy()), act["xq"], "xq")
    assert np.array_equal(v["scores"].cpu().numpy().view(np.uint64), act["scores"])
    assert v["ramax"].item() == np.max(np.abs(act["r"]))
    assert np.array_equal(v["sel"].cpu().numpy(), act["sel"])
    # the masked residual: in full (decode kernel) or at S only, compacted
    # (prefill kernel), with its tensor scale either way
    assert v["rq_gscale"].cpu().numpy().view(np.uint32).tolist() == \
        np.array([act["rq"]["s_enc"], act["rq"]["s_dec"]], np.float32).view(np.uint32).tolist()
    form = Q.lib().moe_w4a4_grouped_gemm_residual_form(R, 2 * I, H, E, Ks, Q.QD_EPI_SWIGLU)
    if ks is not None:
        assert form == 1       # the dense residual pass reads the masked residual
    if form == 1:
        assert_nvfp4_equal(dict(packed=v["rq_codes"].cpu().numpy(),
                                scales=v["rq_scales"].cpu().numpy(),
                                gscale=v["rq_gscale"].cpu().numpy()), act["rq"], "rq")
    else:
        ref_un = OQ.dequantize_unscaled_f64(act["rq"]["codes"], act["rq"]["scales"])
        got = v["rq_sel"].float().cpu().numpy()
        assert np.array_equal(got[:, :Ks].astype(np.float64), ref_un[:, act["sel"]])
        assert not got[:, Ks:].any()

    # A6 on the rows of the experts with weights; every other row of h is
    # exactly zero
    rows = np.concatenate([np.arange(offs_np[e], offs_np[e + 1]) for e in S])
    other = np.ones(R, bool)
    other[rows] = False
    rows_dev = torch.from_numpy(rows).to(DEV)
    od = torch.from_numpy(other).to(DEV)
    gu, mag_gu = OL.w13_stage(act["xq"], act["rq"] if Ks else None, perm["row_token"], offs_np,
                              W13, rows=rows)
    h_or = OL.swiglu(gu, I)
    mag_h = (np.abs(OL.silu(gu[:, :I])) * mag_gu[:, I:] +
             1.1 * np.abs(gu[:, I:]) * mag_gu[:, :I])
    h_gpu = v["h"]
    check_close_bf16(np_bf16(h_gpu[rows_dev]), h_or, mag_h, "h (SwiGLU)")
    if other.any():
        assert h_gpu[od].abs().max().item() == 0.0

    # A7 on the oracle's h (zero outside the rows with weights), bit-exact; a
    # zero row appended to the oracle's input gives the expected zero rows
    hq_or = OQ.quantize(np.vstack([h_or, np.zeros((1, I))]).astype(np.float32))
    h_full = torch.zeros((R, I), dtype=torch.bfloat16, device=DEV)
    h_full[rows_dev] = bf16_tensor(h_or)
    hq, _, _ = ops.quantize_act(h_full)
    hq_c, hq_s = hq.codes[0], hq.scales[0]
    assert np.array_equal(hq_c[rows_dev].cpu().numpy(), hq_or["packed"][:-1])
    assert np.array_equal(hq_s[rows_dev].cpu().numpy(), hq_or["scales"][:-1])
    if other.any():
        assert bool((hq_c[od] == torch.from_numpy(hq_or["packed"][-1]).to(DEV)).all())
        assert bool((hq_s[od] == torch.from_numpy(hq_or["scales"][-1]).to(DEV)).all())
    assert hq.gscale[0].cpu().numpy().view(np.uint32).tolist() == \
        np.array([hq_or["s_enc"], hq_or["s_dec"]], np.float32).view(np.uint32).tolist()

    # A8 on that hq: the oracle's rows, compacted (row_token maps a row to
    # its place among the rows with weights)
    z, _ = ops.grouped_gemm(hq, w2, R, None, v["offsets"])
    hh = OQ.dequantize_f64(hq_or["codes"][:-1], hq_or["scales"][:-1], hq_or["s_dec"])
    place = np.zeros(R, np.int64)
    place[rows] = np.arange(rows.size)
    z_or, mag_z = OL.grouped_gemm(hh, place, offs_np, W2, rows=rows)
    check_close_bf16(np_bf16(z[rows_dev]), z_or, mag_z, "z")
    if other.any():
        assert z[od].abs().max().item() == 0.0

    # A9 on the oracle's z (zero row appended for the zero experts' rows)
    from oracle.formats import bf16_round_f64
    zb = np.vstack([bf16_round_f64(z_or), np.zeros((1, H))])
    place[other] = rows.size
    w32 = ref_w.astype(np.float32)
    z_full = torch.zeros((R, H), dtype=torch.bfloat16, device=DEV)
    z_full[rows_dev] = bf16_tensor(zb[:-1])
    y_st = ops.unpermute_combine(z_full, v["inv_row"], torch.from_numpy(w32).to(DEV))
    inv_c = place[perm["inv_row"]]
    y_or, mag_y = OL.combine(zb, inv_c, w32)
    check_close_bf16(np_bf16(y_st), y_or, mag_y, "y")

    # free-running: the layer's own y against the oracle's chain
    yb = bf16_round_f64(y_or)
    yg = np_bf16(y)
    rel = np.linalg.norm(yg - yb) / max(np.linalg.norm(yb), 1e-30)
    assert rel <= 1e-3, f"free-running rel-L2 {rel:.3e}"
    untouched = ~np.isin(perm["inv_row"], rows).any(axis=1)
    assert np.all(yg[untouched] == 0.0)


def test_layer_graph_replay():
    """The whole layer captured in a HIP graph: every replay, with eager work
    and synchronisations in between, reproduces the eager output bit for bit
    (the library records no memset nodes; flags and offsets are cleared by
    kernels)."""
    for case in (SMALL[0], next(c for c in SMALL if c[0] == "tile_rac")):
        name, T, H, E, k, I, Ks, _ = case
        inp = _run_small(case)
        x = inp.x.to(DEV)
        logits = inp.logits.to(DEV)
        w13 = ops.quantize_weight(inp.w13.to(DEV))
        w2 = ops.quantize_weight(inp.w2.to(DEV))
        lay = ops.MoELayer(w13, w2, T, k, Ks)
        y_eager = lay(x, logits).clone()
        torch.cuda.synchronize()
        y = torch.empty_like(y_eager)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            lay(x, logits, y)
        for rep in range(3):
            y.zero_()
            lay(x, logits)                 # eager work on the same workspace in between
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y.view(torch.int16), y_eager.view(torch.int16)), (name, rep)


@pytest.mark.parametrize("chans", [tuple(range(64)), (5, 200, 511), (511,), (0, 63, 64, 127, 448)],
                         ids=["one_stage_64", "spread_3", "last_channel", "stage_edges"])
def test_tile_gemm_rac_clustered_selection(chans):
    """The prefill tile GEMM with RAC (2 experts x 256 rows, K=512, N=256)
    when the selected channels crowd into one 64-channel stage, sit at stage
    edges or on the last channel: the compact weight table is filled stage by
    stage (Sec. 3.3, Eq. (residual-recon)).  The planted channels carry x1000
    outliers, so they are the selection."""
    E, T, K, N = 2, 512, 512, 256
    g = torch.Generator().manual_seed(zlib.crc32(repr(chans).encode()))
    x = torch.randn((T, K), generator=g)
    x[:, list(chans)] *= 1000.0
    x = x.to(torch.bfloat16)
    wb = (torch.randn((E, N, K), generator=g) * 0.02).to(torch.bfloat16)
    w = ops.quantize_weight(wb.to(DEV))
    W = oracle_bank(wb)
    assert_bank_equal(w, W, list(range(E)))
    Ks = len(chans)
    xg = x.to(DEV)
    xq, scores, ramax = ops.quantize_act(xg, rac=True)
    act = OR.rac_activation(np_bf16(x), Ks)
    assert_nvfp4_equal(xq, act["xq"], "xq")
    sel, rq, _, _ = ops.select_channels(xg, xq, Ks, scores, ramax)
    assert np.array_equal(sel.cpu().numpy(), act["sel"])
    assert sorted(act["sel"].tolist()) == sorted(chans)
    offsets = np.array([0, 256, 512])
    out, _ = ops.grouped_gemm(xq, w, T, offsets=torch.tensor(offsets, dtype=torch.int32, device=DEV),
                              rq=rq, sel=sel)
    ref, mag = OL.w13_stage(act["xq"], act["rq"], None, offsets, W)
    check_close_bf16(np_bf16(out), ref, mag, f"tile rac {chans[:3]}")

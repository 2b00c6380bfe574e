"""GPU parity of the per-expert RAC channel sets (reading L7: Sec. 3.3's
Eq. (channel-score)/(channel-select) over each expert's own rows).

Per-expert scores, the per-expert selections and the residual quantised over
all channels match the oracle bit for bit; the compact residual rows hold the
exact unscaled values at each row's expert set; the gate/up GEMM with the
per-expert residual passes the G14 tolerance against the oracle's float64
contraction; the whole layer is compared free-running.
"""

import zlib

import numpy as np
import pytest
import torch

from oracle import layer as OL, quant as OQ, rac as OR, route as ORt
from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

from helpers import (assert_bank_equal, assert_nvfp4_equal, bf16_tensor, check_close_bf16, np_bf16,
                     oracle_bank)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


CASES = [
    # name, T, H, E, k, I, Ks, kwargs
    ("pe_small", 64, 256, 8, 2, 128, 8, {}),
    ("pe_zipf_edges", 96, 512, 16, 4, 128, 24,
     dict(routing="zipf", acts="student_t3", edge_cases=True, outlier_frac=0.0)),
    ("pe_many_rows", 512, 256, 4, 2, 128, 40, {}),
    ("pe_ks_eq_k", 64, 256, 4, 2, 128, 256, {}),
    ("pe_empty_expert", 40, 256, 8, 1, 128, 5, {}),
]


def _stages(T, H, E, k, I, Ks, inp, empty=None):
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    if empty is not None:
        logits[:, empty] = -1e4
    lg = logits.cpu().numpy()
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    W13 = oracle_bank(inp.w13)
    assert_bank_equal(w13, W13, range(E))
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    ref_ids = ORt.topk(lg, k)
    perm = ORt.permute(ref_ids, E)
    assert np.array_equal(row_token.cpu().numpy(), perm["row_token"])
    assert np.array_equal(offs.cpu().numpy(), perm["offsets"])
    if empty is not None:
        assert perm["counts"][empty] == 0
    xf = np_bf16(inp.x)
    xq, _, _ = ops.quantize_act(x)
    act = OR.rac_activation_per_expert(xf, Ks, perm["row_token"], perm["offsets"])
    assert_nvfp4_equal(xq, act["xq"], "xq")
    sel_pe, rq, rq_rows, scores, ramax = ops.select_channels_per_expert(x, xq, Ks, row_token, offs)
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores_pe"]), "scores"
    assert ramax.item() == np.max(np.abs(act["r"]))
    assert np.array_equal(sel_pe.cpu().numpy(), act["sel_pe"]), "selection"
    assert_nvfp4_equal(rq, act["rq"], "rq (all channels)")
    # the compact rows: exact unscaled residual at each row's expert set
    R = T * k
    un = OQ.dequantize_unscaled_f64(act["rq"]["codes"], act["rq"]["scales"])
    eid = OL.expert_of_rows(perm["offsets"], np.arange(R))
    ref_rows = np.stack([un[perm["row_token"][r], act["sel_pe"][eid[r]]] for r in range(R)])
    got = rq_rows.float().cpu().numpy()
    assert np.array_equal(got[:, :Ks].astype(np.float64), ref_rows)
    assert not got[:, Ks:].any()
    # W13 [g; u] with the per-expert residual (plain epilogue)
    gu, _ = ops.grouped_gemm_per_expert(xq, w13, R, row_token, offs, rq, sel_pe, rq_rows,
                                        Q.QD_EPI_NONE)
    ref, mag = OL.w13_stage_per_expert(act["xq"], act["rq"], act["sel_pe"], perm["row_token"],
                                       perm["offsets"], W13)
    check_close_bf16(np_bf16(gu), ref, mag, "W13 [g;u] per-expert sets")
    return act


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_per_expert_stages_and_layer(case):
    name, T, H, E, k, I, Ks, kw = case
    inp = synth.small_moe(name, T, H, E, k, I, Ks, seed=zlib.crc32(name.encode()) % 1000, **kw)
    empty = 2 if name == "pe_empty_expert" else None
    _stages(T, H, E, k, I, Ks, inp, empty)
    # the whole layer, free-running against the oracle's
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    if empty is not None:
        logits[:, empty] = -1e4
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    lay = ops.MoELayerPerExpert(w13, w2, T, k, Ks)
    y = lay(x, logits)
    torch.cuda.synchronize()
    ref = OL.moe_layer(np_bf16(inp.x), logits.cpu().numpy(), oracle_bank(inp.w13),
                       oracle_bank(inp.w2), k, Ks, per_expert=True)
    yg = np_bf16(y).astype(np.float64)
    rel = np.linalg.norm(yg - ref["yb"]) / np.linalg.norm(ref["yb"])
    assert rel <= 1e-3, f"layer rel-L2 {rel:.3e}"


@pytest.mark.parametrize("e", [-70, 40])
def test_per_expert_scores_extreme_scales(e):
    """The per-expert scores at tensor scales 2^e (subnormal squared
    residuals at 2^-70, a negative fixed-point shift at 2^40), bit for bit."""
    rng = np.random.default_rng(200 + e)
    T, H, E, k, Ks = 300, 512, 8, 2, 8
    x = bf16_tensor(rng.standard_normal((T, H)).astype(np.float32) * np.float32(2.0 ** e))
    logits = torch.from_numpy(rng.standard_normal((T, E)).astype(np.float32)).to(DEV)
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    perm = ORt.permute(ORt.topk(logits.cpu().numpy(), k), E)
    assert np.array_equal(row_token.cpu().numpy(), perm["row_token"])
    xq, _, _ = ops.quantize_act(x)
    act = OR.rac_activation_per_expert(np_bf16(x), Ks, perm["row_token"], perm["offsets"])
    sel_pe, rq, rq_rows, scores, ramax = ops.select_channels_per_expert(x, xq, Ks, row_token, offs)
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores_pe"])
    assert ramax.item() == np.max(np.abs(act["r"]))
    assert np.array_equal(sel_pe.cpu().numpy(), act["sel_pe"])


def test_per_expert_layer_matches_global_when_one_expert():
    """One expert and k = 1: the per-expert layer and the global layer give
    the same output bit for bit (the sets coincide)."""
    T, H, E, k, I, Ks = 128, 256, 1, 1, 128, 16
    inp = synth.small_moe("pe_one", T, H, E, k, I, Ks, seed=3)
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    y_pe = ops.MoELayerPerExpert(w13, w2, T, k, Ks)(x, logits)
    y_g = ops.MoELayer(w13, w2, T, k, Ks)(x, logits)
    torch.cuda.synchronize()
    ref = OL.moe_layer(np_bf16(inp.x), inp.logits.numpy(), oracle_bank(inp.w13),
                       oracle_bank(inp.w2), k, Ks, per_expert=True)
    for y in (y_pe, y_g):
        yg = np_bf16(y).astype(np.float64)
        assert np.linalg.norm(yg - ref["yb"]) / np.linalg.norm(ref["yb"]) <= 1e-3


@pytest.mark.parametrize("name", ["moe_decode_t256_h2048", "moe_prefill_t8192_h2048"])
def test_per_expert_full_size(name):
    """The selection stages in full at a workload's size (bit-exact), and the
    gate/up GEMM on the rows of three sampled experts (the others carry zero
    weights, whose rows must come out exactly zero)."""
    wl = synth.WORKLOADS[name]
    lg = synth.generate(name, with_weights=False).logits.numpy()
    ref_ids = ORt.topk_fast(lg, wl.k)
    perm = ORt.permute(ref_ids, wl.E)
    counts = np.diff(perm["offsets"])
    nz = np.nonzero(counts)[0]
    order = nz[np.argsort(counts[nz], kind="stable")]
    S = sorted({int(order[-1]), int(order[0]), int(order[len(order) // 2])})
    inp = synth.generate(name, experts=S)
    T, H, E, k, I, Ks = inp.x.shape[0], wl.H, wl.E, wl.k, wl.I, wl.Ks
    R = T * k
    x = inp.x.to(DEV)
    logits = inp.logits.to(DEV)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    W13 = oracle_bank(inp.w13, S)
    assert_bank_equal(w13, W13, S)
    ids, wts, offs, row_token, inv_row = ops.route_permute(logits, k)
    assert np.array_equal(row_token.cpu().numpy(), perm["row_token"])
    xq, _, _ = ops.quantize_act(x)
    act = OR.rac_activation_per_expert(np_bf16(inp.x), Ks, perm["row_token"], perm["offsets"])
    assert_nvfp4_equal(xq, act["xq"], "xq")
    sel_pe, rq, rq_rows, scores, ramax = ops.select_channels_per_expert(x, xq, Ks, row_token, offs)
    assert np.array_equal(scores.cpu().numpy().view(np.uint64), act["scores_pe"])
    assert np.array_equal(sel_pe.cpu().numpy(), act["sel_pe"])
    assert_nvfp4_equal(rq, act["rq"], "rq")
    h, _ = ops.grouped_gemm_per_expert(xq, w13, R, row_token, offs, rq, sel_pe, rq_rows,
                                       Q.QD_EPI_SWIGLU)
    rows = np.concatenate([np.arange(perm["offsets"][e], perm["offsets"][e + 1]) for e in S])
    gu, mag_gu = OL.w13_stage_per_expert(act["xq"], act["rq"], act["sel_pe"], perm["row_token"],
                                         perm["offsets"], W13, rows=rows)
    h_or = OL.swiglu(gu, I)
    mag_h = (np.abs(OL.silu(gu[:, :I])) * mag_gu[:, I:] + 1.1 * np.abs(gu[:, I:]) * mag_gu[:, :I])
    check_close_bf16(np_bf16(h[torch.from_numpy(rows).to(DEV)]), h_or, mag_h, "h per-expert")
    other = np.ones(R, bool)
    other[rows] = False
    if other.any():
        assert h[torch.from_numpy(other).to(DEV)].abs().max().item() == 0.0

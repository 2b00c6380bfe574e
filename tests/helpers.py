"""Shared helpers for the GPU parity tests: conversions from device tensors
to the oracle's numpy representation and the GEMM tolerance check."""

import numpy as np
import torch

from oracle import formats, quant


def np_bf16(t):
    """bf16 torch tensor -> float32 numpy (exact)."""
    return t.detach().float().cpu().numpy()


def nv_host(t):
    """NVFP4Tensor -> dict of numpy arrays (packed codes, scales, gscale)."""
    return dict(packed=t.codes.cpu().numpy(), scales=t.scales.cpu().numpy(),
                gscale=t.gscale.cpu().numpy())


def oracle_nv(q):
    """oracle quantize() result -> (packed, scales, gscale) shaped like the GPU."""
    return q["packed"], q["scales"], np.array([q["s_enc"], q["s_dec"]], np.float32)


def assert_nvfp4_equal(gpu, ref, name=""):
    """Bit-exact comparison of one NVFP4 group: codes, scales, tensor scales."""
    g = nv_host(gpu) if not isinstance(gpu, dict) else gpu
    rp, rs, rg = oracle_nv(ref)
    gp = g["packed"].reshape(rp.shape)
    gs = g["scales"].reshape(rs.shape)
    bad_c = np.count_nonzero(gp != rp)
    bad_s = np.count_nonzero(gs != rs)
    assert bad_s == 0, f"{name}: {bad_s} block scales differ (first at {np.argwhere(gs != rs)[:3]})"
    assert bad_c == 0, f"{name}: {bad_c} code bytes differ (first at {np.argwhere(gp != rp)[:3]})"
    gg = g["gscale"].reshape(-1)[:2]
    assert gg.view(np.uint32).tolist() == rg.view(np.uint32).tolist(), f"{name}: gscale {gg} vs {rg}"


def unpack_gpu(t, group=0):
    """GPU NVFP4Tensor group -> oracle-style dict with unpacked codes."""
    codes = quant.unpack(t.codes[group].cpu().numpy())
    gs = t.gscale[group].cpu().numpy()
    return dict(codes=codes, scales=t.scales[group].cpu().numpy(), s_enc=gs[0], s_dec=gs[1])


def check_close_bf16(gpu, ref64, mag64, name, rel_l2=1e-3, floor=2.0 ** -20):
    """GEMM-output tolerance.

    gpu: bf16 values (float array); ref64: the oracle's float64 values;
    mag64: sum of |products| behind each value.  Passes if the relative L2
    error against the bf16-rounded reference is <= rel_l2 and every element
    is within 2 bf16 ulp of it plus floor * mag (the float32 accumulation
    error of a near-cancelling sum, which no bf16 ulp bound can cover).
    """
    gpu = np.asarray(gpu, np.float64)
    refb = formats.bf16_round_f64(ref64)
    diff = np.abs(gpu - refb)
    nrm = np.linalg.norm(refb)
    rel = np.linalg.norm(gpu - refb) / (nrm if nrm > 0 else 1.0)
    assert rel <= rel_l2, f"{name}: rel-L2 {rel:.3e} > {rel_l2}"
    bound = 2 * formats.ulp_bf16(refb) + floor * np.asarray(mag64, np.float64)
    bad = diff > bound
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(
            f"{name}: {bad.sum()} of {bad.size} elements outside tolerance; first {tuple(i)}: "
            f"gpu {gpu[tuple(i)]!r} ref {ref64[tuple(i)]!r} bound {bound[tuple(i)]!r}")
    return rel


def bf16_tensor(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).to(device)


def upload_nvfp4(q, device="cuda"):
    """Oracle quantize() result -> GPU NVFP4Tensor holding the same bytes
    (the oracle's own values become the GPU stage's input)."""
    from paper_2607_15810_amd.ops import NVFP4Tensor
    packed = np.ascontiguousarray(q["packed"])
    rows, half = packed.shape
    t = NVFP4Tensor.empty(1, rows, half * 2, device)
    t.codes.copy_(torch.from_numpy(packed).view(1, rows, half))
    t.scales.copy_(torch.from_numpy(np.ascontiguousarray(q["scales"])).view(1, rows, -1))
    t.gscale.copy_(torch.tensor([[float(q["s_enc"]), float(q["s_dec"])]], dtype=torch.float32))
    return t


def oracle_bank(w_bf16, experts=None, threads=None):
    """Oracle quantisation of a bf16 bank [E][N][K]; with `experts` only those
    experts are quantised (the others stay zero and must not be used).

    Experts are independent, so large banks are quantised by the oracle's own
    per-matrix quantize() on a pool of threads (numpy releases the GIL inside
    its array operations); the result is the same as one expert after the
    other."""
    import concurrent.futures as cf
    import os
    E, N, K = w_bf16.shape
    todo = list(range(E)) if experts is None else [int(e) for e in experts]
    codes = np.zeros((E, N, K), np.uint8)
    scales = np.zeros((E, N, K // 16), np.uint8)
    gscale = np.ones((E, 2), np.float32)

    def one(e):
        q = quant.quantize(w_bf16[e].float().numpy())
        codes[e], scales[e] = q["codes"], q["scales"]
        gscale[e] = (q["s_enc"], q["s_dec"])

    n = threads or min(16, os.cpu_count() or 1)
    if n <= 1 or len(todo) <= 1:
        for e in todo:
            one(e)
    else:
        with cf.ThreadPoolExecutor(n) as ex:
            list(ex.map(one, todo))
    return dict(codes=codes, scales=scales, gscale=gscale)


def assert_bank_equal(gpu_bank, ref_bank, experts):
    for e in experts:
        ref = dict(packed=quant.pack(ref_bank["codes"][e]), scales=ref_bank["scales"][e],
                   s_enc=ref_bank["gscale"][e, 0], s_dec=ref_bank["gscale"][e, 1])
        assert_nvfp4_equal(dict(packed=gpu_bank.codes[e].cpu().numpy(),
                                scales=gpu_bank.scales[e].cpu().numpy(),
                                gscale=gpu_bank.gscale[e].cpu().numpy()), ref, f"W[{e}]")

"""qd_moe_layer_forward_noalloc (the layer forward on the library's own
scratch buffer) against qd_moe_layer_forward on a caller workspace: the same
kernels, so the outputs must be identical bit for bit, on two calls in a row
(the second with a smaller batch, so stale scratch contents from the first
call must not leak into it), through the C ABI."""

import ctypes

import pytest
import torch

from paper_2607_15810_amd import ops, synth
from paper_2607_15810_amd import quads as Q

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _forward(lay_args, x, lg, T, noalloc):
    w13, w2, H, E, k, I, Ks, Ks2 = lay_args
    y = torch.full((T, H), float("nan"), dtype=torch.bfloat16, device=DEV)
    s13, s2 = w13.struct(), w2.struct()
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        st = Q.raw("qd_moe_layer_forward_noalloc", x.data_ptr(), lg.data_ptr(), T, H, E, k, I,
                   Ks, Ks2, 1, ctypes.byref(s13), ctypes.byref(s2), y.data_ptr(), stream)
    else:
        n = Q.lib().qd_moe_layer_workspace(T, H, E, k, I)
        ws = torch.empty(n, dtype=torch.uint8, device=DEV)
        st = Q.raw("qd_moe_layer_forward", x.data_ptr(), lg.data_ptr(), T, H, E, k, I, Ks, Ks2,
                   1, ctypes.byref(s13), ctypes.byref(s2), y.data_ptr(), ws.data_ptr(), n,
                   stream)
    assert st == Q.QD_OK, Q.status_string(st)
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("Ks,Ks2", [(32, 0), (24, 16)])
def test_noalloc_matches_workspace_forward(Ks, Ks2):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    T, H, E, k, I = 200, 1024, 32, 8, 256
    inp = synth.small_moe("noalloc", T, H, E, k, I, Ks, seed=11)
    w13 = ops.quantize_weight(inp.w13.to(DEV))
    w2 = ops.quantize_weight(inp.w2.to(DEV))
    args = (w13, w2, H, E, k, I, Ks, Ks2)
    x, lg = inp.x.to(DEV), inp.logits.to(DEV)
    assert Q.lib().qd_moe_layer_workspace(T, H, E, k, I) <= Q.lib().qd_moe_layer_noalloc_max_bytes()
    # first call: the full batch; second call: a smaller one (its first 37
    # tokens), which leaves the first call's intermediates in the scratch
    # buffer beyond its own
    for t in (T, 37):
        xs, ls = x[:t].contiguous(), lg[:t].contiguous()
        ya = _forward(args, xs, ls, t, noalloc=True)
        yb = _forward(args, xs, ls, t, noalloc=False)
        assert not torch.isnan(ya.float()).any()
        assert torch.equal(ya.view(torch.int16), yb.view(torch.int16)), f"T={t}"


def test_noalloc_rejects_oversize_batch():
    # 8192 tokens at H = 2048 need ~553 MiB of intermediates: refused before
    # any device work
    big = Q.lib().qd_moe_layer_workspace(8192, 2048, 128, 8, 768)
    assert big > Q.lib().qd_moe_layer_noalloc_max_bytes()
    F = ctypes.c_void_p(256)
    nv = Q.NVFP4(256, 256, 256, 128, 1536, 2048, None)
    nv2 = Q.NVFP4(256, 256, 256, 128, 2048, 768, None)
    st = Q.raw("qd_moe_layer_forward_noalloc", F, F, 8192, 2048, 128, 8, 768, 64, 0, 1,
               ctypes.byref(nv), ctypes.byref(nv2), F, None)
    assert st == Q.QD_ERR_WORKSPACE

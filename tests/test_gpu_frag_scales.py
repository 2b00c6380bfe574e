"""The fragment-ordered copy of the weight scales (nvfp4_pack_frag_scales).

The copy is a pure re-layout, so the checks are exact: the packed bytes
against a numpy transposition of the standard layout, and the grouped GEMM
(decode-shaped batches, where the kernel reads the copy) bit for bit against
the same call without it.  Shapes include weight-row counts that are not a
multiple of the decode kernel's 256-row unit, where part of a unit's
fragments lie past the last row, and prefill shapes (the tile kernel).
"""

import numpy as np
import pytest
import torch

from paper_2607_15810_amd import ops
from paper_2607_15810_amd import quads as Q

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    Q.lib()
    yield


def _frag_ref(scales):
    """[G][R][C/16] -> [G][R/16][C/256][4][16][4] (numpy)."""
    G, R, C16 = scales.shape
    s = scales.reshape(G, R // 16, 16, C16 // 16, 4, 4)      # [g][f][l][c][q][b]
    return np.ascontiguousarray(s.transpose(0, 1, 3, 4, 2, 5)).reshape(G, R // 16, C16 // 16, 256)


@pytest.mark.parametrize("shape", [(1, 16, 256), (3, 48, 768), (2, 272, 512)])
def test_pack_frag_scales_layout(shape):
    G, R, C = shape
    rng = np.random.default_rng(R * 7 + C)
    t = ops.NVFP4Tensor.empty(G, R, C, DEV)
    t.codes.copy_(torch.from_numpy(rng.integers(0, 256, t.codes.shape, dtype=np.uint8)))
    sc = rng.integers(0, 127, t.scales.shape, dtype=np.uint8)
    t.scales.copy_(torch.from_numpy(sc))
    t.gscale.fill_(1.0)
    out = ops.pack_frag_scales(t).cpu().numpy()
    assert np.array_equal(out, _frag_ref(sc))


def _routing(T, E, k, seed):
    g = torch.Generator().manual_seed(seed)
    logits = torch.randn(T, E, generator=g).to(DEV)
    return ops.route_permute(logits, k)


CASES = [
    # name, T, K, E, k, N, epilogue, Ks
    ("swiglu_partial_unit_rac", 64, 512, 8, 2, 288, Q.QD_EPI_SWIGLU, 24),
    ("plain_partial_unit", 48, 512, 8, 4, 272, Q.QD_EPI_NONE, 0),
    ("swiglu_two_passes", 96, 256, 4, 2, 512, Q.QD_EPI_SWIGLU, 8),
    # many rows per expert: the prefill tile kernel reads the copy too
    ("tile_swiglu_rac", 512, 512, 4, 2, 256, Q.QD_EPI_SWIGLU, 16),
    ("tile_plain", 400, 768, 4, 2, 384, Q.QD_EPI_NONE, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_grouped_gemm_frag_scales_bitwise(case):
    name, T, K, E, k, N, epi, Ks = case
    g = torch.Generator().manual_seed(len(name) * 31 + K)
    x = torch.randn(T, K, generator=g).to(torch.bfloat16).to(DEV)
    w = (torch.randn(E, N, K, generator=g) * 0.02).to(torch.bfloat16).to(DEV)
    wq = ops.quantize_weight(w, frag_scales=False)
    assert wq.scales_frag is None
    wf = ops.NVFP4Tensor(wq.codes, wq.scales, wq.gscale, wq.groups, wq.rows, wq.cols,
                         ops.pack_frag_scales(wq))
    _, _, offs, row_token, _ = _routing(T, E, k, 3 + K)
    R = T * k
    xq, scores, ramax = ops.quantize_act(x, rac=True)
    if Ks:
        sel, rq, _, _ = ops.select_channels(x, xq, Ks, scores, ramax)
        kw = dict(rq=rq, sel=sel)
    else:
        kw = {}
    y0, a0 = ops.grouped_gemm(xq, wq, R, row_token, offs, epilogue=epi, want_amax=True, **kw)
    y1, a1 = ops.grouped_gemm(xq, wf, R, row_token, offs, epilogue=epi, want_amax=True, **kw)
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    assert torch.equal(a0, a1)

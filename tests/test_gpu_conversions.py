"""Exhaustive checks of the two hardware conversions the GPU path relies on
(the E2M1 format of Sec. 2.2, "FP4" paragraph).

1. f32 -> E2M1: the quantisers take their codes from the hardware's scaled
   FP4 conversion with a unit scale.  Every float32 bit pattern in [0, 8)
   and every negative one in (-8, -0] goes through nvfp4_quantize_act (f32
   input) with a static tensor amax of 6, each 16-element block anchored by
   a 6.0: then s_enc = 448, every block scale is 448 (code 0x7E) and the
   per-block multiplier enc = s_enc / 448 is exactly 1, so each code must be
   sign | E2M1_RNE(|x|) as the oracle rounds it.  The oracle's encoder is
   evaluated at its own transition points (found by bisection over bit
   patterns; round-to-nearest is monotone in |x|), which fixes its value at
   every pattern in between.

2. E2M1 code x E4M3 scale -> MFMA operand: the GEMMs decode every operand
   with the hardware's scaled FP4 -> f16 conversion (power-of-two scale)
   and one packed f16 multiply by the scale.  All 16 codes x 127 finite
   scale bytes are decoded in each GEMM kernel (few rows per expert, many
   rows per expert, the generic fallback), on the weight side and on the
   activation side: the other operand is one-hot (value 1.0, tensor scales
   1), so every bf16 output is one decoded value, which must equal the
   oracle's exact e2m1 * e4m3.
"""

import numpy as np
import pytest
import torch

from oracle import formats, quant as OQ
from paper_2607_15810_amd import ops

DEV = "cuda"

LIMIT = 0x41000000          # bit pattern of 8.0: patterns [0, LIMIT) are [0, 8)


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _oracle_code(pattern):
    x = np.array([pattern], dtype=np.uint32).view(np.float32)
    return int(formats.e2m1_encode_mag(np.abs(x))[0])


def _transitions():
    """For c = 1..7 the first non-negative float32 pattern whose oracle code
    is >= c (bisection; checked on both sides of each point)."""
    out = []
    lo = 0
    for c in range(1, 8):
        a, b = lo, LIMIT - 1          # oracle(b) = 7 >= c
        assert _oracle_code(b) == 7
        while a < b:
            m = (a + b) // 2
            if _oracle_code(m) >= c:
                b = m
            else:
                a = m + 1
        assert _oracle_code(a) == c and _oracle_code(a - 1) == c - 1
        out.append(a)
        lo = a
    return np.array(out, dtype=np.uint32)


def test_transitions_are_the_rounding_thresholds():
    """The oracle's transitions sit where round-to-nearest-even puts them:
    0.25 and 1.25, 2.5, 5 round down (to the even code), 0.75, 1.75 and 3.5
    round up."""
    t = _transitions().view(np.float32)
    up = lambda v: np.nextafter(np.float32(v), np.float32(10))
    assert list(t) == [up(0.25), np.float32(0.75), up(1.25), np.float32(1.75), up(2.5),
                       np.float32(3.5), up(5.0)]


@pytest.mark.gpu
def test_e2m1_encode_every_pattern():
    """The enumeration is built on the device with torch (it is an input: a
    plain count over bit patterns), and the oracle's code of every pattern,
    the number of its transitions at or below the pattern, is expanded there
    too; the library's codes are unpacked and compared on the device."""
    _need_gpu()
    trans = _transitions()
    tr_dev = torch.from_numpy(trans.astype(np.int64)).to(DEV)
    per_block = 15
    cols = 4096
    vals_per_row = cols // 16 * per_block
    chunk = vals_per_row * 65536                    # 251,658,240 patterns
    amax = torch.tensor([6.0], device=DEV)
    anchor = int(np.float32(6.0).view(np.uint32))
    checked = 0
    for sign in (0, 0x80000000):
        for start in range(0, LIMIT, chunk):
            stop = min(start + chunk, LIMIT)
            n = stop - start
            nrow = (n + vals_per_row - 1) // vals_per_row
            pat = torch.arange(start, start + nrow * vals_per_row, dtype=torch.int64, device=DEV)
            pat = torch.clamp(pat, max=stop - 1)     # the last row's tail repeats the last pattern
            body = (pat | sign).view(-1, per_block)
            blocks = torch.cat([torch.full((body.shape[0], 1), anchor, dtype=torch.int64,
                                           device=DEV), body], dim=1)
            # int64 holding 32-bit patterns -> the same bits as int32 -> float32
            x = torch.where(blocks >= (1 << 31), blocks - (1 << 32), blocks).to(torch.int32)
            x = x.view(torch.float32).reshape(nrow, cols)
            del blocks, body
            q, _, _ = ops.quantize_act(x, amax_partials=amax)
            gs = q.gscale[0].cpu().numpy()
            assert gs.tolist() == [np.float32(448.0), np.float32(1.0) / np.float32(448.0)]
            assert bool((q.scales == 0x7E).all()), "block scale is not 448"
            pk = q.codes[0].to(torch.int32)
            codes = torch.stack([pk & 15, pk >> 4], dim=-1).reshape(-1, 16)
            assert bool((codes[:, 0] == 7).all()), "anchor 6.0 not encoded as 6"
            got = codes[:, 1:].reshape(-1)
            exp = (pat[:, None] >= tr_dev[None, :]).sum(dim=1).to(torch.int32)
            if sign:
                exp = exp | 8
            bad = torch.nonzero(got != exp).flatten()
            if bad.numel():
                i = int(bad[0])
                raise AssertionError(
                    f"{bad.numel()} codes differ; first pattern {int(pat[i]) | sign:#010x}: "
                    f"gpu {int(got[i]):#x} oracle {int(exp[i]):#x}")
            checked += n
            del x, q, pk, codes, got, exp, pat
    assert checked == 2 * LIMIT


def _pattern_bank(groups, rows, K, salt):
    """NVFP4 [groups][rows][K] covering every (code, scale byte) pair: block b
    of row n of group g has scale byte (salt + 4096 g + 16 n + b) % 127 and
    element i of it the code (i + n + b + g) % 16.  Tensor scales 1."""
    g = np.arange(groups)[:, None, None, None]
    n = np.arange(rows)[None, :, None, None]
    b = np.arange(K // 16)[None, None, :, None]
    i = np.arange(16)[None, None, None, :]
    codes = ((i + n + b + g) % 16).astype(np.uint8).reshape(groups, rows, K)
    scales = ((salt + 4096 * g + 16 * n + b) % 127).astype(np.uint8).reshape(groups, rows, K // 16)
    return codes, scales


def _one_hot(rows, K, ch):
    """rows one-hot NVFP4 rows: row r holds 1.0 (code 2, scale 0x38) at
    channel ch[r]; every block scale is 0x38 and the tensor scale 1."""
    codes = np.zeros((rows, K), np.uint8)
    codes[np.arange(rows), ch] = 2
    scales = np.full((rows, K // 16), 0x38, np.uint8)
    return codes, scales


def _nv_from(codes, scales, frag=False):
    G, R, K = codes.shape
    t = ops.NVFP4Tensor.empty(G, R, K, DEV)
    t.codes.copy_(torch.from_numpy(OQ.pack(codes.reshape(G * R, K)).reshape(G, R, K // 2)))
    t.scales.copy_(torch.from_numpy(scales))
    t.gscale.fill_(1.0)
    if frag:
        t.scales_frag = ops.pack_frag_scales(t)
    return t


def _check_pairs_seen(codes, scales, used):
    """every (code, scale byte) pair among the decoded values `used` (a mask
    over codes) -- 16 x 127 of them"""
    sc = np.repeat(scales, 16, axis=-1)
    pairs = set(zip(codes[used].tolist(), sc[used].tolist()))
    assert len(pairs) == 16 * 127, len(pairs)


# (kernel, experts, rows per expert, N, K): the plans the grouped GEMM picks
DECODE_CASES = [
    ("few_rows_frag_scales", 8, 32, 256, 256),    # decode kernel, fragment-ordered scales
    ("few_rows", 8, 32, 256, 256),                # decode kernel, standard scales
    ("many_rows", 1, 256, 256, 256),              # tile kernel
    ("fallback", 1, 256, 240, 256),               # N % 128 != 0: the generic kernel
]


@pytest.mark.gpu
@pytest.mark.parametrize("kind,E,per,N,K", DECODE_CASES, ids=[c[0] for c in DECODE_CASES])
def test_decode_all_pairs_weight_side(kind, E, per, N, K):
    _need_gpu()
    rows = E * per
    wc, wsc = _pattern_bank(E, N, K, salt=5)
    w = _nv_from(wc, wsc, frag=kind.endswith("frag_scales"))
    # row r of expert e probes channel r % K (each expert sees its own rows)
    ch = np.arange(rows) % K
    ac, asc = _one_hot(rows, K, ch)
    a = _nv_from(ac[None], asc[None])
    offs = torch.arange(0, rows + 1, per, dtype=torch.int32, device=DEV)
    out, _ = ops.grouped_gemm(a, w, rows, offsets=offs)
    got = out.float().cpu().numpy().astype(np.float64)          # [rows][N]
    ref = np.empty((rows, N))
    used = np.zeros(wc.shape, bool)
    for r in range(rows):
        e = r // per
        v = OQ.dequantize_unscaled_f64(wc[e], wsc[e])             # [N][K]
        ref[r] = v[:, ch[r]]
        used[e, :, ch[r]] = True
    _check_pairs_seen(wc, wsc, used)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} decoded weights differ (first {bad[0]})"


@pytest.mark.gpu
@pytest.mark.parametrize("kind,E,per,N,K", DECODE_CASES, ids=[c[0] for c in DECODE_CASES])
def test_decode_all_pairs_activation_side(kind, E, per, N, K):
    _need_gpu()
    rows = E * per
    ac, asc = _pattern_bank(1, rows, K, salt=11)
    a = _nv_from(ac, asc)
    # weight row n of every expert is one-hot at channel n % K
    wc1, wsc1 = _one_hot(N, K, np.arange(N) % K)
    w = _nv_from(np.repeat(wc1[None], E, 0), np.repeat(wsc1[None], E, 0),
                 frag=kind.endswith("frag_scales"))
    offs = torch.arange(0, rows + 1, per, dtype=torch.int32, device=DEV)
    out, _ = ops.grouped_gemm(a, w, rows, offsets=offs)
    got = out.float().cpu().numpy().astype(np.float64)
    v = OQ.dequantize_unscaled_f64(ac[0], asc[0])                 # [rows][K]
    ref = v[:, np.arange(N) % K]
    used = np.zeros(ac.shape, bool)
    used[0][:, np.arange(N) % K] = True
    _check_pairs_seen(ac, asc, used)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} decoded activations differ (first {bad[0]})"

"""Pins for the oracle's number formats (E2M1, E4M3FN, BF16).

Each check compares the oracle with something other than itself: the values
printed in the paper (golden files), a library routine (torch's float8 and
bfloat16 casts), or an independently written closed form.
"""

import os

import numpy as np
import pytest
import torch

from oracle import formats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [float(l) for l in f if l.strip() and not l.startswith("#")]


def test_e2m1_values_match_paper():
    assert list(formats.E2M1_MAG) == _golden("e2m1_magnitudes.txt")
    codes = np.arange(16, dtype=np.uint8)
    vals = formats.e2m1_decode(codes)
    mags = _golden("e2m1_magnitudes.txt")
    assert list(vals[:8]) == mags
    assert list(-vals[8:]) == mags
    assert np.signbit(vals[8])          # code 8 is negative zero


def _e2m1_interval_table(a):
    """Round-to-nearest-even onto {0,.5,1,1.5,2,3,4,6} with saturation,
    written as the interval table that follows from the midpoints
    0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5 (each midpoint goes to the neighbour
    whose code is even)."""
    out = np.empty(a.shape, dtype=np.uint8)
    for i, v in enumerate(a.reshape(-1)):
        v = float(v)
        if v <= 0.25:
            c = 0
        elif v < 0.75:
            c = 1
        elif v <= 1.25:
            c = 2
        elif v < 1.75:
            c = 3
        elif v <= 2.5:
            c = 4
        elif v < 3.5:
            c = 5
        elif v <= 5.0:
            c = 6
        else:
            c = 7
        out.reshape(-1)[i] = c
    return out


def test_e2m1_rounding_against_interval_table():
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], dtype=np.float32)
    pts = [mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(10)),
           formats.E2M1_MAG.astype(np.float32),
           np.array([0.0, 1e-30, 6.0, 6.5, 7.0, 100.0, 3.4e38], dtype=np.float32)]
    rng = np.random.default_rng(0)
    pts.append((rng.random(20000) * 8).astype(np.float32))
    a = np.concatenate(pts).astype(np.float32)
    assert np.array_equal(formats.e2m1_encode_mag(a), _e2m1_interval_table(a))


def test_e2m1_ties_go_to_even_code():
    # midpoint -> (lower code, upper code); the even one wins
    cases = {0.25: 0, 0.75: 2, 1.25: 2, 1.75: 4, 2.5: 4, 3.5: 6, 5.0: 6}
    for v, c in cases.items():
        assert formats.e2m1_encode_mag(np.array([v], np.float32))[0] == c


def test_e4m3_decode_matches_torch_for_all_codes():
    codes = torch.arange(256, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = formats.e4m3_decode(np.arange(256))
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(ours))
    assert np.array_equal(ref[~nan], ours[~nan])
    assert formats.E4M3_POS.max() == _golden("e4m3_max.txt")[0]


def test_e4m3_encode_matches_torch_cast():
    rng = np.random.default_rng(1)
    vals = [formats.E4M3_POS.astype(np.float32)]
    mids = ((formats.E4M3_POS[1:] + formats.E4M3_POS[:-1]) / 2).astype(np.float32)
    vals += [mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(1e9))]
    vals.append(np.exp(rng.uniform(np.log(1e-5), np.log(448), 50000)).astype(np.float32))
    vals.append(np.array([0.0, 2.0 ** -10, 2.0 ** -11, 1.5 * 2.0 ** -9, 448.0, 17, 19],
                         dtype=np.float32))
    t = np.clip(np.concatenate(vals), 0, 448).astype(np.float32)
    ours = formats.e4m3_encode_pos(t)
    ref = torch.from_numpy(t).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref)


def test_e4m3_rejects_out_of_range():
    with pytest.raises(ValueError):
        formats.e4m3_encode_pos(np.array([449.0], np.float32))


def test_bf16_round_f32_matches_torch():
    rng = np.random.default_rng(2)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 1e3,
                        (rng.standard_normal(1000) * 1e-39).astype(np.float32),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8)],
                                 dtype=np.float32)])
    ours = formats.bf16_round_f32(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_round_f64_nearest_and_even():
    rng = np.random.default_rng(3)
    v = np.concatenate([rng.standard_normal(50000) * 10.0 ** rng.integers(-30, 30, 50000),
                        [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 2.0 ** -130 * 1.5, 0.0]])
    r = formats.bf16_round_f64(v)
    # representable: a float32 -> bfloat16 round trip leaves it unchanged
    r32 = r.astype(np.float32)
    assert np.array_equal(r32.astype(np.float64), r)
    back = torch.from_numpy(r32).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(back, r32)
    # nearest: within half a unit in the last place
    u = formats.ulp_bf16(r)
    assert np.all(np.abs(v - r) <= u / 2)
    # ties to even
    assert formats.bf16_round_f64(np.array([1.0 + 2 ** -8]))[0] == 1.0
    assert formats.bf16_round_f64(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6
    # float32 inputs: same answer as the float32 rounding
    x32 = rng.standard_normal(10000).astype(np.float32)
    assert np.array_equal(formats.bf16_round_f64(x32.astype(np.float64)),
                          formats.bf16_round_f32(x32).astype(np.float64))


def test_ulp_bf16():
    assert formats.ulp_bf16(np.array([1.0]))[0] == 2.0 ** -7
    assert formats.ulp_bf16(np.array([1.9999]))[0] == 2.0 ** -7
    assert formats.ulp_bf16(np.array([2.0]))[0] == 2.0 ** -6
    assert formats.ulp_bf16(np.array([0.0]))[0] == 2.0 ** -133

"""Number formats used by NVFP4: E2M1 element codes, E4M3FN block scales, BF16.

Paper, Sec. 2.2 ("FP4" paragraph): the NVFP4 core is E2M1 with magnitudes
{0, 0.5, 1, 1.5, 2, 3, 4, 6} per sign; sixteen consecutive elements share an
E4M3 block scale; a per-tensor FP32 scale gives a second level of range.
Paper, Sec. 2.2 ("FP8" paragraph): E4M3 has three mantissa bits and a maximum
magnitude of 448.

The unified formula Eq. (quant-unified) has no exponent bias and no
subnormals, so it cannot produce E2M1's 0 and 0.5; the value set printed in
the FP4 paragraph is taken as the definition instead, and E4M3 is the
finite-only "FN" variant (bias 7, max 448, code 0x7F is NaN, no infinity,
subnormals m * 2^-9).

All encoders here are nearest-value searches over the explicit value tables
(round to nearest, ties to the even code), i.e. the definition of
round-to-nearest-even written out, not a bit trick.
"""

import numpy as np

# --- E2M1 -----------------------------------------------------------------

# Magnitude of E2M1 code c (c = 0..7); the sign is bit 3 of a 4-bit code.
E2M1_MAG = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)


def e2m1_decode(codes):
    """4-bit codes (uint8, 0..15) -> float64 values (sign in bit 3)."""
    codes = np.asarray(codes, dtype=np.uint8)
    mag = E2M1_MAG[codes & 7]
    return np.where((codes >> 3) & 1, -mag, mag)


def e2m1_encode_mag(a):
    """Round non-negative float32 magnitudes to the nearest E2M1 magnitude.

    Returns the 3-bit magnitude code.  Ties go to the even code (mantissa bit
    0), values above 6 saturate to 6 (6 is the nearest representable value).
    Brute force: the distance to each of the eight values, in turn, is
    computed in float64 (exact for the float32 inputs at every tie point)
    and the closest so far is kept; an exact tie keeps the even code.
    """
    a = np.asarray(a, dtype=np.float32).astype(np.float64)
    # every value above 6 has 6 as its nearest magnitude; clamping at 8 keeps
    # the distances below distinguishable in float64 for huge inputs
    a = np.minimum(a, 8.0)
    best_d = np.full(a.shape, np.inf)
    best_c = np.zeros(a.shape, dtype=np.uint8)
    for c, m in enumerate(E2M1_MAG):
        d = np.abs(a - m)
        # candidates are visited in increasing order, so a tie is always
        # between codes c-1 and c; the even one of the two wins
        take = (d < best_d) | ((d == best_d) & (c % 2 == 0))
        best_d = np.where(take, d, best_d)
        best_c = np.where(take, np.uint8(c), best_c)
    return best_c


# --- E4M3FN ---------------------------------------------------------------

def _e4m3_table():
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        s = -1.0 if c & 0x80 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            vals[c] = np.nan
        elif e == 0:
            vals[c] = s * m * 2.0 ** -9
        else:
            vals[c] = s * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


E4M3_VALUES = _e4m3_table()          # code -> value (NaN for 0x7F / 0xFF)
E4M3_POS = E4M3_VALUES[:127].copy()  # codes 0x00..0x7E, strictly increasing
E4M3_MAX = 448.0


def e4m3_decode(codes):
    """E4M3FN byte codes -> float64 values."""
    return E4M3_VALUES[np.asarray(codes, dtype=np.uint8)]


def e4m3_encode_pos(t):
    """Round non-negative float32 values in [0, 448] to E4M3FN, RNE.

    Nearest of the 127 finite non-negative E4M3FN values; an exact midpoint
    goes to the even code.  Callers clamp to 448 first (the format has no
    infinity; the paper's maximum is 448).
    """
    t = np.asarray(t, dtype=np.float32).astype(np.float64)
    if np.any(t < 0) or np.any(t > E4M3_MAX) or np.any(np.isnan(t)):
        raise ValueError("e4m3_encode_pos expects values in [0, 448]")
    hi = np.searchsorted(E4M3_POS, t, side="left").clip(0, 126)
    lo = (hi - 1).clip(0, 126)
    d_hi = np.abs(E4M3_POS[hi] - t)
    d_lo = np.abs(t - E4M3_POS[lo])
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    return np.where(pick_lo, lo, hi).astype(np.uint8)


# --- BF16 -----------------------------------------------------------------

def bf16_round_f32(x):
    """float32 -> nearest bfloat16 value (RNE), returned as float32.

    Written as the definition: the bfloat16 neighbours of x are obtained by
    truncating the float32 significand to 8 bits, and the nearer one (the
    even one on a tie) is chosen.
    """
    x = np.asarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    down = (u & 0xFFFF0000).astype(np.uint32).view(np.float32).astype(np.float64)
    up_bits = ((u & 0xFFFF0000) + 0x10000).astype(np.uint32)
    up = up_bits.view(np.float32).astype(np.float64)
    xv = x.astype(np.float64)
    d_down = np.abs(xv - down)
    d_up = np.abs(up - xv)
    down_even = ((u >> 16) & 1) == 0
    pick_down = (d_down < d_up) | ((d_down == d_up) & down_even)
    res = np.where(pick_down, down, up)
    return res.astype(np.float32)


def bf16_round_f64(v):
    """float64 -> nearest bfloat16 value (RNE, single rounding), as float64.

    Normal range: keep 8 significant bits with np.rint (ties to even);
    below 2^-126 the quantum is the bfloat16 subnormal step 2^-133.
    """
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)                      # v = m * 2^e, 0.5 <= |m| < 1
    e_eff = np.maximum(e, -125)             # 2^-126 = 0.5 * 2^-125
    q = np.ldexp(np.ones_like(v), e_eff - 8)  # quantum: 8 significant bits
    return np.rint(v / q) * q


def ulp_bf16(v):
    """Spacing of bfloat16 numbers at |v| (the unit in the last place)."""
    v = np.abs(np.asarray(v, dtype=np.float64))
    _, e = np.frexp(v)                      # |v| in [2^(e-1), 2^e)
    e = np.where(v > 0, np.maximum(e - 1, -126), -126)
    return np.ldexp(1.0, e - 7)

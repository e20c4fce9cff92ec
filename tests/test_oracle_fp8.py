"""Pins for the E4M3 rounding of the oracle (CPU only).

Hand-computed codes from the format definition (sign, 4 exponent bits with
bias 7, 3 mantissa bits, no infinities, S.1111.111 = NaN), the fixed points of
the rounding (every code's value), ties to even at every midpoint, the
half-ulp error bound, saturation and monotonicity.
"""

import math

import numpy as np

from oracle import E4M3_MAX, decode_e4m3, encode_e4m3, round_e4m3

# value -> code, worked by hand from the bit layout
HAND = [
    (1.0, 0x38),             # 0 0111 000: 2^(7-7)
    (-2.0, 0xC0),            # 1 1000 000
    (0.1015625, 0x1D),       # 1.625 * 2^-4: 0 0011 101 (the nearest value to 0.1)
    (448.0, 0x7E),           # 0 1111 110: 1.75 * 2^8, the largest finite value
    (256.0, 0x78),           # 0 1111 000
    (240.0, 0x77),           # 0 1110 111: 1.875 * 2^7
    (2.0 ** -6, 0x08),       # smallest normal
    (7 / 8 * 2.0 ** -6, 0x07),  # largest subnormal
    (2.0 ** -9, 0x01),       # smallest subnormal
    (0.0, 0x00),
]


def _finite_codes():
    return [c for c in range(256) if not math.isnan(decode_e4m3(c))]


def test_hand_codes():
    for v, code in HAND:
        assert decode_e4m3(code) == v
        assert encode_e4m3(v) == code
        assert round_e4m3(v) == v
    assert round_e4m3(0.1) == 0.1015625
    assert math.isnan(decode_e4m3(0x7F)) and math.isnan(decode_e4m3(0xFF))


def test_codes_are_fixed_points():
    codes = _finite_codes()
    assert len(codes) == 254
    vals = np.array([decode_e4m3(c) for c in codes])
    assert np.array_equal(round_e4m3(vals), vals)
    for c in codes:
        assert encode_e4m3(decode_e4m3(c)) == c


def test_midpoints_round_to_even_and_others_to_nearest():
    pos = sorted({decode_e4m3(c) for c in _finite_codes() if decode_e4m3(c) >= 0})
    rng = np.random.default_rng(0)
    for a, b in zip(pos[:-1], pos[1:]):
        mid = (a + b) / 2
        even = a if encode_e4m3(a) % 2 == 0 else b
        assert round_e4m3(mid) == even and round_e4m3(-mid) == -even
        for f in rng.uniform(0.0, 1.0, size=8):
            x = a + f * (b - a)
            if x != mid:
                assert round_e4m3(x) == (a if x < mid else b)


def test_error_bound_saturation_monotonic():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.normal(0, 3, 20000), rng.uniform(-500, 500, 5000), rng.normal(0, 1e-3, 5000)])
    r = round_e4m3(x)
    normal = (np.abs(x) >= 2.0 ** -6) & (np.abs(x) <= E4M3_MAX)
    assert np.all(np.abs(r - x)[normal] <= 2.0 ** -4 * np.abs(x)[normal])   # half an ulp of 3 mantissa bits
    sub = np.abs(x) < 2.0 ** -6
    assert np.all(np.abs(r - x)[sub] <= 2.0 ** -10)                            # half the subnormal quantum
    assert np.all(np.abs(r) <= E4M3_MAX)
    assert np.array_equal(round_e4m3([500.0, -1e9, 464.0]), [448.0, -448.0, 448.0])
    xs = np.sort(x)
    assert np.all(np.diff(round_e4m3(xs)) >= 0)

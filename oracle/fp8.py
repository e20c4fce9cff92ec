"""OCP 8-bit floating point E4M3 (the "FP8 Formats for Deep Learning" E4M3),
used for FP8 storage of the KV cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

E4M3 has a sign bit, 4 exponent bits (bias 7) and 3 mantissa bits:
normal values (-1)^s 2^(e-7) (1 + m/8) for e = 1..15 except the pattern
e = 15, m = 7, which is NaN; subnormals (-1)^s 2^-6 (m/8); no infinities.
The largest finite value is 448, the smallest subnormal 2^-9.

Conversion here rounds to nearest, ties to even, and saturates: magnitudes
beyond 448 become 448 (the KV cache stores finite values only).
"""

import math

import numpy as np

E4M3_MAX = 448.0
_MIN_NORMAL = 2.0 ** -6
_SUB_QUANTUM = 2.0 ** -9


def _rint_even(x):
    return np.rint(x)  # numpy rounds halves to even


def round_e4m3(x) -> np.ndarray:
    """Nearest E4M3 value (ties to even), saturating at +-448; float64 in and out."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    out = np.empty_like(a)
    sub = a < _MIN_NORMAL
    out[sub] = _rint_even(a[sub] / _SUB_QUANTUM) * _SUB_QUANTUM
    nrm = ~sub
    if nrm.any():
        _, e2 = np.frexp(a[nrm])            # a = f * 2^e2 with f in [0.5, 1)
        quantum = np.ldexp(1.0, e2 - 1 - 3)  # 3 mantissa bits below the leading one
        out[nrm] = _rint_even(a[nrm] / quantum) * quantum
    out = np.minimum(out, E4M3_MAX)
    return np.copysign(out, x)


def decode_e4m3(code: int) -> float:
    """Value of an E4M3 bit pattern (NaN for the two NaN patterns)."""
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return math.nan
    if e == 0:
        return s * (m / 8.0) * _MIN_NORMAL
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


def encode_e4m3(v: float) -> int:
    """Bit pattern of an E4M3 value (v must be representable; -0.0 keeps its sign)."""
    s = 0x80 if math.copysign(1.0, v) < 0 else 0
    a = abs(v)
    if a == 0.0:
        return s
    if a < _MIN_NORMAL:
        m = a / _SUB_QUANTUM
        assert m == int(m) and 1 <= m <= 7, v
        return s | int(m)
    f, e2 = math.frexp(a)                 # a = f * 2^e2, f in [0.5, 1)
    e = e2 - 1 + 7
    m = (f * 2.0 - 1.0) * 8.0
    assert 1 <= e <= 15 and m == int(m) and not (e == 15 and m == 7), v
    return s | (e << 3) | int(m)

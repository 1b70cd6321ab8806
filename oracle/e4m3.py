"""OCP FP8 E4M3 (E4M3FN) reference encoder/decoder -- test infrastructure only.

The paper communicates gradients in FP8 (Sec. I; NCCL's native FP8) and scales
with the amax rule ``S_X = amax(X) / E4M3_MAX`` it quotes from COAT (Sec. I).
The format is the OCP 8-bit floating point E4M3 variant: 1 sign bit, 4 exponent
bits with bias 7, 3 mantissa bits, subnormals at exponent field 0, no
infinities, NaN = S.1111.111, largest finite value 448 (S.1111.110).

Rounding reading (the paper is silent): round to nearest, ties to the even
mantissa, saturating finite overflow to +-448, keeping the sign of zero, and
mapping NaN to 0x7F.
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
NAN_CODE = 0x7F


def decode_code(code: int) -> float:
    """Value of one E4M3 bit pattern, read from its fields."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    exp = (code >> 3) & 0xF
    mant = code & 0x7
    if exp == 0xF and mant == 0x7:
        return float("nan")
    if exp == 0:
        return sign * (mant / 8.0) * 2.0 ** (1 - 7)
    return sign * (1.0 + mant / 8.0) * 2.0 ** (exp - 7)


def decode_table() -> np.ndarray:
    """All 256 code values as float64 (NaN for 0x7F and 0xFF)."""
    return np.array([decode_code(c) for c in range(256)], dtype=np.float64)


_TABLE = decode_table()
# magnitude -> code for the 127 finite non-negative patterns 0x00..0x7E
_POS_CODES = np.arange(0x7F)
_POS_VALUES = _TABLE[:0x7F]


def dequantize(codes: np.ndarray) -> np.ndarray:
    """Exact float64 values of E4M3 codes (every E4M3 value is an fp32 value)."""
    return _TABLE[np.asarray(codes, dtype=np.uint8)]


def quantize(y: np.ndarray) -> np.ndarray:
    """Saturating round-to-nearest-even E4M3 codes of float32 values ``y``.

    ``|y|`` is located in its binade ``[2^e, 2^(e+1))`` (``e >= -6``; below that
    the subnormal spacing ``2^-9`` applies), divided by the spacing
    ``2^(e-3)``, rounded half-to-even and multiplied back.  Because ``y`` is a
    float32 value the division and product are exact in float64, so there is a
    single rounding.  Results at or above 448 saturate to 448.
    """
    y = np.asarray(y, dtype=np.float32)
    with np.errstate(invalid="ignore"):
        yd = y.astype(np.float64)
    a = np.abs(yd)
    sign = np.signbit(y).astype(np.uint8) << 7
    nan = np.isnan(yd)
    a_safe = np.where(nan | (a == 0) | np.isinf(a), 1.0, a)
    _, k = np.frexp(a_safe)              # a = f * 2^k, f in [0.5, 1)
    e = np.maximum(k - 1, -6)            # binade exponent, clamped to normal min
    spacing = np.ldexp(1.0, e - 3)
    q = np.round(a_safe / spacing) * spacing     # numpy rounds half to even
    q = np.where(a == 0, 0.0, q)
    q = np.minimum(np.where(np.isinf(a), E4M3_MAX, q), E4M3_MAX)
    idx = np.searchsorted(_POS_VALUES, q)
    assert np.all(_POS_VALUES[np.minimum(idx, 0x7E)][~nan] == q[~nan])
    codes = (idx.astype(np.uint8) | sign).astype(np.uint8)
    codes[nan] = NAN_CODE
    return codes

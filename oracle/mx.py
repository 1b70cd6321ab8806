"""MXFP4 reference (OCP Microscaling Formats v1.0) -- test infrastructure only.

The paper (Sec. I; Sec. VI, Discussion) holds that the coordinate change is not
tied to FP8 and points to FP4 communication as future work without fixing a
format; this is the OCP MX FP4 format gfx950 supports natively, applied to the
same transformed gradient the FP8 codec quantizes:

* Elements: FP4 E2M1 -- 1 sign, 2 exponent bits (bias 1), 1 mantissa bit;
  code ``s e1 e0 m``; value ``(-1)^s 2^(e-1) (1 + m/2)`` for ``e > 0`` and
  ``(-1)^s m/2`` for ``e = 0``: magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6.
* Blocks: 32 consecutive elements of a row share one scale ``X = 2^k``,
  stored as E8M0 (``k + 127`` in a byte; 255 = NaN).
* Conversion of a block ``v``: ``k = floor(log2(max |v|)) - 2`` (2 = the
  exponent of E2M1's largest value, 6 = 1.5 * 2^2), clamped to ``k >= -127``
  (an all-zero block takes ``k = -127``); each element ``v / X`` rounds to
  the nearest E2M1 value, ties to the even code (mantissa bit 0), and
  magnitudes above 6 saturate to 6 (the clamp the MX conversion applies to
  normal values).  The sign of zero is kept.
* Readings where the specification leaves a choice: a block holding a NaN or
  an infinity gets the NaN scale (255) and element codes 0; two codes share
  a byte, element 2i in the low nibble.
* Rank sum and error feedback as for FP8: ``mean = fl32(acc / N)`` with
  ``acc = fl32(acc + deq_j)`` in rank order, ``R = fl32(U - deq)``.

Pins (tests/test_oracle_mx.py): the E2M1 values from the bit-field formula,
brute-force nearest-value rounding at every midpoint, scale closed forms
(amax 6 -> X = 1, amax 8 -> X = 2, saturation between 6 and 8), zero and
NaN blocks, and the quantization error bound (half an E2M1 grid step of the
scaled value) below saturation, packing and exact rank sums; the residual by
its exactness (deq + R == U in float32, by Sterbenz's lemma), its half-step
bound and NaN residuals of NaN / Inf blocks.
"""

from __future__ import annotations

import numpy as np

BLOCK = 32
EMAX_ELEM = 2
SCALE_NAN = 255


def e2m1_value(code: int) -> float:
    """Value of a 4-bit E2M1 code from its bit fields."""
    s = (code >> 3) & 1
    e = (code >> 1) & 3
    m = code & 1
    mag = 2.0 ** (e - 1) * (1.0 + m / 2.0) if e > 0 else m / 2.0
    return -mag if s else mag


E2M1_TABLE = np.array([e2m1_value(c) for c in range(16)], dtype=np.float64)


def round_e2m1(y: np.ndarray) -> np.ndarray:
    """Nearest E2M1 code of each (already scaled) value: ties to the even code,
    magnitudes above 6 saturate, sign kept (also for zero)."""
    y = np.asarray(y, dtype=np.float64)
    mags = E2M1_TABLE[:8]                          # 0, 0.5, ..., 6
    a = np.minimum(np.abs(y), 6.0)
    d = np.abs(a[..., None] - mags)                # distance to every magnitude
    best = d.min(axis=-1, keepdims=True)
    cand = d == best
    # among equally near magnitudes take the even code (mantissa bit 0)
    even = cand & (np.arange(8) % 2 == 0)
    pick = np.where(even.any(axis=-1), np.argmax(even, axis=-1), np.argmax(cand, axis=-1))
    neg = np.signbit(y)
    return (pick + 8 * neg).astype(np.uint8)


def block_scale_exp(amax: np.ndarray) -> np.ndarray:
    """E8M0 byte of each block maximum (float32 values >= 0, or NaN / inf)."""
    a = np.asarray(amax, dtype=np.float64)
    out = np.full(a.shape, SCALE_NAN, dtype=np.uint8)
    fin = np.isfinite(a)
    k = np.full(a.shape, -127, dtype=np.int64)
    pos = fin & (a > 0)
    k[pos] = np.floor(np.log2(a[pos])).astype(np.int64) - EMAX_ELEM
    # log2 of a float32 is exact enough to floor correctly except next to a
    # power of two: fix those against 2^k exactly
    kk = k[pos] + EMAX_ELEM
    lo = np.ldexp(1.0, kk)
    kk = np.where(lo > a[pos], kk - 1, np.where(np.ldexp(1.0, kk + 1) <= a[pos], kk + 1, kk))
    k[pos] = kk - EMAX_ELEM
    k = np.maximum(k, -127)
    out[fin] = (k[fin] + 127).astype(np.uint8)
    return out


def quantize(Ut: np.ndarray):
    """MXFP4 encode of ``[N, m, n]`` float32 (n % 32 == 0) along rows.

    Returns ``(codes [N, m, n] uint8 (one 4-bit code per element), scales
    [N, m, n / 32] uint8 E8M0)``.
    """
    U = np.asarray(Ut, dtype=np.float32)
    N, m, n = U.shape
    assert n % BLOCK == 0
    blocks = U.reshape(N, m, n // BLOCK, BLOCK).astype(np.float64)
    with np.errstate(invalid="ignore"):
        amax = np.abs(blocks).max(axis=-1)
    bad = ~np.isfinite(blocks).all(axis=-1)
    amax = np.where(bad, np.nan, amax)
    scales = block_scale_exp(amax)
    X = np.ldexp(1.0, scales.astype(np.int64) - 127)
    with np.errstate(invalid="ignore"):
        y = blocks / X[..., None]
    codes = round_e2m1(np.where(bad[..., None], 0.0, y))
    return codes.reshape(N, m, n), scales


def dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """float32 values of codes ``[N, m, n]`` with E8M0 scales ``[N, m, n/32]``."""
    c = np.asarray(codes, dtype=np.uint8)
    s = np.asarray(scales, dtype=np.uint8)
    N, m, n = c.shape
    X = np.where(s == SCALE_NAN, np.nan, np.ldexp(1.0, s.astype(np.int64) - 127))
    v = E2M1_TABLE[c & 15].reshape(N, m, n // BLOCK, BLOCK) * X[..., None]
    return v.reshape(N, m, n).astype(np.float32)


def pack(codes: np.ndarray) -> np.ndarray:
    """Two codes per byte, element 2i in the low nibble: ``[..., n] -> [..., n/2]``."""
    c = np.asarray(codes, dtype=np.uint8)
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def unpack(packed: np.ndarray) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.uint8)
    out[..., 0::2] = p & 15
    out[..., 1::2] = p >> 4
    return out


def reduce_local(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Rank mean ``fl32(acc / N)``, ``acc = fl32(acc + deq_j)`` in rank order."""
    deq = dequantize(codes, scales)
    N = deq.shape[0]
    acc = np.zeros(deq.shape[1:], dtype=np.float32)
    for j in range(N):
        acc = (acc + deq[j]).astype(np.float32)
    return (acc / np.float32(N)).astype(np.float32)


def residual(Ut: np.ndarray, codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Error-feedback residual ``fl32(U - deq)``."""
    with np.errstate(invalid="ignore"):
        return (np.asarray(Ut, dtype=np.float32) - dequantize(codes, scales)).astype(np.float32)

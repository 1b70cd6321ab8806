"""Pins of the oracle's FP8 E4M3 encoder/decoder (CPU only).

The quantizer is checked against a brute-force nearest-value search over all
finite E4M3 values (ties to the even code), on every code value, every
rounding midpoint and its float32 neighbours, subnormals, the saturation range
and special values; against the OCP specification's values; and against
torch's float8_e4m3fn cast inside the finite range.
"""

import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import e4m3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_force_codes(y):
    """Nearest finite E4M3 value by exhaustive search; ties go to the even code."""
    table = e4m3.decode_table()
    finite_codes = np.array([c for c in range(0x7F)])     # 0x00..0x7E, values >= 0
    finite_vals = table[finite_codes]
    out = np.empty(len(y), dtype=np.uint8)
    for idx, v in enumerate(np.asarray(y, dtype=np.float32)):
        if np.isnan(v):
            out[idx] = 0x7F
            continue
        a = abs(float(v))
        if a <= 1024.0:
            # both operands are float32 values within 2^-149..2^10 of each other's
            # grid, so every distance near a tie is exact in float64
            d = np.abs(finite_vals - a)
            cands = finite_codes[d == d.min()]
        else:
            # exact rational distances (float64 would lose the 448-sized gaps)
            fa = Fraction(a) if np.isfinite(a) else Fraction(10) ** 400
            d = [abs(Fraction(float(x)) - fa) for x in finite_vals]
            best = min(d)
            cands = finite_codes[[i for i, x in enumerate(d) if x == best]]
        even = [c for c in cands if c % 2 == 0]
        code = int(even[0] if even else cands[0])
        out[idx] = code | (0x80 if np.signbit(v) else 0)
    return out


def test_decode_matches_ocp_spec():
    with open(os.path.join(GOLDEN, "e4m3_ocp_values.txt")) as fh:
        rows = [ln.split() for ln in fh if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 20
    for code_s, val_s in rows:
        v = e4m3.decode_code(int(code_s, 16))
        if val_s == "nan":
            assert np.isnan(v)
        else:
            ref = float(val_s)
            assert v == ref and np.signbit(v) == np.signbit(ref), code_s


def test_table_is_monotone_and_symmetric():
    t = e4m3.decode_table()
    pos = t[:0x7F]
    assert np.all(np.diff(pos) > 0)
    assert pos[-1] == 448.0
    assert np.all(t[0x80:0xFF] == -pos)
    assert np.isnan(t[0x7F]) and np.isnan(t[0xFF])
    # 254 distinct finite values (+0 and -0 compare equal)
    assert len(set(t[np.isfinite(t)].tolist())) == 253


def _probe_values():
    t = e4m3.decode_table()
    pos = t[:0x7F]
    mids = 0.5 * (pos[1:] + pos[:-1])
    vals = [pos, mids, [448.0, 449.0, 463.99997, 464.0, 464.00003, 480.0, 1e6, 3e38,
                        np.inf, 2.0 ** -10, 2.0 ** -11, 2.0 ** -126, 1e-45]]
    base = np.concatenate([np.asarray(v, dtype=np.float64) for v in vals]).astype(np.float32)
    up = np.nextafter(base, np.float32(np.inf))
    dn = np.nextafter(base, np.float32(0))
    allv = np.concatenate([base, up, dn])
    allv = allv[np.isfinite(allv) | np.isinf(allv)]
    return np.concatenate([allv, -allv, np.array([0.0, -0.0, np.nan], dtype=np.float32)])


def test_quantize_equals_brute_force_on_midpoints_and_codes():
    y = _probe_values()
    got = e4m3.quantize(y)
    ref = brute_force_codes(y)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(float(y[i]), hex(got[i]), hex(ref[i])) for i in bad[:10]]


def test_quantize_equals_brute_force_random():
    rng = np.random.default_rng(7)
    # random float32 bit patterns spanning every exponent, plus dense values near the range
    bits = rng.integers(0, 2 ** 32, size=20000, dtype=np.uint64).astype(np.uint32)
    y = np.concatenate([bits.view(np.float32),
                        rng.uniform(-500, 500, 20000).astype(np.float32),
                        rng.uniform(-0.05, 0.05, 20000).astype(np.float32)])
    np.testing.assert_array_equal(e4m3.quantize(y), brute_force_codes(y))


def test_special_values():
    y = np.array([0.0, -0.0, np.nan, -np.nan, np.inf, -np.inf, 448.0, -448.0, 1e-30, -1e-30],
                 dtype=np.float32)
    q = e4m3.quantize(y)
    assert list(q) == [0x00, 0x80, 0x7F, 0x7F, 0x7E, 0xFE, 0x7E, 0xFE, 0x00, 0x80]


def test_matches_torch_float8_e4m3fn_inside_range():
    rng = np.random.default_rng(3)
    y = np.concatenate([rng.uniform(-448, 448, 50000),
                        rng.standard_normal(50000) * 0.01]).astype(np.float32)
    ours = e4m3.quantize(y)
    theirs = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(ours, theirs)


def test_dequantize_round_trips_every_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    vals = e4m3.dequantize(codes).astype(np.float32)
    np.testing.assert_array_equal(e4m3.quantize(vals), codes)

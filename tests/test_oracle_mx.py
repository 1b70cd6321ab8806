"""Pins of the MXFP4 oracle (CPU only): OCP MX v1.0 definitions written out
independently of oracle.mx's table and search."""

import numpy as np

from oracle import mx


def test_e2m1_values_from_the_format():
    # the eight magnitudes the OCP specification lists for E2M1
    assert mx.E2M1_TABLE[:8].tolist() == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert mx.E2M1_TABLE[8:].tolist() == [-0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]
    assert np.signbit(mx.E2M1_TABLE[8])


def test_rounding_midpoints_ties_to_even_and_saturation():
    # (value, expected magnitude): midpoints go to the neighbour whose code is
    # even (mantissa bit 0), just off a midpoint to the nearer neighbour
    cases = [(0.25, 0.0), (0.2500001, 0.5), (0.75, 1.0), (0.7499999, 0.5), (1.25, 1.0),
             (1.2500001, 1.5), (1.75, 2.0), (2.5, 2.0), (2.5000002, 3.0), (3.5, 4.0),
             (3.4999998, 3.0), (5.0, 4.0), (5.0000005, 6.0), (6.0, 6.0), (7.99, 6.0), (1e30, 6.0),
             (0.0, 0.0), (1e-30, 0.0)]
    for v, want in cases:
        for sgn in (1.0, -1.0):
            c = int(mx.round_e2m1(np.array([sgn * v]))[0])
            assert mx.E2M1_TABLE[c] == sgn * want, (v, sgn, c)
    assert int(mx.round_e2m1(np.array([-0.0]))[0]) == 8        # sign of zero kept


def test_rounding_is_nearest_on_random_values():
    rng = np.random.default_rng(3)
    y = rng.uniform(-6.0, 6.0, 20000)
    c = mx.round_e2m1(y)
    got = np.abs(mx.E2M1_TABLE[c] - y)
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], dtype=np.float64)
    best = np.min(np.abs(np.abs(y)[:, None] - grid), axis=1)
    assert np.allclose(got, best, rtol=0, atol=0)


def test_scale_closed_forms():
    # X = 2^(floor(log2 amax) - 2): amax 6 -> X = 1 (byte 127), amax 8 -> X = 2,
    # amax just below 8 -> X = 1 and the top element saturates to 6
    for amax, byte in [(6.0, 127), (8.0, 128), (7.99, 127), (4.0, 127), (3.99, 126), (1.0, 125),
                       (2.0 ** -120, 127 - 122), (0.0, 0), (2.0 ** -140, 0), (np.inf, 255),
                       (np.nan, 255)]:
        assert int(mx.block_scale_exp(np.array([amax]))[0]) == byte, amax
    v = np.zeros((1, 1, 32), np.float32)
    v[0, 0, 0] = 7.5
    v[0, 0, 1] = 0.3
    codes, scales = mx.quantize(v)
    assert scales[0, 0, 0] == 127
    assert mx.dequantize(codes, scales)[0, 0, 0] == 6.0
    assert mx.dequantize(codes, scales)[0, 0, 1] == 0.5


def test_blocks_zero_nan_and_error_bound():
    rng = np.random.default_rng(5)
    U = (rng.standard_normal((2, 3, 96)) * np.exp(rng.uniform(-20, 20, (2, 3, 1)))).astype(np.float32)
    U[0, 1, 32:64] = 0.0
    U[1, 2, 70] = np.nan
    codes, scales = mx.quantize(U)
    assert scales.shape == (2, 3, 3)
    assert scales[0, 1, 1] == 0 and np.all(codes[0, 1, 32:64] == 0)
    assert scales[1, 2, 2] == 255 and np.all(np.isnan(mx.dequantize(codes, scales)[1, 2, 64:]))
    deq = mx.dequantize(codes, scales)
    X = np.ldexp(1.0, scales.astype(np.int64) - 127)
    ok = np.isfinite(deq)
    Xe = np.repeat(X, 32, axis=-1)
    unsat = ok & (np.abs(U) <= 6 * Xe)
    # below saturation every element lies within half a grid step, and the
    # grid step of E2M1 at magnitude a is at most a / 2 (at least 0.5 X)
    err = np.abs(deq.astype(np.float64) - U)
    assert np.all(err[unsat] <= np.maximum(0.25 * Xe[unsat], np.abs(U[unsat]) / 4 + 1e-30) + 1e-30)


def test_pack_and_rank_sum():
    c = np.arange(16, dtype=np.uint8).reshape(1, 1, 16)
    p = mx.pack(c)
    assert p.tolist() == [[[0x10, 0x32, 0x54, 0x76, 0x98, 0xBA, 0xDC, 0xFE]]]
    assert np.array_equal(mx.unpack(p), c)
    # exact sums of representable values
    codes = np.zeros((3, 1, 32), np.uint8)
    codes[:, 0, 0] = [2, 4, 7]          # 1, 2, 6 at scale 2^0
    scales = np.full((3, 1, 1), 127, np.uint8)
    assert mx.reduce_local(codes, scales)[0, 0] == np.float32(3.0)

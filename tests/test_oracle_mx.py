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


def _e2m1_half_step(a):
    """Half the distance to the next E2M1 magnitude above |a| (scaled units):
    grid 0, 0.5, 1, 1.5, 2, 3, 4, 6, written out from the format's fields
    (spacing 0.5 below 2, 1 from 2 to 4, 2 from 4 to 6)."""
    a = np.abs(a)
    return np.where(a < 2.0, 0.25, np.where(a < 4.0, 0.5, 1.0))


def test_residual_is_exact_by_sterbenz():
    # Error feedback keeps R = fl32(U - deq).  Below saturation deq is U
    # rounded to the nearest grid value, which lies within a factor 2 of U
    # (or is 0, and then R = U); above it deq = 6 X and U < 8 X (X is the
    # block's power-of-two scale), again within a factor 2.  So by Sterbenz
    # the subtraction is exact: deq + R == U with no rounding anywhere.
    rng = np.random.default_rng(11)
    U = (rng.standard_normal((3, 4, 128)) * np.exp(rng.uniform(-30, 30, (3, 4, 1)))).astype(np.float32)
    U[0, 0, :32] = np.float32(2.0 ** -130)      # subnormal block: X = 2^-127 floor
    U[1, 2, 32:64] = np.clip(U[1, 2, 32:64], -0.1, 0.1)
    U[1, 2, 40] = np.float32(7.5 * 2.0 ** -3)   # block max 7.5 X with X = 2^-3: saturates
    U[2, 1, 64:96] = 0.0
    codes, scales = mx.quantize(U)
    deq = mx.dequantize(codes, scales)
    R = mx.residual(U, codes, scales)
    assert R.dtype == np.float32
    np.testing.assert_array_equal(deq.astype(np.float64) + R.astype(np.float64), U.astype(np.float64))
    # the zero block leaves a zero residual; the saturated element leaves
    # U - 6 X, at most a third of U
    assert np.all(R[2, 1, 64:96] == 0)
    X = np.ldexp(1.0, scales.astype(np.int64) - 127)
    Xe = np.repeat(X, 32, axis=-1)
    sat = np.abs(U) > 6 * Xe
    assert sat[1, 2, 40]
    assert np.all(np.abs(R[sat]) < np.abs(U[sat]) / 3)


def test_residual_is_within_half_a_grid_step_below_saturation():
    rng = np.random.default_rng(12)
    U = (rng.uniform(-1, 1, (2, 8, 64)) * np.exp(rng.uniform(-8, 8, (2, 8, 1)))).astype(np.float32)
    codes, scales = mx.quantize(U)
    R = mx.residual(U, codes, scales).astype(np.float64)
    X = np.repeat(np.ldexp(1.0, scales.astype(np.int64) - 127), 32, axis=-1)
    y = U.astype(np.float64) / X                     # scaled value, exact (X a power of two)
    unsat = np.abs(y) <= 6.0
    assert unsat.mean() > 0.9
    # |R| <= half the grid spacing at the scaled value, times X; a residual
    # of the wrong sign or a dropped scale would break this or the identity
    # of the previous test
    assert np.all(np.abs(R[unsat]) <= _e2m1_half_step(y[unsat]) * X[unsat])
    # and it is the signed remainder: deq = U - R is a grid value times X
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], dtype=np.float64)
    g = np.abs((U.astype(np.float64) - R) / X)
    assert np.all(np.min(np.abs(g[..., None] - grid), axis=-1) == 0)


def test_residual_of_a_nan_block_is_nan():
    U = np.ones((1, 1, 64), np.float32)
    U[0, 0, 3] = np.nan
    U[0, 0, 40] = np.inf
    codes, scales = mx.quantize(U)
    R = mx.residual(U, codes, scales)
    assert np.all(np.isnan(R[0, 0, :32]))        # NaN scale: every element NaN
    assert np.all(np.isnan(R[0, 0, 32:64]))      # inf block: NaN scale as well

"""Pins of the oracle's iterative factor (CPU only).

The float64 subspace-iteration mirror is fixed by the published Philox
known-answer vectors, by orthonormality/reconstruction of Cholesky QR, and by
convergence to the exact eigendecomposition (``codec.lowrank_factor``) where
theory guarantees it: spiked spectra with a large gap.
"""

import os

import numpy as np
import pytest

from oracle import codec, subspace
from synth import factor_inputs, haar

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as fh:
        rows = [ln.split() for ln in fh if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for row in rows:
        v = [int(x, 16) for x in row]
        out = subspace.philox4x32_10(*v[:6])
        assert [int(o) for o in out] == v[6:]


def test_start_block_range_and_exactness():
    Q = subspace.start_block(50, 12, seed=123456789012)
    assert Q.shape == (50, 12)
    assert np.all(Q >= -1) and np.all(Q < 1)
    np.testing.assert_array_equal(Q.astype(np.float32).astype(np.float64), Q)
    # entries are multiples of 2^-23 and the block has full column rank
    np.testing.assert_array_equal(np.round(Q * 2 ** 23), Q * 2 ** 23)
    assert np.linalg.matrix_rank(Q) == 12
    # different seeds / entries differ (counter-based: no repeats)
    assert not np.array_equal(Q, subspace.start_block(50, 12, seed=1))


def test_cholqr2_orthonormal_basis():
    rng = np.random.default_rng(0)
    Y = rng.standard_normal((200, 16)) * np.logspace(0, -3, 16)   # cond ~ 1e3
    Q = subspace.cholqr2(Y)
    np.testing.assert_allclose(Q.T @ Q, np.eye(16), atol=1e-13)
    # span is preserved: Y = Q (Q^T Y)
    np.testing.assert_allclose(Q @ (Q.T @ Y), Y, atol=1e-12)
    R = subspace.cholesky_upper(Y.T @ Y)
    np.testing.assert_allclose(R.T @ R, Y.T @ Y, rtol=1e-12, atol=1e-15)
    assert np.allclose(R, np.triu(R))


def test_cholesky_floor_keeps_rank_deficient_blocks_finite():
    Y = np.zeros((30, 6))
    Y[:, :2] = np.random.default_rng(1).standard_normal((30, 2))
    Q = subspace.cholqr2(Y)
    assert np.all(np.isfinite(Q))
    np.testing.assert_allclose(Q[:, :2].T @ Q[:, :2], np.eye(2), atol=1e-12)


def test_converges_to_exact_factor_on_spiked_spectrum():
    dim, r = 96, 6
    q = haar(np.random.default_rng(2), dim, dim)
    spec = np.full(dim, 0.05)
    spec[:r] = [10.0, 7.0, 5.0, 3.0, 2.0, 1.5]
    A = (q * spec) @ q.T
    exact = codec.lowrank_factor(A, r)
    f, Q = subspace.subspace_factor(A, r, iters=6, seed=7)
    np.testing.assert_allclose(f.lam, exact.lam, rtol=1e-10)
    assert f.sigma2 == pytest.approx(exact.sigma2, rel=1e-10)
    np.testing.assert_allclose(f.inverse_root(), exact.inverse_root(), atol=1e-9)
    np.testing.assert_allclose(Q.T @ Q, np.eye(2 * r), atol=1e-12)


def test_power_law_capture_and_warm_start():
    X, _ = factor_inputs(77, 2048, 256)
    A = codec.factor_statistics(X)
    r = 16
    exact = codec.lowrank_factor(A, r)
    f, Q = subspace.subspace_factor(A, r, iters=10, seed=3)
    w = np.sort(np.linalg.eigvalsh(A))[::-1]
    captured = np.trace(f.U.T @ A @ f.U) / w[:r].sum()
    assert captured > 0.999
    # subspace angle between the iterative and exact top-r spaces
    s = np.linalg.svd(exact.U.T @ f.U, compute_uv=False)
    assert s.min() > 0.9
    # warm start: one more iteration from the returned block changes little
    f2, _ = subspace.subspace_factor(A, r, iters=1, seed=3, start=Q)
    np.testing.assert_allclose(f2.lam, f.lam, rtol=2e-2)


def test_rank_zero_and_zero_trace_are_identity():
    f, Q = subspace.subspace_factor(np.eye(10), 0, iters=3)
    assert f.rank == 0 and Q is None
    f, _ = subspace.subspace_factor(np.zeros((10, 10)), 3, iters=3)
    np.testing.assert_array_equal(f.inverse_root(), np.eye(10))

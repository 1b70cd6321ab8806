"""Pins of the oracle's codec (CPU only).

Each test fixes part of ``oracle.codec`` by something other than the code
itself: closed forms, identities the paper states (eq. design_kfac_norm_vec /
trace, design_sphere_proof, design_vec_whiten, design_input_side_sphere), the
identity-transform special case (Euclidean FP8), exact arithmetic on inputs
chosen to be representable, and the paper's own printed metrics.
"""

import os

import numpy as np
import pytest
import scipy.linalg

from oracle import codec, e4m3
from synth import factor_inputs, gradient_set, haar, layer_gradients

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(s=0):
    return np.random.default_rng(s)


def _spiked(dim, lams, sigma2, seed=1):
    """A = Q diag(lams, sigma2, ..., sigma2) Q^T built exactly from a Haar Q."""
    q = haar(_rng(seed), dim, dim)
    spec = np.full(dim, sigma2)
    spec[:len(lams)] = lams
    return (q * spec) @ q.T, q


# ---------------------------------------------------------------- statistics

def test_statistics_orthogonal_columns_give_diagonal():
    T, n = 64, 8
    q = haar(_rng(2), T, n)
    norms = np.arange(1, n + 1, dtype=np.float64)
    X = q * norms                      # orthogonal columns with known norms
    A = codec.factor_statistics(X)
    np.testing.assert_allclose(A, np.diag(norms ** 2 / T), atol=1e-14)


def test_statistics_psd_and_scale():
    X, _ = factor_inputs(5, 256, 32)
    A = codec.factor_statistics(X)
    assert np.allclose(A, A.T)
    assert np.linalg.eigvalsh(A).min() > -1e-12
    # E[x x^T] of 2x is 4 E[x x^T]
    np.testing.assert_allclose(codec.factor_statistics(2 * X.astype(np.float64)), 4 * A, rtol=1e-13)


# ---------------------------------------------------------------- low-rank factor

def test_spiked_covariance_closed_form():
    dim, lams, s2 = 40, np.array([9.0, 4.0, 2.5, 1.7]), 0.3
    A, q = _spiked(dim, lams, s2)
    f = codec.lowrank_factor(A, 4)
    assert f.sigma2 == pytest.approx(s2, rel=1e-12)
    expect = np.eye(dim) + (q[:, :4] * (np.sqrt(s2 / lams) - 1.0)) @ q[:, :4].T
    np.testing.assert_allclose(f.inverse_root(), expect, atol=1e-12)
    np.testing.assert_allclose(f.c_inv, np.sqrt(lams / s2) - 1.0, rtol=1e-12)


def test_whitening_identity():
    A = codec.factor_statistics(factor_inputs(9, 400, 24)[0])
    for r in (1, 5, 12):
        f = codec.lowrank_factor(A, r)
        w, v = np.linalg.eigh(A)
        w, v = w[::-1], v[:, ::-1]
        Ar = (v[:, :r] * f.lam) @ v[:, :r].T + f.sigma2 * (np.eye(24) - v[:, :r] @ v[:, :r].T)
        Si = f.inverse_root()
        np.testing.assert_allclose(Si @ Ar @ Si, f.sigma2 * np.eye(24), atol=1e-12 * np.trace(A))
        # S is the sigma-normalised symmetric root of A_r
        S = f.root()
        np.testing.assert_allclose(S @ S * f.sigma2, Ar, atol=1e-12 * np.trace(A))


def test_full_rank_is_sigma_times_inverse_sqrt():
    A = codec.factor_statistics(factor_inputs(11, 300, 16)[0])
    f = codec.lowrank_factor(A, 16)
    assert f.sigma2 == pytest.approx(np.trace(A) / 16, rel=1e-12)
    ref = np.sqrt(f.sigma2) * np.linalg.inv(np.real(scipy.linalg.sqrtm(A)))
    np.testing.assert_allclose(f.inverse_root(), ref, atol=1e-9)


def test_factor_is_invariant_to_scaling_A():
    A = codec.factor_statistics(factor_inputs(12, 200, 20)[0])
    f1, f2 = codec.lowrank_factor(A, 6), codec.lowrank_factor(7.5 * A, 6)
    np.testing.assert_allclose(f1.inverse_root(), f2.inverse_root(), atol=1e-12)


def test_coefficients_are_mutual_inverses_and_floor():
    A = codec.factor_statistics(factor_inputs(13, 200, 20)[0])
    f = codec.lowrank_factor(A, 8)
    np.testing.assert_allclose((1 + f.c_fwd) * (1 + f.c_inv), 1.0, rtol=1e-14)
    assert np.all(f.c_fwd <= 0) and np.all(f.c_inv >= 0)
    # rank-deficient A: the damping floor keeps sigma^2 positive
    X = np.zeros((50, 20)); X[:, :3] = _rng(4).standard_normal((50, 3))
    g = codec.lowrank_factor(codec.factor_statistics(X), 5, damping=1e-6)
    assert g.sigma2 == pytest.approx(1e-6 * np.trace(codec.factor_statistics(X)) / 20, rel=1e-9)
    assert np.all(np.isfinite(g.c_fwd))


# ---------------------------------------------------------------- transform / inverse

def test_forward_then_inverse_is_identity_float64():
    grads = gradient_set(1000, 1100, 2, 48, 40)
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(1001, 256, 40)[0]), 8)
    fG = codec.lowrank_factor(codec.factor_statistics(factor_inputs(1002, 256, 48)[0]), 8)
    for a, g in ((fA, None), (None, fG), (fA, fG)):
        back = codec.inverse(codec.forward(grads, a, g), a, g)
        rel = np.linalg.norm(back - grads) / np.linalg.norm(grads)
        assert rel <= 1e-10


def test_two_sided_equals_kronecker_vec():
    # eq. design_vec_whiten with column-major vec, at 8 x 6
    m, n = 8, 6
    W = _rng(5).standard_normal((m, n))
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(21, 64, n)[0]), 2)
    fG = codec.lowrank_factor(codec.factor_statistics(factor_inputs(22, 64, m)[0]), 3)
    Wt = codec.forward(W, fA, fG)
    vec = lambda M: M.reshape(-1, order="F")
    np.testing.assert_allclose(vec(Wt), np.kron(fA.inverse_root(), fG.inverse_root()) @ vec(W),
                               atol=1e-12)


def test_kfac_norm_vec_trace_and_sphere():
    # eq. design_kfac_norm_vec == eq. design_kfac_norm_trace == ||L_G^T dW L_A||_F^2
    m, n = 7, 5
    rng = _rng(6)
    dW = rng.standard_normal((m, n))
    A = codec.factor_statistics(rng.standard_normal((40, n))) + 0.1 * np.eye(n)
    G = codec.factor_statistics(rng.standard_normal((40, m))) + 0.1 * np.eye(m)
    vec = dW.reshape(-1, order="F")
    v1 = vec @ np.kron(A, G) @ vec
    v2 = np.trace(A @ dW.T @ G @ dW)
    LA, LG = np.linalg.cholesky(A), np.linalg.cholesky(G)
    v3 = np.linalg.norm(LG.T @ dW @ LA) ** 2
    assert v1 == pytest.approx(v2, rel=1e-12) and v2 == pytest.approx(v3, rel=1e-12)
    # eq. design_input_side_sphere
    assert np.trace(A @ dW.T @ dW) == pytest.approx(np.linalg.norm(dW @ LA) ** 2, rel=1e-12)


def test_sigma_normalised_roots_give_the_ball():
    # with S S = A_r / sigma^2:  ||S_G dW S_A||^2 = tr(A_r dW^T G_r dW) / (sigma_A^2 sigma_G^2)
    m, n = 12, 10
    rng = _rng(8)
    A = codec.factor_statistics(rng.standard_normal((80, n)) * np.linspace(3, 0.2, n))
    G = codec.factor_statistics(rng.standard_normal((80, m)) * np.linspace(2, 0.3, m))
    fA, fG = codec.lowrank_factor(A, 3), codec.lowrank_factor(G, 4)
    SA, SG = fA.root(), fG.root()
    Ar, Gr = fA.sigma2 * SA @ SA, fG.sigma2 * SG @ SG
    dW = rng.standard_normal((m, n))
    lhs = np.linalg.norm(SG @ dW @ SA) ** 2
    rhs = np.trace(Ar @ dW.T @ Gr @ dW) / (fA.sigma2 * fG.sigma2)
    assert lhs == pytest.approx(rhs, rel=1e-10)


# ---------------------------------------------------------------- scale and quantize

def test_identity_transform_is_euclidean_fp8():
    grads = gradient_set(2000, 2100, 3, 32, 48)
    base_codes, base_s, wt = codec.encode(grads, None, None)
    np.testing.assert_array_equal(wt, grads)
    # direct Euclidean FP8: codes of fl32(x * fl32(448/amax)) per rank
    for j in range(3):
        a = np.float32(np.abs(grads[j]).max())
        inv = np.float32(448.0) / a
        np.testing.assert_array_equal(base_codes[j], e4m3.quantize((grads[j] * inv).astype(np.float32)))
        assert base_s[j, 0, 0] == np.float32(a / np.float32(448.0))
    # a factor whose coefficients are zero, and a rank-0 factor, are the identity
    zero = codec.Factor(haar(_rng(3), 48, 4), np.zeros(4), np.zeros(4), 1.0)
    for f in (zero, codec.identity_factor(48)):
        c, s, _ = codec.encode(grads, f, None)
        np.testing.assert_array_equal(c, base_codes)
        np.testing.assert_array_equal(s, base_s)


def test_amax_element_maps_to_448_and_zero_blocks():
    grads = gradient_set(3000, 3100, 2, 40, 64)
    grads[1, :, 32:] = 0.0
    codes, s, _ = codec.encode(grads, block_cols=32)
    for j in range(2):
        for b in range(2):
            blk = grads[j, :, 32 * b:32 * (b + 1)]
            if not blk.any():
                assert s[j, 0, b] == 0.0
                assert np.all(codes[j, :, 32 * b:32 * (b + 1)] == 0)
                continue
            i = np.unravel_index(np.argmax(np.abs(blk)), blk.shape)
            assert codes[j, i[0], 32 * b + i[1]] in (0x7E, 0xFE)


def test_shared_scale_is_max_over_ranks():
    grads = gradient_set(3500, 3600, 4, 16, 16)
    grads[2] *= 3.0
    _, s_loc = codec.quantize_transformed(grads)
    _, s_sh = codec.quantize_transformed(grads, shared=True)
    assert np.all(s_sh == s_loc.max(axis=0))


def test_block_grid_partial_edges():
    assert codec.block_grid(100, 300, 0, 128) == (100, 128, 1, 3)
    assert codec.block_grid(100, 300, 30, 0) == (30, 300, 4, 1)
    Wt = np.arange(2 * 5 * 7, dtype=np.float32).reshape(2, 5, 7)
    am = codec.block_amax(Wt, 2, 3)
    assert am.shape == (2, 3, 3)
    assert am[1, 2, 2] == Wt[1, 4, 6] and am[0, 0, 0] == Wt[0, 1, 2]


def test_block_amax_nan_wins():
    # A NaN anywhere in a block makes that block's maximum NaN (and with it
    # the scale and every code of the block), so a NaN gradient cannot pass
    # as a finite one.  A maximum that skips NaN (np.nanmax) fails this.
    Wt = np.arange(2 * 4 * 6, dtype=np.float32).reshape(2, 4, 6) - 20.0
    Wt[1, 3, 1] = np.nan
    am = codec.block_amax(Wt, 2, 3)
    assert np.isnan(am[1, 1, 0])
    finite = ~np.isnan(am)
    assert finite.sum() == am.size - 1
    # the other blocks keep their plain maxima of |x|
    assert am[1, 1, 1] == np.abs(Wt[1, 2:4, 3:6]).max()
    assert am[0, 0, 0] == 20.0 and am[1, 0, 0] == np.abs(Wt[1, 0:2, 0:3]).max()
    s, inv = codec.scales_from_amax(am)
    assert np.isnan(s[1, 1, 0])
    codes = codec.quantize_blocks(Wt, inv, 2, 3)
    assert np.all(codes[1, 2:4, 0:3] & 0x7F == 0x7F)    # every code of the block is NaN
    # an infinity is an ordinary maximum: inf amax, scale inf, multiplier 0
    Wi = np.ones((1, 2, 2), np.float32)
    Wi[0, 0, 0] = -np.inf
    ai = codec.block_amax(Wi)
    assert np.isposinf(ai[0, 0, 0])


def test_scale_edge_cases():
    s, inv = codec.scales_from_amax(np.array([0.0, 448.0, np.inf, 1e-40], dtype=np.float32))
    assert s[0] == 0 and inv[0] == 0
    assert s[1] == 1.0 and inv[1] == 1.0
    assert np.isinf(s[2]) and inv[2] == 0
    assert inv[3] == np.finfo(np.float32).max


# ---------------------------------------------------------------- Cholesky-form variants

def _psd(dim, seed, decay=1.2):
    x = factor_inputs(seed, 4 * dim, dim, decay=decay)[0].astype(np.float64)
    return codec.factor_statistics(x)


def test_chol_full_gives_the_inverse_metric_norm():
    # ||W L^-T||_F^2 = tr(W (A + dI)^-1 W^T): the gradient's norm under the
    # inverse of the input-side metric (eq. design_input_side_sphere dualised);
    # a transposed factor (W L^-1) or a dropped shift fails it
    A = _psd(24, 3)
    damp = 1e-3
    f = codec.chol_factor(A, 0, damp)
    Areg = A + codec.chol_shift(A, damp) * np.eye(24)
    W = _rng(5).standard_normal((9, 24))
    Wt = codec.forward(W, f)
    want = np.trace(W @ np.linalg.inv(Areg) @ W.T)
    assert np.isclose((Wt ** 2).sum(), want, rtol=1e-10)
    L = f.lower()
    assert np.allclose(np.triu(L, 1), 0.0) and np.all(np.diag(L) > 0)
    assert np.allclose(L @ L.T, Areg, rtol=1e-12, atol=1e-12 * np.abs(Areg).max())


def test_chol_two_sided_is_the_kronecker_whitening():
    # ||L_G^-1 W L_A^-T||^2 = vec(W)^T (A^-1 kron G^-1) vec(W) (eq. design_vec_whiten)
    A, G = _psd(7, 11), _psd(5, 12)
    fA, fG = codec.chol_factor(A, 0, 1e-2), codec.chol_factor(G, 0, 1e-2)
    Ar = A + codec.chol_shift(A, 1e-2) * np.eye(7)
    Gr = G + codec.chol_shift(G, 1e-2) * np.eye(5)
    W = _rng(6).standard_normal((5, 7))
    Wt = codec.forward(W, fA, fG)
    v = W.reshape(-1, order="F")
    want = v @ np.kron(np.linalg.inv(Ar), np.linalg.inv(Gr)) @ v
    assert np.isclose((Wt ** 2).sum(), want, rtol=1e-10)
    assert np.allclose(codec.inverse(Wt, fA, fG), W, rtol=1e-10, atol=1e-12)


def test_chol_diag_is_column_scaling():
    A = _psd(20, 4)
    damp = 1e-4
    f = codec.chol_factor(A, 1, damp)
    d = np.diag(A) + damp * np.trace(A) / 20
    W = _rng(7).standard_normal((6, 20))
    assert np.allclose(codec.forward(W, f), W / np.sqrt(d), rtol=1e-13)
    assert np.allclose(codec.forward(W.T, None, f), W.T / np.sqrt(d)[:, None], rtol=1e-13)
    assert f.R.shape == (20, 1, 1)


def test_chol_block_matches_full_on_block_diagonal_matrices():
    # a block-diagonal A (blocks of 4, a ragged block of 2) has a
    # block-diagonal Cholesky factor, so block-A-4 equals full-A on it
    dim, b = 10, 4
    A = np.zeros((dim, dim))
    for k in range(0, dim, b):
        kv = min(b, dim - k)
        A[k:k + kv, k:k + kv] = _psd(kv, 20 + k) + 0.1 * np.eye(kv)
    fb, ff = codec.chol_factor(A, b, 1e-3), codec.chol_factor(A, 0, 1e-3)
    assert fb.R.shape == (3, 4, 4)
    assert np.allclose(fb.R[2, 2:, 2:], np.eye(2)) and np.allclose(fb.R[2, :2, 2:], 0)
    assert np.allclose(fb.lower(), ff.lower(), rtol=1e-12, atol=1e-14)
    W = _rng(8).standard_normal((3, dim))
    assert np.allclose(codec.forward(W, fb), codec.forward(W, ff), rtol=1e-12)
    # on a general A the blocks see only their own diagonal blocks of A
    G = _psd(dim, 30)
    g = codec.chol_factor(G, b, 1e-3)
    Gr = G + codec.chol_shift(G, 1e-3) * np.eye(dim)
    for k in range(0, dim, b):
        kv = min(b, dim - k)
        Lk = g.lower()[k:k + kv, k:k + kv]
        assert np.allclose(Lk @ Lk.T, Gr[k:k + kv, k:k + kv], rtol=1e-12)
    assert np.allclose(codec.chol_factor(G, dim, 1e-3).R, codec.chol_factor(G, 0, 1e-3).R)
    assert np.allclose(codec.chol_factor(G, 50, 1e-3).R, codec.chol_factor(G, 0, 1e-3).R)


def test_chol_round_trip_and_identity_cases():
    A = _psd(16, 9)
    for b in (0, 1, 5, 16):
        f = codec.chol_factor(A, b, 1e-6)
        W = _rng(b).standard_normal((4, 16))
        assert np.allclose(codec.inverse(codec.forward(W, f), f), W, rtol=1e-9, atol=1e-12)
    z = codec.chol_factor(np.zeros((6, 6)), 4, 1e-3)
    assert np.all(z.R == np.eye(4)) and np.all(z.Rinv == np.eye(4))


def test_layer_gradients_are_the_inputs_product():
    # the study's generator: every rank's gradient is D_j^T X_j / T up to the
    # one common rescale, so the factor statistics describe that gradient
    g, xa, xg = layer_gradients(3, 2, 64, 12, 20, spike_frac=1 / 32, spike=5.0)
    assert g.shape == (2, 12, 20) and xa.shape == (128, 20) and xg.shape == (128, 12)
    prods = [xg[64 * j:64 * (j + 1)].astype(np.float64).T @ xa[64 * j:64 * (j + 1)] / 64 for j in range(2)]
    c = g[0, 0, 0] / prods[0][0, 0]
    for j in range(2):
        assert np.allclose(g[j], c * prods[j], rtol=1e-5, atol=1e-12)


# ---------------------------------------------------------------- boundary hits

def test_boundary_hits_hand_example():
    # One block whose amax is 448, so the multiplier is exactly 1 and the
    # values are quantized as they stand.  In E4M3 the neighbours of 448 are
    # 416 (odd mantissa) and nothing above, so |y| >= 432 (the midpoint, tie
    # to the even 448) encodes to 448; the smallest subnormal is 2^-9, so
    # |y| <= 2^-10 (the midpoint, tie to the even zero) encodes to zero.
    t = 2.0 ** -10
    x = np.array([448, 432, 431.99, 447, -440, t, -t, t * 1.0001, 1e-30, 0.0, -0.0,
                  416, -2.0 ** -9, 1.0], dtype=np.float32)
    codes, s = codec.quantize_transformed(x.reshape(1, 1, -1))
    assert s[0, 0, 0] == 1.0
    hits = codec.boundary_hits(x.reshape(1, 1, -1), codes)
    assert hits.tolist() == [[4, 3]]


def test_boundary_hits_threshold_closed_form():
    rng = _rng(41)
    N, m, n = 3, 24, 40
    mag = np.exp(rng.uniform(np.log(1e-6), np.log(448.0), size=(N, m, n)))
    x = (mag * rng.choice([-1.0, 1.0], size=mag.shape)).astype(np.float32)
    x[:, 0, 0] = 448.0                     # every rank's amax: multiplier 1
    x[0, 1, :8] = 0.0
    x[1, 2, :5] = np.float32(2.0 ** -10)    # the lower tie
    x[2, 3, :5] = np.float32(432.0)         # the upper tie
    codes, s = codec.quantize_transformed(x)
    assert np.all(s == 1.0)
    a = np.abs(x)
    up = (a >= 432.0).reshape(N, -1).sum(axis=1)
    lo = ((a > 0) & (a <= 2.0 ** -10)).reshape(N, -1).sum(axis=1)
    hits = codec.boundary_hits(x, codes)
    assert hits[:, 0].tolist() == up.tolist()
    assert hits[:, 1].tolist() == lo.tolist()
    assert np.all(up >= 1) and lo[1] >= 5


def test_boundary_hits_every_block_max_is_an_upper_hit():
    grads = gradient_set(5000, 5100, 3, 64, 96)
    grads[2, :, 48:] = 0.0
    codes, s, Wt = codec.encode(grads, block_rows=32, block_cols=48)
    hits = codec.boundary_hits(Wt, codes)
    nonzero_blocks = (s > 0).reshape(3, -1).sum(axis=1)
    assert np.all(hits[:, 0] >= nonzero_blocks)
    # zero inputs are never lower hits; a shared scale can only add lower hits
    codes_sh = codec.quantize_transformed(Wt, 32, 48, shared=True)[0]
    assert np.all(codec.boundary_hits(Wt, codes_sh)[:, 1] >= hits[:, 1])


# ---------------------------------------------------------------- rank sum

def test_reduce_exact_on_representable_inputs():
    # values = E4M3 value * 2^-12 with the block amax at 448 * 2^-12: scale exactly 2^-12,
    # every step exact, so the mean is the exact float64 mean of the inputs
    rng = _rng(10)
    table = e4m3.decode_table()
    finite = table[np.isfinite(table)]
    N, m, n = 4, 9, 13
    vals = rng.choice(finite, size=(N, m, n)) * 2.0 ** -12
    vals[:, 0, 0] = 448.0 * 2.0 ** -12
    vals[:, 0, 1] = -448.0 * 2.0 ** -12
    g = vals.astype(np.float32)
    codes, s, _ = codec.encode(g)
    assert np.all(s == np.float32(2.0 ** -12))
    np.testing.assert_array_equal(e4m3.dequantize(codes) * 2.0 ** -12, vals)
    M = codec.reduce_local(codes, s)
    np.testing.assert_array_equal(M.astype(np.float64), vals.sum(axis=0) / N)


def test_reduce_single_rank_and_identical_ranks():
    g = gradient_set(4000, 4100, 1, 20, 30)
    codes, s, _ = codec.encode(g)
    M1 = codec.reduce_local(codes, s)
    np.testing.assert_array_equal(M1, (e4m3.dequantize(codes[0]) * s[0, 0, 0]).astype(np.float32))
    # two identical ranks: v + v is exact and /2 is exact
    c2, s2 = np.repeat(codes, 2, axis=0), np.repeat(s, 2, axis=0)
    np.testing.assert_array_equal(codec.reduce_local(c2, s2), M1)


def test_round_trip_error_is_fp8_sized():
    g = gradient_set(4500, 4600, 4, 64, 64)
    out = codec.round_trip(g)
    fid = codec.fidelity(out, g.astype(np.float64).mean(axis=0))
    # E4M3 has 3 mantissa bits: per-element relative error <= 2^-4 above the subnormals
    assert 5e-3 < fid["RelL2"] < 6.25e-2 and fid["Cos"] > 0.998


# ---------------------------------------------------------------- metrics

def test_fidelity_special_cases():
    g = _rng(11).standard_normal((5, 6))
    f = codec.fidelity(g, g)
    assert f["RelL2"] == 0 and f["Cos"] == pytest.approx(1.0) and f["MSE"] == 0
    f2 = codec.fidelity(2 * g, g)
    assert f2["RelL2"] == pytest.approx(1.0) and f2["Cos"] == pytest.approx(1.0)
    assert f2["MSE"] == pytest.approx(np.mean(g * g)) and f2["MaxErr"] == pytest.approx(np.abs(g).max())


def test_paper_metric_definitions_are_consistent():
    # Tables I-II measure one gradient g, so MSE / RelL2^2 = ||g||^2 / n on every row
    # (eq. recon_metrics); the 67.4% reduction follows from the RelL2 column.
    rows = {}
    with open(os.path.join(GOLDEN, "paper_table2_relL2.txt")) as fh:
        for ln in fh:
            if ln.strip() and not ln.startswith("#"):
                name, *vals = ln.split()
                rows[name] = [float(v) for v in vals]
    ratios = np.array([r[3] / r[0] ** 2 for r in rows.values()])
    assert ratios.std() / ratios.mean() < 2e-4
    red = 100 * (rows["euclidean"][0] - rows["lowrank_32"][0]) / rows["euclidean"][0]
    assert round(red, 1) == 67.4
    # the same relation holds for the oracle's metrics
    g = gradient_set(5000, 5100, 1, 30, 30)[0]
    fid = codec.fidelity(codec.round_trip(g[None]), g)
    assert fid["MSE"] / fid["RelL2"] ** 2 == pytest.approx(np.mean(g.astype(np.float64) ** 2), rel=1e-9)


# ---------------------------------------------- error feedback (Sec. V-E)

def test_error_feedback_zero_residual_is_plain_encode():
    grads = gradient_set(41, 42, 3, 24, 40)
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(43, 400, 40)[0]), 6).to_f32()
    codes, s, Ut, R = codec.encode_ef(grads, np.zeros_like(grads), fA, None, 0, 8)
    c0, s0, t0 = codec.encode(grads, fA, None, 0, 8)
    np.testing.assert_array_equal(codes, c0)
    np.testing.assert_array_equal(s, s0)
    np.testing.assert_array_equal(Ut, t0)
    # the residual is what the dequantized codes miss
    np.testing.assert_array_equal(R, (t0 - codec.dequantize_blocks(codes, s, 0, 8)).astype(np.float32))


def test_error_feedback_residual_is_exact_and_bounded():
    # Sterbenz: a value and its E4M3 round-off (relative error <= 2^-4 on
    # normals) are within a factor 2, so U~ - deq is exact and deq + R == U~
    rng = np.random.default_rng(7)
    U = (rng.standard_normal((2, 30, 50)) * 1e-3).astype(np.float32)
    R0 = (rng.standard_normal(U.shape) * 1e-5).astype(np.float32)
    codes, s, Ut, R = codec.encode_ef(U, R0)
    np.testing.assert_array_equal(Ut, (U + R0).astype(np.float32))
    deq = codec.dequantize_blocks(codes, s).astype(np.float64)
    np.testing.assert_array_equal(deq + R.astype(np.float64), Ut.astype(np.float64))
    # half an E4M3 spacing: 2^-4 relative on normals, 2^-10 s on subnormals
    bound = np.abs(Ut.astype(np.float64)) * 2.0 ** -4 + s.reshape(-1, 1, 1) * 2.0 ** -9
    assert np.all(np.abs(R) <= bound)


def test_error_feedback_telescopes():
    # sum of what was sent + the final residual == sum of the inputs
    rng = np.random.default_rng(8)
    R = np.zeros((1, 16, 24), np.float32)
    sent = np.zeros((1, 16, 24), np.float64)
    total = np.zeros((1, 16, 24), np.float64)
    for step in range(6):
        U = (rng.standard_normal(R.shape) * 10.0 ** -(step % 3)).astype(np.float32)
        codes, s, Ut, R = codec.encode_ef(U, R)
        sent += codec.dequantize_blocks(codes, s)
        total += U
    np.testing.assert_allclose(sent + R, total, rtol=0, atol=1e-6 * np.abs(total).max())

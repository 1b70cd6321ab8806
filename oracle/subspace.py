"""Iterative rank-r factor (float64 mirror) -- test infrastructure only.

The paper approximates the input-side factor by its leading eigenpairs
(Sec. V-B, eq. impl_A_lowrank) and refreshes it every K steps (Sec. V-E,
Algorithm 1) but does not say how the eigenpairs are obtained.  The GPU path
uses block subspace iteration with Rayleigh-Ritz extraction; this module is
that algorithm in float64 so that the GPU factor can be checked against the
same method.  ``codec.lowrank_factor`` (exact eigendecomposition) remains the
definition of the factor; this mirror is pinned to it on spiked spectra, where
the iteration provably converges.

Algorithm (block subspace iteration, e.g. Golub & Van Loan, "Matrix
Computations", Sec. 8.2.4, with Rayleigh-Ritz, Sec. 8.1.6):

1. ``k = min(dim, 2r)`` columns (oversampling p = r).  The start block ``Q0``
   comes from the counter-based generator below (or from the previous
   refresh).
2. Orthonormalize by Cholesky QR applied twice (CholeskyQR2: Fukaya, Nakatsukasa,
   Yanagisawa, Yamamoto, 2014): ``R = chol(Y^T Y)``, ``Q = Y R^-1``.  Pivots are
   floored at ``1e-12 * tr(Y^T Y) / k`` so a rank-deficient block cannot
   produce NaN.
3. ``iters`` times: ``Q <- CholQR2(A Q)``.
4. Rayleigh-Ritz: ``B = Q^T A Q`` (symmetrised), ``B = V diag(theta) V^T`` with
   theta descending; ``U = Q V[:, :r]``, ``lambda = max(theta[:r], 0)``.
5. ``sigma^2`` and the coefficients as in ``codec.coefficients``.

Random start: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11).  Entry ``(i, j)`` of the ``dim x k``
start block is word 0 of Philox4x32-10 with counter ``(i, j, 0, 0)`` and key
``(seed mod 2^32, seed div 2^32)``, read as a signed 32-bit integer, shifted
right arithmetically by 8 and multiplied by ``2^-23``: a value in [-1, 1) that
float32 represents exactly, so both sides start from identical numbers.
"""

from __future__ import annotations

import numpy as np

from .codec import Factor, coefficients, identity_factor

_MASK = np.uint64(0xFFFFFFFF)
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32 with 10 rounds on uint32 arrays; returns four uint32 arrays."""
    c = [np.asarray(x, dtype=np.uint64) & _MASK for x in (c0, c1, c2, c3)]
    k0 = np.uint64(int(k0) & 0xFFFFFFFF)
    k1 = np.uint64(int(k1) & 0xFFFFFFFF)
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    for rnd in range(10):
        if rnd > 0:
            k0 = np.uint64((int(k0) + PHILOX_W0) & 0xFFFFFFFF)
            k1 = np.uint64((int(k1) + PHILOX_W1) & 0xFFFFFFFF)
        p0 = m0 * c[0]
        p1 = m1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return [x.astype(np.uint32) for x in c]


def start_block(dim: int, k: int, seed: int) -> np.ndarray:
    """``dim x k`` start block with entries in [-1, 1) (exact float32 values)."""
    i, j = np.meshgrid(np.arange(dim, dtype=np.uint64), np.arange(k, dtype=np.uint64),
                       indexing="ij")
    z = np.zeros_like(i)
    w0 = philox4x32_10(i, j, z, z, seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)[0]
    return (w0.view(np.int32) >> 8).astype(np.float64) * 2.0 ** -23


def cholesky_upper(G: np.ndarray) -> np.ndarray:
    """Upper ``R`` with ``R^T R = G`` (column by column), pivots floored."""
    G = np.asarray(G, dtype=np.float64)
    k = G.shape[0]
    floor = 1e-12 * max(float(np.trace(G)), 0.0) / max(k, 1) + 1e-300
    R = np.zeros_like(G)
    for j in range(k):
        d = G[j, j] - R[:j, j] @ R[:j, j]
        R[j, j] = np.sqrt(max(d, floor))
        if j + 1 < k:
            R[j, j + 1:] = (G[j, j + 1:] - R[:j, j] @ R[:j, j + 1:]) / R[j, j]
    return R


def cholqr2(Y: np.ndarray) -> np.ndarray:
    """Orthonormal basis of span(Y) by Cholesky QR applied twice."""
    Q = np.asarray(Y, dtype=np.float64)
    for _ in range(2):
        R = cholesky_upper(Q.T @ Q)
        Q = Q @ np.linalg.inv(R)
    return Q


def subspace_factor(A: np.ndarray, r: int, iters: int, seed: int = 0,
                    damping: float = 1e-6, start: np.ndarray | None = None):
    """Rank-r factor by subspace iteration; returns ``(Factor, Q)``.

    ``Q`` (dim x k) is the final orthonormal block, the warm start of the next
    refresh.  ``start`` overrides the generated start block.
    """
    A = np.asarray(A, dtype=np.float64)
    dim = A.shape[0]
    r = min(int(r), dim)
    trace = float(np.trace(A))
    if r == 0:
        return identity_factor(dim), None
    if trace <= 0.0:
        return Factor(np.zeros((dim, r)), np.zeros(r), np.zeros(r), 0.0, np.zeros(r)), None
    k = min(dim, 2 * r)
    Q = start_block(dim, k, seed) if start is None else np.asarray(start, np.float64)
    Q = cholqr2(Q)
    for _ in range(int(iters)):
        Q = cholqr2(A @ Q)
    B = Q.T @ (A @ Q)
    B = 0.5 * (B + B.T)
    th, V = np.linalg.eigh(B)
    order = np.argsort(th)[::-1]
    th, V = th[order], V[:, order]
    U = Q @ V[:, :r]
    sigma2, lam, c_fwd, c_inv = coefficients(np.maximum(th[:r], 0.0), trace, dim, damping)
    return Factor(U, c_fwd, c_inv, sigma2, lam), Q

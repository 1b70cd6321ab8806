"""GIFT codec reference (float64 numpy) -- test infrastructure only.

What the codec computes, step by step, in the paper's order (Algorithm 1 and
Sec. IV-A, V-A, V-B).  Notation follows the paper: a weight gradient
``W_g in R^{d_out x d_in}`` (eq. design_Wg), written ``W`` here with
``m = d_out`` and ``n = d_in``; input-side factor ``A = E[a a^T]`` (n x n) and
output-side factor ``G = E[delta delta^T]`` (m x m) (eq. kfac_fisher_block);
``N`` data-parallel ranks (eq. dp_grad_avg, Algorithm 1).

Readings where the paper is silent (each also listed with its reason in the
design notes of the repository):

* Low-rank transform (Sec. V-B, eq. impl_A_lowrank says only that the transform
  is built from ``U_r Lambda_r U_r^T``): the symmetric square root ``S`` of the
  rank-r-plus-isotropic model ``A_r = U_r Lambda_r U_r^T + sigma^2 (I - U_r
  U_r^T)``, normalised by ``sigma`` so that the complement maps to itself:
  ``S^-1 = I + U_r diag(c) U_r^T`` with ``c_i = sqrt(sigma^2/lambda_i) - 1`` and
  ``S = I + U_r diag(c') U_r^T`` with ``c'_i = sqrt(lambda_i/sigma^2) - 1``.
  ``sigma^2`` is the mean of the discarded eigenvalues, floored at
  ``damping * tr(A)/n`` (the "regularized" factors of eq. design_chol), and
  ``lambda_i`` is floored at ``sigma^2``.  With ``r = n`` nothing is discarded:
  ``sigma^2 = tr(A)/n`` only normalises, eigenvalues are floored at
  ``damping * tr(A)/n``, and ``S^-1 = sigma A^-1/2`` (the full-A input-side
  transform).  ``S`` plays the role of ``L_A``: any
  square root of ``A`` turns the metric ellipsoid into a ball
  (eq. design_sphere_proof).
* Cholesky-form variants (eq. design_chol with Table II's full-A, diag-A and
  block-A-b): ``L`` is the Cholesky factor of ``A + delta I`` with ``delta =
  damping * tr(A)/dim`` (the regularisation the equation asks for without
  fixing it); diag-A and block-A-b keep only the diagonal, or the ``b x b``
  diagonal blocks (the last one ragged), of ``A + delta I`` and factor those.
  No ``sigma`` normalisation: the amax scale absorbs a common factor.  A zero
  trace gives the identity.
* Scale (Algorithm 1's ``Scale``; the amax rule quoted from COAT in Sec. I):
  ``s = fl32(amax/448)`` is the stored (dequantization) scale and values are
  quantized as ``fl32(x * fl32(448/amax))``; amax = 0 gives s = 0 and a zero
  multiplier; a multiplier that overflows float32 is clamped to FLT_MAX.
* Rank sum under local scales (Algorithm 1 sums codes and dequantizes with the
  local scale, which is only well defined when the scales agree): every rank
  is dequantized with its own scale, the values are summed in float32 in rank
  order and divided by N (eq. dp_grad_avg).  With a shared scale this equals
  the algorithm's sum-then-dequantize up to float rounding.
* Blocks: ``block_rows x block_cols`` tiles of each rank's matrix, partial
  edge blocks allowed; 0 means the whole dimension.
* Boundary hits (Sec. V-C ranks layers by the frequency of FP8 values at
  the top and bottom of the format's range but leaves both undefined): an
  upper hit is a code of magnitude 448, the largest finite E4M3 value (under
  amax scaling every block's maximum lands there, and so does every
  saturated value); a lower hit is a nonzero value whose code is +-0, i.e.
  that underflowed.  NaN values count in neither.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import scipy.linalg

from . import e4m3

F32_MAX = np.float32(np.finfo(np.float32).max)


# --------------------------------------------------------------------------
# Kronecker-factor statistics (eq. kfac_fisher_block, eq. impl_A_psd)
# --------------------------------------------------------------------------

def factor_statistics(x: np.ndarray) -> np.ndarray:
    """Uncentred second moment ``E[x x^T] = X^T X / T`` in float64.

    ``x`` is ``[T, dim]`` (tokens by features).  Pins: orthogonal-column inputs
    give a known diagonal; the result is symmetric positive semidefinite.
    """
    x = np.asarray(x, dtype=np.float64)
    return (x.T @ x) / x.shape[0]


# --------------------------------------------------------------------------
# Low-rank factor (Sec. V-B, eq. impl_A_lowrank)
# --------------------------------------------------------------------------

@dataclass
class Factor:
    """One side's low-rank transform: ``S^-1 = I + U diag(c_fwd) U^T``."""

    U: np.ndarray          # [dim, r]
    c_fwd: np.ndarray      # [r]
    c_inv: np.ndarray      # [r]
    sigma2: float
    lam: np.ndarray = None  # [r] floored eigenvalues (informational)

    @property
    def dim(self) -> int:
        return self.U.shape[0]

    @property
    def rank(self) -> int:
        return self.U.shape[1]

    def to_f32(self) -> "Factor":
        """The factor as the GPU stores it (every field rounded to float32)."""
        f = lambda a: np.asarray(a, dtype=np.float32).astype(np.float64)
        return Factor(f(self.U), f(self.c_fwd), f(self.c_inv),
                      float(np.float32(self.sigma2)),
                      None if self.lam is None else f(self.lam))

    def inverse_root(self) -> np.ndarray:
        """Dense ``S^-1`` (dim x dim)."""
        return np.eye(self.dim) + (self.U * self.c_fwd) @ self.U.T

    def root(self) -> np.ndarray:
        """Dense ``S`` (dim x dim)."""
        return np.eye(self.dim) + (self.U * self.c_inv) @ self.U.T


def coefficients(lam_top: np.ndarray, trace: float, dim: int, damping: float):
    """``sigma^2``, floored eigenvalues and the forward/inverse coefficients.

    ``lam_top`` holds the r leading eigenvalues (descending, >= 0).
    Returns ``(sigma2, lam, c_fwd, c_inv)``; a zero trace gives the identity.
    """
    r = lam_top.shape[0]
    lam_top = np.maximum(np.asarray(lam_top, dtype=np.float64), 0.0)
    if trace <= 0.0 or r == 0:
        z = np.zeros(r)
        return 0.0, lam_top, z, z.copy()
    floor = damping * trace / dim
    if r >= dim:
        # nothing is discarded: sigma^2 only normalises, S^-1 = sigma A^-1/2
        sigma2 = trace / dim
        lam = np.maximum(lam_top, floor)
    else:
        sigma2 = max((trace - lam_top.sum()) / (dim - r), floor)
        lam = np.maximum(lam_top, sigma2)
    c_fwd = np.sqrt(sigma2 / lam) - 1.0
    c_inv = np.sqrt(lam / sigma2) - 1.0
    return sigma2, lam, c_fwd, c_inv


def lowrank_factor(A: np.ndarray, r: int, damping: float = 1e-6) -> Factor:
    """Exact rank-r factor of a PSD matrix from its eigendecomposition.

    Pins: spiked covariance closed form; ``S^-1 A_r S^-1 = sigma^2 I``;
    ``r = dim`` gives ``sigma * A^-1/2``; invariance to scaling ``A``.
    """
    A = np.asarray(A, dtype=np.float64)
    dim = A.shape[0]
    r = min(int(r), dim)
    w, v = np.linalg.eigh(0.5 * (A + A.T))
    order = np.argsort(w)[::-1]
    w, v = w[order], v[:, order]
    sigma2, lam, c_fwd, c_inv = coefficients(np.maximum(w[:r], 0.0),
                                             float(np.trace(A)), dim, damping)
    return Factor(v[:, :r].copy(), c_fwd, c_inv, sigma2, lam)


def identity_factor(dim: int) -> Factor:
    return Factor(np.zeros((dim, 0)), np.zeros(0), np.zeros(0), 0.0, np.zeros(0))


# --------------------------------------------------------------------------
# Cholesky-form factors (eq. design_chol; Sec. V-B, Table II: full, diagonal
# and block-diagonal approximations of A)
# --------------------------------------------------------------------------

@dataclass
class CholFactor:
    """One side's Cholesky transform ``A + delta I = L L^T`` (eq. design_chol).

    ``L`` is block-diagonal with ``b x b`` diagonal blocks (``b = dim``: the
    full factor; ``b = 1``: the diagonal of A), each block the Cholesky factor
    of the matching diagonal block of ``A + delta I``.  Stored per block as
    ``R = L_k^T`` (upper triangular) and ``R^-1 = L_k^-T``, ``[nblk, b, b]``;
    the last block, when ``dim`` is not a multiple of ``b``, holds its
    ``kv x kv`` part in the top-left corner and the identity elsewhere.
    """

    R: np.ndarray        # [nblk, b, b]
    Rinv: np.ndarray     # [nblk, b, b]
    dim: int

    @property
    def block(self) -> int:
        return self.R.shape[1]

    @property
    def rank(self) -> int:   # a Cholesky factor is never the identity transform
        return self.dim

    def to_f32(self) -> "CholFactor":
        f = lambda a: np.asarray(a, dtype=np.float32).astype(np.float64)
        return CholFactor(f(self.R), f(self.Rinv), self.dim)

    def _dense(self, blocks: np.ndarray) -> np.ndarray:
        b = self.block
        out = np.zeros((self.dim, self.dim))
        for k in range(blocks.shape[0]):
            kv = min(b, self.dim - k * b)
            out[k * b:k * b + kv, k * b:k * b + kv] = blocks[k, :kv, :kv]
        return out

    def lower(self) -> np.ndarray:
        """Dense ``L`` (dim x dim, lower triangular)."""
        return self._dense(self.R).T

    def right_fwd(self) -> np.ndarray:
        """``L^-T``: the input side's forward map ``W -> W L^-T``."""
        return self._dense(self.Rinv)

    def left_fwd(self) -> np.ndarray:
        """``L^-1``: the output side's forward map ``W -> L^-1 W``."""
        return self._dense(self.Rinv).T

    def right_inv(self) -> np.ndarray:
        """``L^T``: the input side's inverse map ``M -> M L^T``."""
        return self._dense(self.R)

    def left_inv(self) -> np.ndarray:
        """``L``: the output side's inverse map ``M -> L M``."""
        return self._dense(self.R).T


def chol_shift(A: np.ndarray, damping: float) -> float:
    """Regularisation ``delta = damping * tr(A) / dim`` of eq. design_chol."""
    A = np.asarray(A, dtype=np.float64)
    return float(damping * np.trace(A) / A.shape[0])


def chol_factor(A: np.ndarray, block: int = 0, damping: float = 1e-6) -> CholFactor:
    """Block-diagonal Cholesky factor of ``A + delta I`` (eq. design_chol).

    ``block = 0`` or ``>= dim`` is the full factor (Table II's full-A),
    ``1`` the diagonal (diag-A), ``b`` the ``b x b`` diagonal blocks
    (block-A-b).  A zero trace gives the identity.  Each block is factored by
    ``numpy.linalg.cholesky`` and inverted by a triangular solve.
    """
    A = np.asarray(A, dtype=np.float64)
    dim = A.shape[0]
    b = dim if block <= 0 or block >= dim else int(block)
    nblk = -(-dim // b)
    R = np.zeros((nblk, b, b))
    Rinv = np.zeros((nblk, b, b))
    tr = float(np.trace(A))
    delta = chol_shift(A, damping)
    for k in range(nblk):
        kv = min(b, dim - k * b)
        R[k] = np.eye(b)
        Rinv[k] = np.eye(b)
        if tr <= 0.0:
            continue
        blk = A[k * b:k * b + kv, k * b:k * b + kv]
        blk = 0.5 * (blk + blk.T) + delta * np.eye(kv)
        Lk = np.linalg.cholesky(blk)
        R[k, :kv, :kv] = Lk.T
        Rinv[k, :kv, :kv] = scipy.linalg.solve_triangular(Lk.T, np.eye(kv), lower=False)
    return CholFactor(R, Rinv, dim)


def _right_fwd(f):
    return f.right_fwd() if isinstance(f, CholFactor) else f.inverse_root()


def _left_fwd(f):
    return f.left_fwd() if isinstance(f, CholFactor) else f.inverse_root()


def _right_inv(f):
    return f.right_inv() if isinstance(f, CholFactor) else f.root()


def _left_inv(f):
    return f.left_inv() if isinstance(f, CholFactor) else f.root()


# --------------------------------------------------------------------------
# Transform and inverse (eq. design_full_transform / design_input_side_transform,
# eq. design_full_inverse_transform / design_input_side_inverse)
# --------------------------------------------------------------------------

def forward(W: np.ndarray, fA=None, fG=None) -> np.ndarray:
    """``W~ = L_G^-1 W L_A^-T`` in float64 (a missing side is the identity).

    ``W`` is ``[m, n]`` or ``[N, m, n]``.  For a low-rank ``Factor`` both maps
    are the symmetric ``S^-1`` (``L = S``); for a ``CholFactor`` they are the
    triangular ``L^-1`` and ``L^-T`` of eq. design_full_transform.
    """
    W = np.asarray(W, dtype=np.float64)
    out = W
    if fA is not None and fA.rank > 0:
        out = out @ _right_fwd(fA)
    if fG is not None and fG.rank > 0:
        out = _left_fwd(fG) @ out
    return out


def inverse(M: np.ndarray, fA=None, fG=None) -> np.ndarray:
    """``W^ = L_G M L_A^T`` in float64 (eq. design_full_inverse_transform)."""
    M = np.asarray(M, dtype=np.float64)
    out = M
    if fA is not None and fA.rank > 0:
        out = out @ _right_inv(fA)
    if fG is not None and fG.rank > 0:
        out = _left_inv(fG) @ out
    return out


# --------------------------------------------------------------------------
# Scaling and quantization (Algorithm 1: Scale, Q, AllReduce_MAX)
# --------------------------------------------------------------------------

def block_grid(m: int, n: int, block_rows: int, block_cols: int):
    br = m if block_rows <= 0 else min(block_rows, m)
    bc = n if block_cols <= 0 else min(block_cols, n)
    return br, bc, -(-m // br), -(-n // bc)


def block_amax(Wt: np.ndarray, block_rows: int = 0, block_cols: int = 0) -> np.ndarray:
    """``[N, nbr, nbc]`` float32 max of ``|W~|`` per rank and block (NaN wins)."""
    Wt = np.asarray(Wt, dtype=np.float32)
    N, m, n = Wt.shape
    br, bc, nbr, nbc = block_grid(m, n, block_rows, block_cols)
    out = np.zeros((N, nbr, nbc), dtype=np.float32)
    for bi in range(nbr):
        for bj in range(nbc):
            blk = np.abs(Wt[:, bi * br:(bi + 1) * br, bj * bc:(bj + 1) * bc])
            out[:, bi, bj] = blk.reshape(N, -1).max(axis=1)
    return out


def scales_from_amax(amax: np.ndarray):
    """``s = fl32(a / 448)`` and the quantization multiplier ``fl32(448 / a)``."""
    a = np.asarray(amax, dtype=np.float32)
    s = (a / np.float32(e4m3.E4M3_MAX)).astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        inv = (np.float32(e4m3.E4M3_MAX) / a).astype(np.float32)
    inv = np.where(a == 0, np.float32(0.0), inv)
    inv = np.where(np.isposinf(inv), F32_MAX, inv).astype(np.float32)
    return s, inv


def expand_blocks(per_block: np.ndarray, m: int, n: int, block_rows: int, block_cols: int):
    """Broadcast ``[N, nbr, nbc]`` block values to ``[N, m, n]``."""
    br, bc, _, _ = block_grid(m, n, block_rows, block_cols)
    rows = np.arange(m) // br
    cols = np.arange(n) // bc
    return per_block[:, rows[:, None], cols[None, :]]


def quantize_blocks(Wt: np.ndarray, inv: np.ndarray, block_rows: int = 0,
                    block_cols: int = 0) -> np.ndarray:
    """Codes ``Q(fl32(x * inv_block))`` for ``[N, m, n]`` float32 ``W~``."""
    Wt = np.asarray(Wt, dtype=np.float32)
    N, m, n = Wt.shape
    mult = expand_blocks(np.asarray(inv, dtype=np.float32), m, n, block_rows, block_cols)
    with np.errstate(over="ignore", invalid="ignore"):
        y = (Wt * mult).astype(np.float32)
    return e4m3.quantize(y)


def encode(grads: np.ndarray, fA: Factor | None = None, fG: Factor | None = None,
           block_rows: int = 0, block_cols: int = 0, shared: bool = False):
    """Per-rank encode: transform, scale, quantize (Algorithm 1).

    Returns ``(codes [N,m,n] uint8, scales [N,nbr,nbc] float32,
    transformed [N,m,n] float32)``.  ``shared`` takes the maximum of the
    per-rank amax over ranks first (AllReduce_MAX, Algorithm 1), else each rank
    keeps its local scale (the GIFT branch's default, Sec. V-E).
    """
    grads = np.asarray(grads, dtype=np.float32)
    Wt = forward(grads, fA, fG).astype(np.float32)
    return quantize_transformed(Wt, block_rows, block_cols, shared) + (Wt,)


def quantize_transformed(Wt: np.ndarray, block_rows: int = 0, block_cols: int = 0,
                         shared: bool = False):
    """Scale + quantize an already transformed ``[N, m, n]`` float32 tensor."""
    Wt = np.asarray(Wt, dtype=np.float32)
    amax = block_amax(Wt, block_rows, block_cols)
    if shared:
        amax = np.broadcast_to(amax.max(axis=0, keepdims=True), amax.shape).copy()
    s, inv = scales_from_amax(amax)
    codes = quantize_blocks(Wt, inv, block_rows, block_cols)
    return codes, s.astype(np.float32)


def boundary_hits(Wt: np.ndarray, codes: np.ndarray) -> np.ndarray:
    """Per-rank boundary hits of an encode (Sec. V-C's vulnerability profile).

    ``Wt`` is the ``[N, m, n]`` float32 tensor the codes encode (the
    transformed gradient, plus the residual with error feedback), ``codes``
    its ``[N, m, n]`` E4M3 codes.  Returns ``[N, 2]`` int64: column 0 counts
    codes whose value has magnitude 448 (the format's largest finite value),
    column 1 counts nonzero values of ``Wt`` encoded as a zero.
    """
    Wt = np.asarray(Wt, dtype=np.float32)
    val = e4m3.dequantize(np.asarray(codes, dtype=np.uint8))
    N = Wt.shape[0]
    out = np.zeros((N, 2), dtype=np.int64)
    for j in range(N):
        v = val[j]
        out[j, 0] = int(np.count_nonzero(np.abs(v) == 448.0))
        out[j, 1] = int(np.count_nonzero((v == 0.0) & (Wt[j] != 0.0)))
    return out


def dequantize_blocks(codes: np.ndarray, scales: np.ndarray, block_rows: int = 0,
                      block_cols: int = 0) -> np.ndarray:
    """Per-rank ``fl32(val(q) * s_block)`` of ``[N, m, n]`` codes."""
    codes = np.asarray(codes, dtype=np.uint8)
    N, m, n = codes.shape
    sc = expand_blocks(np.asarray(scales, dtype=np.float32), m, n, block_rows, block_cols)
    with np.errstate(over="ignore", invalid="ignore"):
        return (e4m3.dequantize(codes).astype(np.float32) * sc).astype(np.float32)


def encode_ef(grads: np.ndarray, residual: np.ndarray, fA: Factor | None = None,
              fG: Factor | None = None, block_rows: int = 0, block_cols: int = 0,
              shared: bool = False):
    """Encode with error feedback in the transformed coordinates.

    The GIFT branch of the selective-communication algorithm (Sec. V-E):
    ``U = W S^-1``, ``U~ = U + R``, scale and quantize ``U~``, and the new
    residual ``R <- U~ - Dequantize(Q(U~))``, all float32 values
    (``U~ = fl32(U + R)``, ``R = fl32(U~ - fl32(val * s))``).  Returns
    ``(codes, scales, U~, R_new)``.
    """
    grads = np.asarray(grads, dtype=np.float32)
    U = forward(grads, fA, fG).astype(np.float32)
    Ut = (U + np.asarray(residual, dtype=np.float32)).astype(np.float32)
    codes, s = quantize_transformed(Ut, block_rows, block_cols, shared)
    return codes, s, Ut, residual_after(Ut, codes, s, block_rows, block_cols)


def residual_after(Ut: np.ndarray, codes: np.ndarray, scales: np.ndarray, block_rows: int = 0,
                   block_cols: int = 0) -> np.ndarray:
    """Error-feedback residual ``fl32(U~ - fl32(val(q) * s))``."""
    deq = dequantize_blocks(codes, scales, block_rows, block_cols)
    with np.errstate(over="ignore", invalid="ignore"):
        return (np.asarray(Ut, dtype=np.float32) - deq).astype(np.float32)


# --------------------------------------------------------------------------
# Rank sum (eq. dp_grad_avg; Algorithm 1 AllReduce_SUM + Dequantize / N)
# --------------------------------------------------------------------------

def reduce_local(codes: np.ndarray, scales: np.ndarray, block_rows: int = 0,
                 block_cols: int = 0) -> np.ndarray:
    """``M = fl32(acc / N)``, ``acc = fl32(acc + fl32(val(q_j) * s_j))`` in rank order."""
    codes = np.asarray(codes, dtype=np.uint8)
    N, m, n = codes.shape
    sc = expand_blocks(np.asarray(scales, dtype=np.float32), m, n, block_rows, block_cols)
    acc = np.zeros((m, n), dtype=np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        for j in range(N):
            v = e4m3.dequantize(codes[j]).astype(np.float32)
            acc = (acc + (v * sc[j]).astype(np.float32)).astype(np.float32)
        return (acc / np.float32(N)).astype(np.float32)


def decode(mean: np.ndarray, fA: Factor | None = None, fG: Factor | None = None) -> np.ndarray:
    """Inverse transform of the rank mean, cast to float32."""
    return inverse(mean, fA, fG).astype(np.float32)


def round_trip(grads, fA=None, fG=None, block_rows=0, block_cols=0, shared=False):
    """encode -> reduce_local -> decode; returns the decoded float32 ``[m, n]``."""
    codes, s, _ = encode(grads, fA, fG, block_rows, block_cols, shared)
    return decode(reduce_local(codes, s, block_rows, block_cols), fA, fG)


# --------------------------------------------------------------------------
# Reconstruction metrics (eq. recon_metrics)
# --------------------------------------------------------------------------

def fidelity(ghat: np.ndarray, g: np.ndarray) -> dict:
    """RelL2, Cos, MaxErr and MSE of a reconstruction ``ghat`` of ``g``."""
    gh = np.asarray(ghat, dtype=np.float64).ravel()
    g = np.asarray(g, dtype=np.float64).ravel()
    d = gh - g
    return {
        "RelL2": float(np.linalg.norm(d) / np.linalg.norm(g)),
        "Cos": float(gh @ g / (np.linalg.norm(gh) * np.linalg.norm(g))),
        "MaxErr": float(np.max(np.abs(d))),
        "MSE": float(d @ d / d.size),
    }

"""Seeded synthetic inputs for the GIFT gradient codec.

This module only draws random inputs; it holds none of the codec's arithmetic.
Both the CPU oracle (through the tests) and the GPU path (through the tests and
the benchmark) take their inputs from here, so that the two sides see the same
numbers.

Recipe (stands in for the paper's profiled OpenWebText-trained Llama gradients
and activations, which are not available; Sec. VI-A):

* Gradient of one linear layer, ``W_g`` of shape ``d_out x d_in`` (Sec. IV-A):
  ``G_base = U diag(s) V^T`` with Haar-random orthonormal ``U`` (m x k) and
  ``V`` (n x k), ``k = min(m, n)``, power-law singular values ``s_i = i^-1.5``.
  Data-parallel rank ``j`` receives ``G_j = G_base + 0.01 * rms(G_base) * t_j``
  with independent Student-t(3) noise ``t_j`` scaled to unit variance
  (``t / sqrt(3)``).  The whole set is rescaled so that ``rms(G_base)`` is
  2.15e-4, the rms implied by the MSE and RelL2 the paper reports for its
  profiled layer (Table I).  The codec is scale-free (amax scaling), so the
  rescale only makes magnitudes realistic.
* Kronecker-factor inputs (Sec. II-B, eq. kfac_fisher_block): layer input
  activations ``X`` (T x d_in) and output gradients ``Delta`` (T x d_out) are
  ``Z diag(i^-0.6) Q^T`` with standard normal ``Z`` and Haar ``Q``, so that
  their covariance has the power-law spectrum ``i^-1.2``.  For bf16 workloads
  the values are rounded to bfloat16 (round to nearest even) and both sides use
  the rounded values.
* Seeds: numpy PCG64 with ``seed = 1000*cfg + {0: base, 1: X, 2: Delta,
  100+j: noise of rank j}``, plus ``10000*layer + 100*matrix_kind`` for the
  multi-layer gradient sets.

Large gradient sets (the Llama-shaped sets) would take minutes to draw with
numpy on a few host cores, so :func:`gradient_set_torch` and
:func:`factor_inputs_torch` draw the same recipe with a seeded torch generator
on the device that holds the data.  Their streams differ from numpy's; tests
that compare against the oracle copy those device inputs to the host.
"""

from __future__ import annotations

import numpy as np

PAPER_GRAD_RMS = 2.15e-4

__all__ = [
    "PAPER_GRAD_RMS",
    "seed_for",
    "haar",
    "gradient_set",
    "factor_inputs",
    "bf16_round",
    "bf16_bits",
    "gradient_set_torch",
    "factor_inputs_torch",
]


def seed_for(cfg: int, role: int, layer: int = 0, kind: int = 0) -> int:
    """Seed layout: 1000*cfg + role (+ 10000*layer + 100*kind for layer sets)."""
    return 1000 * cfg + role + 10000 * layer + 100 * kind


def haar(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    """Haar-distributed orthonormal columns: QR of a Gaussian with sign fix."""
    z = rng.standard_normal((rows, cols))
    q, r = np.linalg.qr(z)
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return q * d


def gradient_set(seed_base: int, noise_seed: int, N: int, m: int, n: int,
                 decay: float = 1.5, noise: float = 0.01,
                 target_rms: float = PAPER_GRAD_RMS) -> np.ndarray:
    """``[N, m, n]`` float32 rank gradients (row-major per rank).

    ``seed_base`` seeds the shared low-rank-plus-power-law base; rank ``j``'s
    noise uses ``noise_seed + j``.
    """
    rng = np.random.Generator(np.random.PCG64(seed_base))
    k = min(m, n)
    u = haar(rng, m, k)
    v = haar(rng, n, k)
    s = np.arange(1, k + 1, dtype=np.float64) ** (-decay)
    base = (u * s) @ v.T
    rms = float(np.sqrt(np.mean(base * base)))
    out = np.empty((N, m, n), dtype=np.float32)
    for j in range(N):
        nrng = np.random.Generator(np.random.PCG64(noise_seed + j))
        t = nrng.standard_t(3.0, size=(m, n)) / np.sqrt(3.0)
        g = base + noise * rms * t
        out[j] = (g * (target_rms / rms)).astype(np.float32)
    return out


def layer_gradients(seed: int, N: int, T: int, m: int, n: int, decay: float = 1.2,
                    spike_frac: float = 0.0, spike: float = 1.0,
                    target_rms: float = PAPER_GRAD_RMS):
    """Weight gradients of one linear layer together with the inputs behind them.

    Rank ``j`` sees ``T`` tokens: layer inputs ``X_j`` ``[T, n]`` and output
    gradients ``D_j`` ``[T, m]``, each row drawn with covariance spectrum
    ``i^-decay`` in a Haar basis shared by all ranks (the law of
    :func:`factor_inputs`), and its weight gradient is ``D_j^T X_j / T``.  A
    fraction ``spike_frac`` of every rank's tokens has both rows multiplied by
    ``spike`` (tokens with large activations and gradients), which plants a
    few large rank-one terms in the gradient.  All gradients are rescaled by
    one common factor to rms ``target_rms`` over the ranks.

    Returns ``(grads [N, m, n] float32, acts [N*T, n] float32,
    out_grads [N*T, m] float32)``; ``acts`` / ``out_grads`` stack the ranks'
    tokens in rank order.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    qa = haar(rng, n, n)
    qg = haar(rng, m, m)
    sda = np.arange(1, n + 1, dtype=np.float64) ** (-decay / 2.0)
    sdg = np.arange(1, m + 1, dtype=np.float64) ** (-decay / 2.0)
    acts = np.empty((N * T, n), dtype=np.float32)
    outg = np.empty((N * T, m), dtype=np.float32)
    grads = np.empty((N, m, n), dtype=np.float64)
    for j in range(N):
        X = (rng.standard_normal((T, n)) * sda) @ qa.T
        D = (rng.standard_normal((T, m)) * sdg) @ qg.T
        if spike_frac > 0.0:
            k = max(1, int(round(T * spike_frac)))
            idx = rng.choice(T, k, replace=False)
            X[idx] *= spike
            D[idx] *= spike
        X = X.astype(np.float32)
        D = D.astype(np.float32)
        acts[j * T:(j + 1) * T] = X
        outg[j * T:(j + 1) * T] = D
        grads[j] = D.astype(np.float64).T @ X.astype(np.float64) / T
    rms = float(np.sqrt(np.mean(grads * grads)))
    return (grads * (target_rms / rms)).astype(np.float32), acts, outg


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); float32 out."""
    b = bf16_bits(x)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of float32 values, round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    rounded = np.where(nan, (u >> 16) | 0x40, rounded)
    return rounded.astype(np.uint16)


def factor_inputs(seed: int, T: int, dim: int, decay: float = 1.2,
                  dtype: str = "f32"):
    """``[T, dim]`` samples with covariance spectrum ``i^-decay``.

    Returns ``(values_f32, bits)``: ``bits`` is the uint16 bfloat16 pattern
    array when ``dtype == "bf16"`` (and ``values_f32`` holds exactly those
    rounded values), else ``None``.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    q = haar(rng, dim, dim)
    z = rng.standard_normal((T, dim))
    sd = np.arange(1, dim + 1, dtype=np.float64) ** (-decay / 2.0)
    x = ((z * sd) @ q.T).astype(np.float32)
    if dtype == "bf16":
        bits = bf16_bits(x)
        return (bits.astype(np.uint32) << 16).view(np.float32), bits
    if dtype != "f32":
        raise ValueError(f"dtype must be 'f32' or 'bf16', not {dtype!r}")
    return x, None


def _torch_haar(torch, gen, rows, cols, device):
    # The Gaussian block is drawn on the device; its QR runs on the host in
    # float64 (numpy), which keeps the GPU solver library out of the process.
    z = torch.randn(rows, cols, generator=gen, device=device, dtype=torch.float32)
    q, r = np.linalg.qr(z.cpu().numpy().astype(np.float64))
    d = np.sign(np.diagonal(r))
    d[d == 0] = 1.0
    return torch.from_numpy((q * d).astype(np.float32)).to(device)


def gradient_set_torch(seed: int, N: int, m: int, n: int, device,
                       decay: float = 1.5, noise: float = 0.01,
                       target_rms: float = PAPER_GRAD_RMS):
    """Same recipe as :func:`gradient_set`, drawn with torch on ``device``."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    k = min(m, n)
    u = _torch_haar(torch, gen, m, k, device)
    v = _torch_haar(torch, gen, n, k, device)
    s = torch.arange(1, k + 1, device=device, dtype=torch.float32) ** (-decay)
    base = (u * s) @ v.T
    rms = torch.sqrt(torch.mean(base * base))
    out = torch.empty((N, m, n), device=device, dtype=torch.float32)
    for j in range(N):
        z = torch.randn(m, n, generator=gen, device=device)
        # Student-t(3) = Z / sqrt(chi2_3 / 3); chi2_3 = 2 * Gamma(1.5).
        chi2 = 2.0 * torch._standard_gamma(torch.full((m, n), 1.5, device=device),
                                           generator=gen)
        t = z / torch.sqrt(chi2 / 3.0) / (3.0 ** 0.5)
        out[j] = (base + noise * rms * t) * (target_rms / rms)
    return out


def factor_inputs_torch(seed: int, T: int, dim: int, device, decay: float = 1.2,
                        dtype: str = "bf16"):
    """Same recipe as :func:`factor_inputs`, drawn with torch on ``device``.

    Returns a ``[T, dim]`` tensor in float32 or bfloat16.
    """
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    q = _torch_haar(torch, gen, dim, dim, device)
    sd = torch.arange(1, dim + 1, device=device, dtype=torch.float32) ** (-decay / 2.0)
    x = torch.empty((T, dim), device=device, dtype=torch.float32)
    step = 4096
    for t0 in range(0, T, step):
        t1 = min(T, t0 + step)
        z = torch.randn(t1 - t0, dim, generator=gen, device=device)
        x[t0:t1] = (z * sd) @ q.T
    if dtype == "bf16":
        return x.to(torch.bfloat16)
    return x

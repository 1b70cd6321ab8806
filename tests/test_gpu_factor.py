"""GPU factor refresh against the oracle (runs on an MI355X).

The GPU runs the iterative rank-r factor (subspace iteration, CholeskyQR2,
Rayleigh-Ritz) on float32 statistics; the oracle mirrors the same algorithm
in float64 (``oracle.subspace``) and also gives the exact eigendecomposition
(``oracle.codec.lowrank_factor``).  Agreement is measured on what the codec
uses: the eigenvalues, sigma^2, and the action of S^-1 on a test matrix.
"""

import numpy as np
import pytest
import torch

from oracle import codec, subspace
from synth import bf16_round, factor_inputs, haar

pytestmark = pytest.mark.gpu

gift = pytest.importorskip("paper_2607_07494_amd.gift")
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gift.Context()
    yield c
    torch.cuda.synchronize()
    c.close()


def t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def exported(f, side):
    U, cf, ci, s2 = f.export(side)
    torch.cuda.synchronize()
    return codec.Factor(U.cpu().numpy().astype(np.float64), cf.cpu().numpy().astype(np.float64),
                        ci.cpu().numpy().astype(np.float64), float(s2.cpu().numpy()[0]))


def action_gap(fa, fb, dim, seed=0):
    """Relative difference of W S^-1 for two factors on a Gaussian W."""
    W = np.random.default_rng(seed).standard_normal((64, dim))
    a = codec.forward(W, fa)
    b = codec.forward(W, fb)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b - W + 1e-300))


def test_spiked_statistics_recover_exact_factor(ctx):
    say("spiked factor")
    T, n, r = 2048, 128, 6
    rng = np.random.default_rng(1)
    spec = np.full(n, 0.02)
    spec[:r] = [9.0, 6.0, 4.0, 3.0, 2.0, 1.5]
    q = haar(rng, n, n)
    Z = haar(rng, T, n) * np.sqrt(T)
    X = ((Z * np.sqrt(spec)) @ q.T).astype(np.float32)
    f = gift.Factor(ctx, 32, n, r, gift.SIDE_INPUT, seed=3)
    f.update(acts=t(X), iters=6)
    got = exported(f, gift.SIDE_INPUT)
    exact = codec.lowrank_factor(codec.factor_statistics(X), r)
    np.testing.assert_allclose(1 + got.c_fwd, 1 + exact.c_fwd, rtol=1e-4)
    assert got.sigma2 == pytest.approx(exact.sigma2, rel=1e-4)
    assert action_gap(got, exact, n) <= 1e-4
    np.testing.assert_allclose(got.U.T @ got.U, np.eye(r), atol=1e-5)
    f.close()


@pytest.mark.parametrize("T,n,r,iters,dtype", [(1024, 256, 16, 6, "f32"),
                                                (4096, 512, 32, 4, "bf16"),
                                                (2048, 200, 20, 3, "f32"),
                                                # k = 2r = 160 > 128: the global-memory k x k kernels
                                                (2048, 320, 80, 6, "f32")])
def test_matches_float64_mirror(ctx, T, n, r, iters, dtype):
    say(f"factor mirror T={T} n={n} r={r} iters={iters} {dtype}")
    X, bits = factor_inputs(40 + n, T, n, dtype=dtype)
    seed = 1234 + n
    f = gift.Factor(ctx, 16, n, r, gift.SIDE_INPUT, seed=seed)
    if dtype == "bf16":
        xt = t(bits.view(np.int16)).view(torch.bfloat16)
    else:
        xt = t(X)
    f.update(acts=xt, iters=iters)
    got = exported(f, gift.SIDE_INPUT)
    A = codec.factor_statistics(X)
    mirror, _ = subspace.subspace_factor(A, r, iters, seed=seed)
    np.testing.assert_allclose(1 + got.c_fwd, 1 + mirror.c_fwd, rtol=1e-3)
    assert got.sigma2 == pytest.approx(mirror.sigma2, rel=1e-4)
    assert action_gap(got, mirror, n) <= 1e-3
    # quality against the exact top-r space: captured energy
    w = np.sort(np.linalg.eigvalsh(A))[::-1]
    assert np.trace(got.U.T @ A @ got.U) / w[:r].sum() >= 0.999
    f.close()


def test_both_sides_and_warm_start(ctx):
    say("both sides + warm start")
    T, m, n, r = 2048, 96, 160, 8
    X, _ = factor_inputs(70, T, n)
    D, _ = factor_inputs(71, T, m)
    f = gift.Factor(ctx, m, n, r, gift.SIDE_BOTH, seed=77)
    f.update(acts=t(X), out_grads=t(D), iters=6)
    gA, gG = exported(f, gift.SIDE_INPUT), exported(f, gift.SIDE_OUTPUT)
    mA, _ = subspace.subspace_factor(codec.factor_statistics(X), r, 6, seed=77)
    mG, _ = subspace.subspace_factor(codec.factor_statistics(D), r, 6, seed=78)
    assert action_gap(gA, mA, n) <= 1e-3
    assert action_gap(gG, mG, m) <= 1e-3
    # a second refresh on the same statistics, warm-started, stays put
    f.update(acts=t(X), out_grads=t(D), iters=1)
    assert action_gap(exported(f, gift.SIDE_INPUT), gA, n) <= 2e-2
    f.close()


def test_export_import_round_trip_and_errors(ctx):
    say("export/import")
    f = gift.Factor(ctx, 40, 50, 4, gift.SIDE_INPUT)
    X, _ = factor_inputs(90, 512, 50)
    f.update(acts=t(X), iters=3)
    U, cf, ci, s2 = f.export(gift.SIDE_INPUT)
    g = gift.Factor(ctx, 40, 50, 4, gift.SIDE_INPUT)
    g.import_(gift.SIDE_INPUT, U, cf, ci, s2)
    a, b = exported(f, gift.SIDE_INPUT), exported(g, gift.SIDE_INPUT)
    np.testing.assert_array_equal(a.U, b.U)
    np.testing.assert_array_equal(a.c_fwd, b.c_fwd)
    with pytest.raises(gift.GiftError):
        f.export(gift.SIDE_OUTPUT)
    f.close()
    g.close()


def test_batch_equals_single_updates(ctx):
    say("batch refresh == single refreshes")
    T = 1024
    shapes = [(64, 96, 8, gift.SIDE_INPUT), (96, 64, 8, gift.SIDE_BOTH), (48, 96, 8, gift.SIDE_OUTPUT),
              (96, 96, 4, gift.SIDE_INPUT)]
    xs = {d: t(bf16_round(factor_inputs(300 + d, T, d)[0])).to(torch.bfloat16) for d in (48, 64, 96)}
    batch, single = [], []
    for i, (m, n, r, sides) in enumerate(shapes):
        batch.append(gift.Factor(ctx, m, n, r, sides, seed=10 + i))
        single.append(gift.Factor(ctx, m, n, r, sides, seed=10 + i))
    acts = [xs[n] if s & gift.SIDE_INPUT else None for (m, n, r, s) in shapes]
    dgr = [xs[m] if s & gift.SIDE_OUTPUT else None for (m, n, r, s) in shapes]
    for rep in range(2):   # cold, then warm
        gift.factor_update_batch(ctx, batch, acts, dgr, iters=3)
        for f, a, d in zip(single, acts, dgr):
            f.update(acts=a, out_grads=d, iters=3)
        torch.cuda.synchronize()
        for (m, n, r, s), fb, fs in zip(shapes, batch, single):
            for side in (gift.SIDE_INPUT, gift.SIDE_OUTPUT):
                if s & side:
                    a, b = exported(fb, side), exported(fs, side)
                    np.testing.assert_array_equal(a.U, b.U)
                    np.testing.assert_array_equal(a.c_fwd, b.c_fwd)
    for f in batch + single:
        f.close()

"""GPU parity at the size limits (checked on sampled rows, like the full-size
tests): the largest row count the launch grids allow (m = 1048560 = 65535 x 16)
on the Euclidean and the transform paths, and a transform encode whose
per-rank matrix has 2^29 elements or more, which leaves the split-bf16
kernels (32-bit buffer ranges) for the path that stores W~ and quantizes it
in a second pass.  Bars as in the other parity tests: scales from the whole
W~ and codes / rank sum on sampled rows bit-exact, W~ and the decode within
1e-5 of float64."""

import numpy as np
import pytest
import torch

from oracle import codec
from synth import factor_inputs, gradient_set_torch

pytestmark = pytest.mark.gpu

gift = pytest.importorskip("paper_2607_07494_amd.gift")

DEV = "cuda"
MAX_ROWS = 65535 * 16


def say(*a):
    print(*a, flush=True)


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gift.Context()
    yield c
    torch.cuda.synchronize()
    c.close()


def rows_of(m, seed, count=40):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, m - 1], rng.choice(m, count - 2, replace=False)]))


def encode_all(ctx, f, g, bc, mode):
    N, m, n = g.shape
    nbr, nbc = gift.scale_grid(m, n, 0, bc)
    codes = torch.empty((N, m, n), dtype=torch.uint8, device=DEV)
    scales = torch.empty((N, nbr, nbc), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes, scales, 0, bc, mode)
    codes2, scales2 = torch.empty_like(codes), torch.empty_like(scales)
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes2, scales2, 0, bc, mode, transformed=tr)
    torch.cuda.synchronize()
    assert torch.equal(codes, codes2) and torch.equal(scales, scales2)
    del codes2, scales2
    mean = torch.empty((m, n), dtype=torch.float32, device=DEV)
    gift.reduce_local(ctx, codes, scales, mean, 0, bc)
    out = None
    if f is not None:
        out = torch.empty((m, n), dtype=torch.float32, device=DEV)
        gift.decode(ctx, f, mean, out)
    torch.cuda.synchronize()
    return codes, scales, tr, mean, out


def check(codes, scales, tr, mean, rows, bc, shared):
    trh = tr.cpu().numpy()
    amax = codec.block_amax(trh, 0, bc)
    if shared:
        amax = np.broadcast_to(amax.max(axis=0, keepdims=True), amax.shape).copy()
    s_ref, inv = codec.scales_from_amax(amax)
    sc = scales.cpu().numpy()
    np.testing.assert_array_equal(sc, s_ref)
    idx = torch.from_numpy(rows).to(DEV)
    got = codes[:, idx, :].cpu().numpy()
    np.testing.assert_array_equal(got, codec.quantize_blocks(trh[:, rows, :], inv, 0, bc))
    got_mean = mean[idx].cpu().numpy()
    np.testing.assert_array_equal(got_mean, codec.reduce_local(got, sc, 0, bc))
    return trh[:, rows, :], got_mean


def lowrank(ctx, m, n, r, seed):
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(seed, 4 * n, n)[0]), r).to_f32()
    f = gift.Factor(ctx, m, n, r, gift.SIDE_INPUT)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x.astype(np.float32))).to(DEV)
    f.import_(gift.SIDE_INPUT, t(fA.U), t(fA.c_fwd), t(fA.c_inv), t(np.array([fA.sigma2])))
    return f, fA


def test_max_rows_euclidean(ctx):
    N, m, n, bc = 2, MAX_ROWS, 24, 8
    say(f"max rows Euclidean N={N} m={m} n={n} block=(0,{bc})")
    g = gradient_set_torch(71, N, m, n, DEV)
    codes, scales, tr, mean, _ = encode_all(ctx, None, g, bc, gift.SCALE_SHARED)
    assert torch.equal(tr, g)
    check(codes, scales, tr, mean, rows_of(m, 1), bc, True)


@pytest.mark.parametrize("m,n,r", [
    (MAX_ROWS, 64, 16),      # the largest row count on the split-bf16 kernels
    (524800, 1024, 16),      # m n >= 2^29: W~ stored, then quantized
])
def test_large_transform(ctx, m, n, r):
    say(f"large transform N=1 m={m} n={n} r={r} (m n = {m * n}, 2^29 = {1 << 29})")
    g = gradient_set_torch(72 + n, 1, m, n, DEV)
    f, fA = lowrank(ctx, m, n, r, seed=n)
    codes, scales, tr, mean, out = encode_all(ctx, f, g, 0, gift.SCALE_LOCAL)
    rows = rows_of(m, 2)
    tr_rows, got_mean = check(codes, scales, tr, mean, rows, 0, False)
    idx = torch.from_numpy(rows).to(DEV)
    assert rel(tr_rows, codec.forward(g[:, idx, :].cpu().numpy(), fA)) <= 1e-5
    assert rel(out[idx].cpu().numpy(), codec.inverse(got_mean, fA)) <= 1e-5
    f.close()

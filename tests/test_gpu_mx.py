"""GPU parity of the MXFP4 variant (OCP MX v1.0 FP4, gift_encode_mxfp4 /
gift_reduce_local_mxfp4) against the MXFP4 oracle.

Bars: codes (packed) and E8M0 scales bit-exact with the oracle's MXFP4
quantization of the tensor the encode reports it quantized (U = W~ + R), the
residual and the rank sum bit-exact, W~ within 1e-5 of the float64 oracle
transform with the same factor, the decode within 1e-5 of the oracle's
inverse of the GPU's rank mean.  Special values: zero blocks, signed zeros,
subnormal-only blocks, NaN / infinity blocks, every rounding midpoint +- 1 ulp.
"""

import numpy as np
import pytest
import torch

from oracle import codec, mx
from synth import factor_inputs, gradient_set

pytestmark = pytest.mark.gpu

gift = pytest.importorskip("paper_2607_07494_amd.gift")

DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.fixture(scope="module")
def ctx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    c = gift.Context()
    yield c
    torch.cuda.synchronize()
    c.close()


def gpu_mx(ctx, f, grads, ef=None):
    N, m, n = grads.shape
    codes = torch.empty((N, m, n // 2), dtype=torch.uint8, device=DEV)
    scales = torch.empty((N, m, n // 32), dtype=torch.uint8, device=DEV)
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    gift.encode_mxfp4(ctx, f, t(grads), codes, scales, ef=ef, transformed=tr)
    mean = torch.empty((m, n), dtype=torch.float32, device=DEV)
    gift.reduce_local_mxfp4(ctx, codes, scales, mean)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy(), tr.cpu().numpy(), mean


def check_codes(codes, scales, tr):
    ref_codes, ref_scales = mx.quantize(tr)
    np.testing.assert_array_equal(scales, ref_scales)
    np.testing.assert_array_equal(codes, mx.pack(ref_codes))


@pytest.mark.parametrize("N,m,n", [(1, 1, 32), (3, 7, 96), (8, 130, 256), (2, 33, 1024)])
def test_euclidean_mxfp4_bit_exact(ctx, N, m, n):
    say(f"mxfp4 Euclidean N={N} m={m} n={n}")
    grads = gradient_set(300 + m, 301 + n, N, m, n)
    grads *= np.exp(np.random.default_rng(m).uniform(-30, 30, (N, m, 1))).astype(np.float32)
    codes, scales, tr, mean = gpu_mx(ctx, None, grads)
    np.testing.assert_array_equal(tr, grads)
    check_codes(codes, scales, tr)
    np.testing.assert_array_equal(mean.cpu().numpy(), mx.reduce_local(mx.unpack(codes), scales))


def test_special_values_and_midpoints(ctx):
    say("mxfp4 special values and rounding midpoints")
    n = 32 * 12
    x = np.zeros((2, 4, n), np.float32)
    # blocks with amax 6 (scale 2^0): every midpoint of the E2M1 grid and its
    # float32 neighbours, both signs
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    vals = np.concatenate([mids, np.nextafter(mids, 0), np.nextafter(mids, 10)])
    for r in range(2):
        blk = np.zeros(32, np.float32)
        blk[0] = 6.0
        blk[1:1 + len(vals)] = vals * (1 if r == 0 else -1)
        x[0, r, :32] = blk
    x[0, 2, 32:64] = 0.0                                   # zero block
    x[0, 2, 64:96] = -0.0                                  # negative zeros
    x[0, 3, 96:128] = np.float32(1e-42)                    # subnormal block
    x[0, 3, 130] = np.nan                                  # NaN block
    x[1, 0, 200] = np.inf                                  # infinity block
    x[1, 1, 256:288] = np.linspace(-7.9, 7.9, 32, dtype=np.float32)  # saturation in (6, 8)
    x[1, 2, 288:320] = np.float32(3.4e38)                  # near the float32 maximum
    codes, scales, tr, mean = gpu_mx(ctx, None, x)
    check_codes(codes, scales, tr)
    got = mean.cpu().numpy()
    want = mx.reduce_local(mx.unpack(codes), scales)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(want))
    np.testing.assert_array_equal(got[~np.isnan(got)], want[~np.isnan(want)])


def lowrank(ctx, m, n, r, seed):
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(seed, 4 * n, n)[0]), r).to_f32()
    f = gift.Factor(ctx, m, n, r, gift.SIDE_INPUT)
    f.import_(gift.SIDE_INPUT, t(fA.U.astype(np.float32)), t(fA.c_fwd.astype(np.float32)),
              t(fA.c_inv.astype(np.float32)), t(np.array([fA.sigma2], np.float32)))
    return f, fA


def chol(ctx, m, n, block, seed):
    fA = codec.chol_factor(codec.factor_statistics(factor_inputs(seed, 4 * n, n)[0]), block, 1e-4).to_f32()
    f = gift.CholFactor(ctx, m, n, block, gift.SIDE_INPUT, 1e-4)
    f.import_(gift.SIDE_INPUT, t(fA.R.astype(np.float32)), t(fA.Rinv.astype(np.float32)))
    return f, fA


@pytest.mark.parametrize("kind,N,m,n,r", [
    ("lowrank", 4, 200, 512, 64),    # MXFP4 inside the split-bf16 update pass, ragged rows
    ("lowrank", 2, 96, 256, 16),
    ("lowrank", 2, 70, 160, 32),     # last 64-column tile half past n
    ("lowrank", 2, 64, 128, 6),      # rank not a multiple of 4: W~ stored, then quantized
    ("chol", 2, 64, 256, 32), ("chol", 3, 48, 128, 0)])
def test_transform_mxfp4_round_trip(ctx, kind, N, m, n, r):
    say(f"mxfp4 {kind} N={N} m={m} n={n} r/block={r}")
    grads = gradient_set(400 + m, 401 + n, N, m, n)
    f, fA = lowrank(ctx, m, n, r, seed=m) if kind == "lowrank" else chol(ctx, m, n, r, seed=m)
    codes, scales, tr, mean = gpu_mx(ctx, f, grads)
    assert rel(tr, codec.forward(grads, fA)) <= 1e-5
    check_codes(codes, scales, tr)
    mh = mean.cpu().numpy()
    np.testing.assert_array_equal(mh, mx.reduce_local(mx.unpack(codes), scales))
    out = torch.empty_like(mean)
    gift.decode(ctx, f, mean, out)
    torch.cuda.synchronize()
    assert rel(out.cpu().numpy(), codec.inverse(mh, fA)) <= 1e-5
    f.close()


def test_error_feedback_two_steps(ctx):
    N, m, n = 3, 64, 256
    say(f"mxfp4 error feedback N={N} m={m} n={n}")
    f, fA = lowrank(ctx, m, n, 32, seed=7)
    R = torch.zeros((N, m, n), dtype=torch.float32, device=DEV)
    prev = np.zeros((N, m, n), np.float32)
    for step in range(2):
        grads = gradient_set(500 + step, 501 + step, N, m, n)
        codes, scales, tr, _ = gpu_mx(ctx, f, grads, ef=R)
        U = codec.forward(grads, fA).astype(np.float32)
        assert rel(tr, (U + prev).astype(np.float64)) <= 1e-5
        check_codes(codes, scales, tr)
        prev = R.cpu().numpy()
        np.testing.assert_array_equal(prev, mx.residual(tr, mx.unpack(codes), scales))
    f.close()

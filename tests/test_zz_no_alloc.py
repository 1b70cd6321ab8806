"""gift_encode_noalloc against gift_encode (runs on an MI355X).

The allocation-free encode takes its scratch from the library's fixed
per-device array instead of the context's grow-only buffers; everything else
(kernels, arguments, results) is gift_encode's.  Each case makes two calls in
a row through the C ABI, the second on a smaller input (fewer ranks and a
smaller matrix), so the second call runs on an array that still holds the
first call's block maxima and projections: codes, scales, residuals and the
stored W~ must equal gift_encode's bit for bit.  A call that needs more than
the array returns GIFT_ESHAPE and leaves its outputs untouched.
"""

import numpy as np
import pytest
import torch

from oracle import codec
from synth import factor_inputs, gradient_set

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


def lowrank(ctx, m, n, r, sides, seed):
    f = gift.Factor(ctx, m, n, r, sides)
    if sides & gift.SIDE_INPUT:
        fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(seed + 1, 4 * n, n)[0]), r).to_f32()
        f.import_(gift.SIDE_INPUT, t(fA.U.astype(np.float32)), t(fA.c_fwd.astype(np.float32)),
                  t(fA.c_inv.astype(np.float32)), t(np.array([fA.sigma2], np.float32)))
    if sides & gift.SIDE_OUTPUT:
        fG = codec.lowrank_factor(codec.factor_statistics(factor_inputs(seed + 2, 4 * m, m)[0]), r).to_f32()
        f.import_(gift.SIDE_OUTPUT, t(fG.U.astype(np.float32)), t(fG.c_fwd.astype(np.float32)),
                  t(fG.c_inv.astype(np.float32)), t(np.array([fG.sigma2], np.float32)))
    return f


def make_factor(ctx, kind, m, n, seed):
    if kind is None:
        return None
    if kind[0] == "chol":
        f = gift.CholFactor(ctx, m, n, kind[1], gift.SIDE_INPUT, 1e-4)
        x = factor_inputs(seed + 3, 4 * n, n)[0]
        f.update(acts=t(x), iters=0)
        return f
    return lowrank(ctx, m, n, kind[1], kind[2], seed)


def encode_both_ways(ctx, f, N, m, n, br, bc, shared, use_ef, want_t, seed):
    grads = gradient_set(seed, seed + 1, N, m, n)
    if shared:
        grads[min(1, N - 1)] *= 3.0
    g = t(grads)
    nbr, nbc = gift.scale_grid(m, n, br, bc)
    mode = gift.SCALE_SHARED if shared else gift.SCALE_LOCAL
    R0 = gradient_set(seed + 2, seed + 3, N, m, n) * np.float32(0.01) if use_ef else None
    outs = []
    for enc in (gift.encode, gift.encode_noalloc):
        codes = torch.full((N, m, n), 0xAB, dtype=torch.uint8, device=DEV)
        scales = torch.full((N, nbr, nbc), -1.0, dtype=torch.float32, device=DEV)
        ef = t(R0) if use_ef else None
        tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV) if want_t else None
        enc(ctx, f, g, codes, scales, br, bc, mode, ef=ef, transformed=tr)
        torch.cuda.synchronize()
        outs.append((codes, scales, ef, tr))
    (ca, sa, ea, ta), (cb, sb, eb, tb) = outs
    assert torch.equal(sa, sb)
    assert torch.equal(ca, cb)
    if use_ef:
        assert torch.equal(ea, eb)
    if want_t:
        assert torch.equal(ta, tb)
    # and the quantization itself against the oracle, on the regular path's W~
    if want_t:
        ref_codes, ref_scales = codec.quantize_transformed(ta.cpu().numpy(), br, bc, shared)
        np.testing.assert_array_equal(sb.cpu().numpy(), ref_scales)
        np.testing.assert_array_equal(cb.cpu().numpy(), ref_codes)


# (factor kind, sides) -> two calls: (N, m, n, block_rows, block_cols) large then small
CASES = [
    ("euclidean shared", None, [(4, 300, 520, 0, 128), (2, 100, 256, 0, 64)], True, False),
    ("euclidean ragged blocks", None, [(3, 77, 131, 7, 50), (1, 33, 40, 5, 0)], False, True),
    ("input r=64, recomputed", ("lr", 64, gift.SIDE_INPUT), [(8, 320, 384, 0, 128), (4, 160, 256, 0, 128)],
     False, True),
    ("input r=128, recomputed", ("lr", 128, gift.SIDE_INPUT), [(4, 256, 512, 0, 0), (2, 136, 256, 0, 0)],
     False, False),
    ("both r=32", ("lr", 32, gift.SIDE_BOTH), [(3, 260, 520, 0, 0), (2, 96, 128, 0, 32)], True, True),
    ("input r=6, stored W~", ("lr", 6, gift.SIDE_INPUT), [(2, 96, 128, 0, 32), (1, 40, 64, 0, 0)],
     False, True),
    ("cholesky block 32", ("chol", 32), [(2, 120, 96, 0, 0), (1, 64, 64, 0, 32)], False, False),
]


@pytest.mark.parametrize("label,kind,calls,shared,use_ef", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_encode_twice(ctx, label, kind, calls, shared, use_ef):
    for i, (N, m, n, br, bc) in enumerate(calls):
        for want_t in (False, True):
            say(f"noalloc {label}: call {i} N={N} m={m} n={n} block=({br},{bc}) shared={shared} "
                f"ef={use_ef} transformed={want_t}")
            f = make_factor(ctx, kind, m, n, seed=17 * m + n)
            encode_both_ways(ctx, f, N, m, n, br, bc, shared, use_ef, want_t, seed=31 * i + m)
            if f is not None:
                f.close()


def test_noalloc_rejects_oversized_scratch(ctx):
    # 1 x 1 scale blocks: 64 sub-slots per element and rank, 4 x 300 x 256 x
    # 64 x 4 bytes > 64 MiB
    N, m, n = 4, 300, 256
    say(f"noalloc rejection N={N} m={m} n={n} block=(1,1)")
    g = t(gradient_set(5, 6, N, m, n))
    codes = torch.full((N, m, n), 0xAB, dtype=torch.uint8, device=DEV)
    scales = torch.full((N, m, n), -1.0, dtype=torch.float32, device=DEV)
    with pytest.raises(gift.GiftError, match="scratch"):
        gift.encode_noalloc(ctx, None, g, codes, scales, 1, 1)
    torch.cuda.synchronize()
    assert torch.all(codes == 0xAB) and torch.all(scales == -1.0)
    # the same encode through gift_encode works
    gift.encode(ctx, None, g, codes, scales, 1, 1)
    torch.cuda.synchronize()
    assert torch.all(scales >= 0)

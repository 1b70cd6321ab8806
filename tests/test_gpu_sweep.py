"""The encode's sweep kernels against the per-unit update kernel and the oracle
(runs on an MI355X).

The input-side encode with no stored W~, no residual, per-rank scales and no
boundary-hit counts takes the sweep variant of its two passes (rank 64, 96
or 128, N a multiple of 128, every 32 x 64 wave tile inside one scale block):
a workgroup walks a run of 1-4 consecutive 128 x 128 units, copying the
column operand's pre-split image into LDS.  The same encode asked to store W~
takes the per-unit kernel.  Both form the same products in the same order
(eq. design_input_side_transform), so codes and scales must agree bit for
bit; W~ is held to 1e-5 of the float64 transform and its codes to the
oracle's quantization (Algorithm 1, Scale / Q; Sec. I, amax rule).

The two-sided encode at equal ranks takes the two-segment sweep (the rank-2r
update (U_G C_G) Q + L_2 U_A^T of eq. design_full_transform, segment 0's
column operand Q per rank, segment 1's U_A^T shared).  At rank 64 it forms
W~ in both passes (the same checks as above); at rank 96 and 128 its AMAX
pass stores W~ and the quantize pass streams it, whatever the caller asks,
so there the reference kernels are those of the error-feedback encode with a
zero residual (per-unit, W~ + R formed in both passes): codes and scales
bit-identical.

The cases choose the run length (units of the launch: 1 below 1024, then
units / 512, 4 from 2048 on) and make runs cross row blocks (an odd number
of 128-column units per row), ranks (units per rank not a multiple of the
run) and the end of the grid (a partial last run); ragged M leaves rows and
whole waves of the last row block empty; block geometries cover per-tensor,
column slabs of 64, 128 and 256, and block rows of 32 and 64.
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


def t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def run_length(N, m, n):
    units = N * ((m + 127) // 128) * (n // 128)
    return 4 if units >= 2048 else max(1, units // 512)


SWEEP_CASES = [
    # (N, m, n, r, block_rows, block_cols)
    (3, 200, 384, 128, 0, 128),     # run 1; last row block 72 rows (third wave partly, fourth wholly past M)
    (4, 1000, 2048, 96, 0, 128),    # run 1, rank 96
    (6, 1100, 1664, 64, 64, 64),    # run 1, rank 64, block rows of 64, a block per tile
    (10, 1000, 1664, 128, 0, 256),  # run 2 across row blocks (13 units per row)
    (24, 512, 1536, 64, 32, 0),     # run 2, block rows of 32 (one per wave), whole rows
    (20, 640, 2048, 128, 0, 0),     # run 3 across ranks (80 units per rank), per-tensor scale
    (23, 800, 1664, 128, 0, 128),   # run 4 across row blocks and ranks, partial last run
]


@pytest.mark.parametrize("N,m,n,r,br,bc", SWEEP_CASES)
def test_sweep_matches_unit_kernel_and_oracle(ctx, N, m, n, r, br, bc):
    say(f"sweep encode N={N} m={m} n={n} r={r} block=({br},{bc}) run={run_length(N, m, n)}")
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(7 + r, 4 * n, n)[0]), r).to_f32()
    f = gift.Factor(ctx, m, n, r, gift.SIDE_INPUT)
    f.import_(gift.SIDE_INPUT, t(fA.U.astype(np.float32)), t(fA.c_fwd.astype(np.float32)),
              t(fA.c_inv.astype(np.float32)), t(np.array([fA.sigma2], np.float32)))
    grads = gradient_set(300 + m, 400 + n, N, m, n)
    g = t(grads)
    nbr, nbc = gift.scale_grid(m, n, br, bc)
    codes_s = torch.empty((N, m, n), dtype=torch.uint8, device=DEV)
    scales_s = torch.full((N, nbr, nbc), float("nan"), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes_s, scales_s, br, bc, gift.SCALE_LOCAL)        # sweep
    codes_u = torch.empty_like(codes_s)
    scales_u = torch.full_like(scales_s, float("nan"))
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes_u, scales_u, br, bc, gift.SCALE_LOCAL, transformed=tr)   # per unit
    torch.cuda.synchronize()
    assert torch.equal(scales_s, scales_u)
    assert torch.equal(codes_s, codes_u)
    trh = tr.cpu().numpy()
    e = rel(trh, codec.forward(grads, fA, None))
    say(f"  W~ rel. error {e:.2e}")
    assert e <= 1e-5
    # per-rank scales: the oracle quantizes ranks independently, so three of
    # them (first, middle, last) stand for all at the largest sizes
    idx = sorted({0, N // 2, N - 1})
    ref_codes, ref_scales = codec.quantize_transformed(trh[idx], br, bc, False)
    np.testing.assert_array_equal(scales_s.cpu().numpy()[idx], ref_scales)
    np.testing.assert_array_equal(codes_s.cpu().numpy()[idx], ref_codes)
    # a second call on the same context reuses its buffers (the sub-slot sets
    # alternate and are cleared by the quantize pass): the same codes again
    codes_2 = torch.empty_like(codes_s)
    scales_2 = torch.empty_like(scales_s)
    gift.encode(ctx, f, g, codes_2, scales_2, br, bc, gift.SCALE_LOCAL)
    torch.cuda.synchronize()
    assert torch.equal(codes_2, codes_s) and torch.equal(scales_2, scales_s)
    f.close()


EF_CASES = [
    # (N, m, n, r, block_rows, block_cols): ranks 64 (W two tiles ahead), 96 and
    # 128 (one tile ahead), runs across row blocks and ranks
    (10, 1000, 1664, 64, 0, 128),
    (6, 520, 1536, 96, 0, 256),
    (23, 800, 1664, 128, 0, 128),
]


@pytest.mark.parametrize("N,m,n,r,br,bc", EF_CASES)
def test_sweep_error_feedback_matches_unit_kernel(ctx, N, m, n, r, br, bc):
    """Two error-feedback steps (Algorithm 1, GIFT branch: encode W + R, R <-
    W~ - dequantized codes) through the sweep kernels and through the
    per-unit kernel (the encode that stores W~): codes, scales and the
    residual bit-identical after each step."""
    say(f"sweep error feedback N={N} m={m} n={n} r={r} block=({br},{bc}) run={run_length(N, m, n)}")
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(17 + r, 4 * n, n)[0]), r).to_f32()
    f = gift.Factor(ctx, m, n, r, gift.SIDE_INPUT)
    f.import_(gift.SIDE_INPUT, t(fA.U.astype(np.float32)), t(fA.c_fwd.astype(np.float32)),
              t(fA.c_inv.astype(np.float32)), t(np.array([fA.sigma2], np.float32)))
    nbr, nbc = gift.scale_grid(m, n, br, bc)
    ef_s = torch.zeros((N, m, n), dtype=torch.float32, device=DEV)
    ef_u = torch.zeros_like(ef_s)
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    for step in range(2):
        g = t(gradient_set(500 + step + m, 600 + n, N, m, n))
        codes_s = torch.empty((N, m, n), dtype=torch.uint8, device=DEV)
        scales_s = torch.full((N, nbr, nbc), float("nan"), dtype=torch.float32, device=DEV)
        gift.encode(ctx, f, g, codes_s, scales_s, br, bc, gift.SCALE_LOCAL, ef=ef_s)                 # sweep
        codes_u = torch.empty_like(codes_s)
        scales_u = torch.full_like(scales_s, float("nan"))
        gift.encode(ctx, f, g, codes_u, scales_u, br, bc, gift.SCALE_LOCAL, ef=ef_u, transformed=tr)  # per unit
        torch.cuda.synchronize()
        assert torch.equal(scales_s, scales_u), f"step {step}: scales differ"
        assert torch.equal(codes_s, codes_u), f"step {step}: codes differ"
        assert torch.equal(ef_s, ef_u), f"step {step}: residuals differ"
        assert float(ef_s.abs().max()) > 0.0
    f.close()


BOTH_CASES = [
    # (N, m, n, r, block_rows, block_cols)
    (3, 200, 384, 128, 0, 128),     # run 1, ragged last row block
    (4, 1000, 2048, 96, 0, 128),    # run 1, rank 96
    (6, 1100, 1664, 64, 64, 64),    # run 1, rank 64, a block per tile
    (10, 1000, 1664, 128, 0, 256),  # run 2 across row blocks
    (20, 640, 2048, 128, 0, 0),     # run 3 across ranks, per-tensor scale
    (23, 800, 1664, 128, 0, 128),   # run 4 across row blocks and ranks, partial last run
]


@pytest.mark.parametrize("N,m,n,r,br,bc", BOTH_CASES)
def test_two_sided_sweep_matches_unit_kernel_and_oracle(ctx, N, m, n, r, br, bc):
    say(f"two-sided sweep encode N={N} m={m} n={n} r={r} block=({br},{bc}) run={run_length(N, m, n)}")
    fA = codec.lowrank_factor(codec.factor_statistics(factor_inputs(27 + r, 4 * n, n)[0]), r).to_f32()
    fG = codec.lowrank_factor(codec.factor_statistics(factor_inputs(37 + r, 4 * m, m)[0]), r).to_f32()
    f = gift.Factor(ctx, m, n, r, gift.SIDE_BOTH)
    for side, fx in ((gift.SIDE_INPUT, fA), (gift.SIDE_OUTPUT, fG)):
        f.import_(side, t(fx.U.astype(np.float32)), t(fx.c_fwd.astype(np.float32)),
                  t(fx.c_inv.astype(np.float32)), t(np.array([fx.sigma2], np.float32)))
    grads = gradient_set(700 + m, 800 + n, N, m, n)
    g = t(grads)
    nbr, nbc = gift.scale_grid(m, n, br, bc)
    codes_s = torch.empty((N, m, n), dtype=torch.uint8, device=DEV)
    scales_s = torch.full((N, nbr, nbc), float("nan"), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes_s, scales_s, br, bc, gift.SCALE_LOCAL)        # sweep
    codes_u = torch.empty_like(codes_s)
    scales_u = torch.full_like(scales_s, float("nan"))
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes_u, scales_u, br, bc, gift.SCALE_LOCAL, transformed=tr)
    torch.cuda.synchronize()
    assert torch.equal(scales_s, scales_u)
    assert torch.equal(codes_s, codes_u)
    if r >= 96:
        # at rank 96 or 128 both calls above store W~ in the AMAX pass and
        # quantize the stored values; with a (zero) residual the encode
        # forms W~ + R in both passes with the per-unit kernels instead:
        # the same codes and scales
        codes_e = torch.empty_like(codes_s)
        scales_e = torch.full_like(scales_s, float("nan"))
        ef = torch.zeros((N, m, n), dtype=torch.float32, device=DEV)
        gift.encode(ctx, f, g, codes_e, scales_e, br, bc, gift.SCALE_LOCAL, ef=ef)
        torch.cuda.synchronize()
        assert torch.equal(scales_e, scales_s)
        assert torch.equal(codes_e, codes_s)
    # first, middle and last rank against the float64 transform and the
    # oracle's quantization of the stored W~
    idx = sorted({0, N // 2, N - 1})
    trh = tr.cpu().numpy()[idx]
    e = rel(trh, codec.forward(grads[idx], fA, fG))
    say(f"  W~ rel. error {e:.2e}")
    assert e <= 1e-5
    ref_codes, ref_scales = codec.quantize_transformed(trh, br, bc, False)
    np.testing.assert_array_equal(scales_s.cpu().numpy()[idx], ref_scales)
    np.testing.assert_array_equal(codes_s.cpu().numpy()[idx], ref_codes)
    codes_2 = torch.empty_like(codes_s)
    scales_2 = torch.empty_like(scales_s)
    gift.encode(ctx, f, g, codes_2, scales_2, br, bc, gift.SCALE_LOCAL)
    torch.cuda.synchronize()
    assert torch.equal(codes_2, codes_s) and torch.equal(scales_2, scales_s)
    f.close()

"""Full-size parity on the three small workloads (runs on an MI355X).

* single 256 x 256 matrix: 4 ranks, rank-16 input-side factor from 1024 float32
  tokens, per-tensor scales;
* one 1024 x 1024 attention projection: 8 ranks, rank 64, factors from 8192
  float32 tokens (the statistics run on the float32 tile kernel), per-tensor
  scales; input side and both sides;
* the Llama-300M MLP pair: up and gate 2816 x 1024, down 1024 x 2816, 8 ranks,
  rank 64, factors from 16384 bf16 tokens (the bf16 statistics kernel),
  per-128-column scale blocks.

Every call is the API call the benchmark makes, at the workload's own sizes,
and every output is checked whole (these sizes fit the oracle):
* statistics A = X^T X / T element by element under the rigorous float32
  summation bound |A_gpu - A| <= (gamma_T + u) |X|^T |X| / T (eq.
  kfac_fisher_block, eq. impl_A_psd);
* the refreshed factor captures at least 0.999 of the exact top-r eigenvalue
  sum of the oracle's statistics (Sec. V-B; the iterative factor itself is
  not pinned to eigh on these power-law spectra);
* W~ within 1e-5 of the float64 transform with the GPU's factor (eq.
  design_input_side_transform / design_full_transform); codes and scales
  bit-exact against the oracle's quantization of that W~, and the timed
  encode (no stored W~) gives the same codes and scales;
* the rank sum bit-exact (eq. dp_grad_avg); the decode within 1e-5 of the
  oracle's inverse of the GPU rank mean; the decoded gradient within 2e-3 of
  the oracle's own round trip with the same factor.
"""

import numpy as np
import pytest
import torch

from oracle import codec
from synth import factor_inputs, gradient_set, seed_for
from synth.configs import WORKLOADS

pytestmark = pytest.mark.gpu

gift = pytest.importorskip("paper_2607_07494_amd.gift")

DEV = "cuda"
U32 = 2.0 ** -24


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


def device_stats_input(wl, seed, dim):
    x, bits = factor_inputs(seed, wl.T, dim, dtype=wl.act_dtype)
    if wl.act_dtype == "bf16":
        xt = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(DEV)
    else:
        xt = torch.from_numpy(x).to(DEV)
    return x, xt


def check_statistics(ctx, x, xt):
    T, dim = x.shape
    A = torch.full((dim, dim), float("nan"), dtype=torch.float32, device=DEV)
    gift.statistics(ctx, xt, A)
    torch.cuda.synchronize()
    got = A.cpu().numpy().astype(np.float64)
    ref = codec.factor_statistics(x)
    assert np.all(np.isfinite(got))
    ax = np.abs(x.astype(np.float64))
    bound = (T * U32 / (1 - T * U32) + U32) * (ax.T @ ax) / T + 1e-30
    worst = float(np.max(np.abs(got - ref) / bound))
    say(f"  statistics T={T} dim={dim}: worst error / bound {worst:.3f}, "
        f"rel {rel(got, ref):.2e}")
    assert worst <= 1.0
    assert rel(got, ref) <= 5e-6
    return ref


def exported(f, side):
    U, cf, ci, s2 = (t.cpu().numpy().astype(np.float64) for t in f.export(side))
    return codec.Factor(U, cf, ci, float(s2[0]))


def check_energy(A, fx, r, label):
    lam = np.linalg.eigvalsh(A)[::-1][:r]
    captured = float(np.trace(fx.U.T @ A @ fx.U))
    say(f"  {label}: captured energy {captured / lam.sum():.6f} of the top-{r} sum")
    assert captured >= 0.999 * lam.sum()


def run_matrix(ctx, wl, mat, sides):
    N, r = wl.N, wl.rank
    m, n = mat.m, mat.n
    br, bc = wl.block_rows, wl.block_cols
    say(f"config {wl.cfg} {mat.name}: N={N} m={m} n={n} r={r} T={wl.T} {wl.act_dtype} "
        f"sides={sides} block=({br},{bc})")
    grads = gradient_set(seed_for(wl.cfg, 0, 0, mat.kind), seed_for(wl.cfg, 100, 0, mat.kind), N, m, n)
    f = gift.Factor(ctx, m, n, r, sides, seed=seed_for(wl.cfg, 50, 0, mat.kind))
    acts = dg = None
    A = G = None
    if sides & gift.SIDE_INPUT:
        x, acts = device_stats_input(wl, seed_for(wl.cfg, 1, 0, n % 97), n)
        A = check_statistics(ctx, x, acts)
    if sides & gift.SIDE_OUTPUT:
        d, dg = device_stats_input(wl, seed_for(wl.cfg, 2, 0, m % 97), m)
        G = check_statistics(ctx, d, dg)
    f.update(acts=acts, out_grads=dg, iters=6)     # the benchmark's cold refresh, then a warm one
    f.update(acts=acts, out_grads=dg, iters=1)
    torch.cuda.synchronize()
    fA = exported(f, gift.SIDE_INPUT) if A is not None else None
    fG = exported(f, gift.SIDE_OUTPUT) if G is not None else None
    if fA is not None:
        check_energy(A, fA, r, "input side")
    if fG is not None:
        check_energy(G, fG, r, "output side")

    g = torch.from_numpy(grads).to(DEV)
    nbr, nbc = gift.scale_grid(m, n, br, bc)
    codes = torch.empty((N, m, n), dtype=torch.uint8, device=DEV)
    scales = torch.empty((N, nbr, nbc), dtype=torch.float32, device=DEV)
    mean = torch.empty((m, n), dtype=torch.float32, device=DEV)
    out = torch.empty((m, n), dtype=torch.float32, device=DEV)
    # the timed calls
    gift.encode(ctx, f, g, codes, scales, br, bc, gift.SCALE_LOCAL)
    gift.reduce_local(ctx, codes, scales, mean, br, bc)
    gift.decode(ctx, f, mean, out)
    # the same encode storing W~
    codes2 = torch.empty_like(codes)
    scales2 = torch.empty_like(scales)
    tr = torch.empty((N, m, n), dtype=torch.float32, device=DEV)
    gift.encode(ctx, f, g, codes2, scales2, br, bc, gift.SCALE_LOCAL, transformed=tr)
    torch.cuda.synchronize()
    assert torch.equal(codes, codes2) and torch.equal(scales, scales2)
    trh = tr.cpu().numpy()
    e = rel(trh, codec.forward(grads, fA, fG))
    say(f"  W~ rel. error {e:.2e}")
    assert e <= 1e-5
    ref_codes, ref_scales = codec.quantize_transformed(trh, br, bc, False)
    got_codes, got_scales = codes.cpu().numpy(), scales.cpu().numpy()
    np.testing.assert_array_equal(got_scales, ref_scales)
    np.testing.assert_array_equal(got_codes, ref_codes)
    got_mean = mean.cpu().numpy()
    np.testing.assert_array_equal(got_mean, codec.reduce_local(got_codes, got_scales, br, bc))
    got_out = out.cpu().numpy()
    e = rel(got_out, codec.decode(got_mean, fA, fG))
    say(f"  decode rel. error {e:.2e}")
    assert e <= 1e-5
    e = rel(got_out, codec.round_trip(grads, fA, fG, br, bc, False))
    say(f"  round trip vs oracle {e:.2e}")
    assert e <= 2e-3
    f.close()


def test_config1_single_matrix(ctx):
    wl = WORKLOADS[1]
    run_matrix(ctx, wl, wl.matrices[0], gift.SIDE_INPUT)


@pytest.mark.parametrize("sides", [gift.SIDE_INPUT, gift.SIDE_BOTH])
def test_config2_attention_projection(ctx, sides):
    wl = WORKLOADS[2]
    run_matrix(ctx, wl, wl.matrices[0], sides)


@pytest.mark.parametrize("name", ["up", "gate", "down"])
def test_config3_mlp_pair(ctx, name):
    wl = WORKLOADS[3]
    run_matrix(ctx, wl, next(mt for mt in wl.matrices if mt.name == name), gift.SIDE_INPUT)

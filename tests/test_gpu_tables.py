"""Device tables of the factor refresh (runs on an MI355X).

The refresh's member / job tables, the statistics pointer table and the
Cholesky block tables live in context buffers uploaded only when their
contents change.  Two contexts run the same refresh sequence on factors with
the same seeds; one of them also refreshes other factor sets and statistics
inputs in between (forcing new uploads and switches between cached tables).
Every exported factor and every statistics result must be bit-identical
between the two, and a repeated refresh on a context whose tables are cached
must equal one on a fresh context.
"""

import numpy as np
import pytest
import torch

from synth import factor_inputs

pytestmark = pytest.mark.gpu

gift = pytest.importorskip("paper_2607_07494_amd.gift")
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def bf16(seed, T, dim):
    _, bits = factor_inputs(seed, T, dim, dtype="bf16")
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(DEV)


def exported(f):
    out = []
    for side in (gift.SIDE_INPUT, gift.SIDE_OUTPUT):
        if f.sides & side:
            out += [x.cpu().numpy() for x in f.export(side)]
    return out


def test_repeated_refresh_with_cached_and_switched_tables():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    T = 2048
    shapes = [(192, 256, 16, gift.SIDE_INPUT), (256, 256, 16, gift.SIDE_INPUT), (160, 128, 8, gift.SIDE_BOTH)]
    acts = [bf16(70 + i, T, n) for i, (m, n, r, s) in enumerate(shapes)]
    grads = [bf16(80 + i, T, m) if s & gift.SIDE_OUTPUT else None for i, (m, n, r, s) in enumerate(shapes)]
    other_x = bf16(90, T, 512)
    results = []
    for interleave in (False, True):
        say(f"refresh sequence, interleaved work: {interleave}")
        ctx = gift.Context()
        fs = [gift.Factor(ctx, m, n, r, s, seed=5 + i) for i, (m, n, r, s) in enumerate(shapes)]
        other = gift.Factor(ctx, 64, 512, 8, gift.SIDE_INPUT, seed=99)
        chol = gift.CholFactor(ctx, 64, 256, 32, gift.SIDE_INPUT, 1e-4)
        A = torch.empty((512, 512), dtype=torch.float32, device=DEV)
        stats = []
        got = []
        for it, iters in enumerate((6, 1, 1, 2)):
            gift.factor_update_batch(ctx, fs, acts, grads, iters=iters)
            if interleave:
                other.update(acts=other_x, iters=2)             # another refresh table
                chol.update(acts=acts[1], iters=0)              # Cholesky statistics and block tables
                gift.statistics(ctx, other_x, A)                # the statistics pointer table
                stats.append(A.clone())
                gift.statistics(ctx, acts[1], A[:256, :256].contiguous())
            torch.cuda.synchronize()
            got.append([x for f in fs for x in exported(f)])
        if interleave:
            ref = torch.empty_like(A)
            ctx2 = gift.Context()
            gift.statistics(ctx2, other_x, ref)
            torch.cuda.synchronize()
            for s_ in stats:
                assert torch.equal(s_, ref)
            ctx2.close()
        results.append(got)
        for f in fs + [other, chol]:
            f.close()
        ctx.close()
    for a, b in zip(results[0], results[1]):
        assert len(a) == len(b)
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)

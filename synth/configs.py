"""The five synthetic workloads the codec is tested and measured on.

Shapes follow the paper's Llama pretraining setups (Sec. VI-A: ~300M with
hidden 1024, ~600M with hidden 1536) with gradient matrices laid out as
``W_g in R^{d_out x d_in}`` (Sec. IV-A), so ``m = d_out`` and ``n = d_in``.
This module only describes workloads; it computes nothing of the method.

Readings that the paper leaves open (kept in one place so tests and bench
agree):

* Per-block scaling uses column slabs: ``block_rows = m`` (0), ``block_cols =
  128``.
* In the Llama-300M set the GIFT branch covers the MLP matrices (gate, up,
  down, local scale) and the attention projections take the Euclidean branch
  with a shared scale (Algorithm 1).  The embedding and an untied LM head
  (32000 x 1024) are added as Euclidean matrices.
* In the Llama-600M set every projection takes the GIFT branch; the factors
  are refreshed every 50 steps (Sec. V-E).
"""

from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Matrix:
    name: str
    m: int            # d_out
    n: int            # d_in
    gift: bool        # geometry-aware branch (True) or Euclidean branch
    act: str          # key of the activation stream feeding A (shared by
                      # matrices that read the same layer input)
    kind: int         # matrix-kind id used in the seed layout


@dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    N: int                 # simulated data-parallel ranks
    rank: int              # low-rank transform rank r
    T: int                 # tokens behind the factor statistics
    act_dtype: str         # "f32" or "bf16"
    block_rows: int        # 0 = whole m
    block_cols: int        # 0 = whole n
    layers: int
    matrices: tuple = field(default_factory=tuple)   # per layer
    extra: tuple = field(default_factory=tuple)      # once per model
    refresh: int = 1       # factor refresh cadence in steps

    def all_matrices(self):
        """(layer, Matrix) pairs in step order."""
        out = []
        for layer in range(self.layers):
            for mat in self.matrices:
                out.append((layer, mat))
        for mat in self.extra:
            out.append((-1, mat))
        return out

    def grad_elements(self):
        return sum(mat.m * mat.n for _, mat in self.all_matrices())


def _llama_layer(hidden: int, mlp: int, attn_gift: bool):
    return (
        Matrix("q", hidden, hidden, attn_gift, "attn_in", 1),
        Matrix("k", hidden, hidden, attn_gift, "attn_in", 2),
        Matrix("v", hidden, hidden, attn_gift, "attn_in", 3),
        Matrix("o", hidden, hidden, attn_gift, "attn_out", 4),
        Matrix("gate", mlp, hidden, True, "mlp_in", 5),
        Matrix("up", mlp, hidden, True, "mlp_in", 6),
        Matrix("down", hidden, mlp, True, "mlp_mid", 7),
    )


WORKLOADS = {
    1: Workload(1, "single-256x256", N=4, rank=16, T=1024, act_dtype="f32",
                block_rows=0, block_cols=0, layers=1,
                matrices=(Matrix("w", 256, 256, True, "in", 0),)),
    2: Workload(2, "attn-proj-1024x1024", N=8, rank=64, T=8192, act_dtype="f32",
                block_rows=0, block_cols=0, layers=1,
                matrices=(Matrix("w", 1024, 1024, True, "in", 0),)),
    3: Workload(3, "llama300m-mlp-pair", N=8, rank=64, T=16384, act_dtype="bf16",
                block_rows=0, block_cols=128, layers=1,
                matrices=(Matrix("up", 2816, 1024, True, "mlp_in", 6),
                          Matrix("gate", 2816, 1024, True, "mlp_in", 5),
                          Matrix("down", 1024, 2816, True, "mlp_mid", 7))),
    4: Workload(4, "llama300m-gradient-set", N=8, rank=64, T=16384,
                act_dtype="bf16", block_rows=0, block_cols=0, layers=24,
                matrices=_llama_layer(1024, 2816, attn_gift=False),
                extra=(Matrix("embed", 32000, 1024, False, "none", 8),
                       Matrix("lm_head", 32000, 1024, False, "none", 9)),
                refresh=1),
    5: Workload(5, "llama600m-gradient-set", N=16, rank=128, T=32768,
                act_dtype="bf16", block_rows=0, block_cols=128, layers=24,
                matrices=_llama_layer(1536, 4096, attn_gift=True),
                refresh=50),
}

"""Named FFF workloads (shapes, dtypes and seeds), used by tests and the benchmark.

Depth counts edges on a root-to-leaf path, so a tree of depth D has
2**(D+1) - 1 nodes and a token visits D+1 of them (UltraFastBERT-KxD naming,
Section 2.1 and Table 1 of the paper).
"""
from __future__ import annotations

from dataclasses import dataclass, field

from .synth import BF16, F32, n_nodes


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    n_tokens: int
    hidden: int
    depth: int
    n_trees: int
    x_dtype: str
    w_dtype: str
    y_dtype: str
    layers: int = 1
    note: str = ""
    sweep: tuple = field(default_factory=tuple)

    @property
    def nodes(self) -> int:
        return n_nodes(self.depth)

    def w_elem_bytes(self) -> int:
        return 2 if self.w_dtype == BF16 else 4

    def gathered_bytes_per_token(self) -> int:
        """Weight bytes one token reads: one W_in row and one W_out row per visited node."""
        return self.n_trees * (self.depth + 1) * 2 * self.hidden * self.w_elem_bytes()

    def act_elem_bytes(self) -> tuple:
        return (2 if self.x_dtype == BF16 else 4), (2 if self.y_dtype == BF16 else 4)

    def compulsory_bytes(self, n_tokens: int | None = None) -> float:
        """HBM bytes one forward cannot avoid: x read once, y written once, and every weight row
        the batch touches read once.  Under uniform routing level l has 2^l nodes, each reached
        by some token with probability 1 - (1 - 2^-l)^B, and every reached node costs one W_in
        and one W_out row."""
        B = self.n_tokens if n_tokens is None else n_tokens
        sx, sy = self.act_elem_bytes()
        rows = sum(2.0 ** l * (1.0 - (1.0 - 2.0 ** -l) ** B) for l in range(self.depth + 1))
        return B * self.hidden * (sx + sy) + self.n_trees * 2 * self.hidden * self.w_elem_bytes() * rows

    def flops_per_token(self) -> int:
        """Multiply-adds of the dot product and of the output accumulation, 2 flops each."""
        return 4 * self.hidden * self.n_trees * (self.depth + 1)


WORKLOADS = {
    # One tree of depth 3 (15 nodes): the small case the oracle finishes instantly.
    "d3_h768_b128_f32": Workload("d3_h768_b128_f32", 1, 128, 768, 3, 1, F32, F32, F32),
    # UltraFastBERT-1x11 layer at the paper's speed-test batch: 128 sequences x 128 tokens.
    "d11_h768_b16384_f32": Workload("d11_h768_b16384_f32", 2, 16384, 768, 11, 1, F32, F32, F32),
    # Same tree in bf16, 65536 tokens: the headline throughput workload.
    "d11_h768_b65536_bf16": Workload("d11_h768_b65536_bf16", 3, 65536, 768, 11, 1, BF16, BF16, BF16),
    # Same, bf16 weights with fp32 activations in and out.
    "d11_h768_b65536_w_bf16": Workload("d11_h768_b65536_w_bf16", 3, 65536, 768, 11, 1, F32, BF16, F32),
    # UltraFastBERT-4x9: four trees of depth 9 (4 x 1023 nodes), outputs summed.
    "4x9_h768_b16384_f32": Workload("4x9_h768_b16384_f32", 4, 16384, 768, 9, 4, F32, F32, F32),
    # Four trees of depth 8 (4 x 511 nodes).
    "4x8_h768_b16384_f32": Workload("4x8_h768_b16384_f32", 4, 16384, 768, 8, 4, F32, F32, F32),
    # Twelve stacked 4x9 layers with a residual, x <- x + FFF(x).
    "4x9_h768_b16384_f32_x12": Workload("4x9_h768_b16384_f32_x12", 4, 16384, 768, 9, 4, F32, F32, F32,
                                        layers=12),
    # LLM-width tree: depth 15 (65535 nodes) at hidden 4096, batch sweep.
    "d15_h4096_bf16": Workload("d15_h4096_bf16", 5, 8192, 4096, 15, 1, BF16, BF16, BF16,
                               sweep=(1, 64, 1024, 8192)),
}

HEADLINE = "d11_h768_b65536_bf16"


# The UltraFastBERT-KxD family of Table 1: K trees of depth D, all with about
# 4095 trainable neurons per layer (N_T = K * (2**(D+1) - 1)); a token uses
# N_I = K * (D+1) of them.  K = 3072, D = 0 is the dense feedforward layer of
# BERT-base.  Timed with the same kernels at the paper's speed-test batch.
KXD_FAMILY = ((3072, 0), (1536, 1), (512, 2), (256, 3), (128, 4), (64, 5), (32, 6), (16, 7), (8, 8), (4, 9),
              (2, 10), (1, 11))


def kxd_workload(k: int, d: int, dtype: str = BF16, n_tokens: int = 16384, hidden: int = 768) -> Workload:
    return Workload(f"{k}x{d}_h{hidden}_b{n_tokens}_{dtype}", 6, n_tokens, hidden, d, k, dtype, dtype, dtype,
                    note="UltraFastBERT-KxD family (Table 1)")

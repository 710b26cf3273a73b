"""Synthetic workload shapes for the factorized-cache decode path.

Each workload fixes the model shape (layers, depth-window size, KV and query
heads, head dimension), the context length(s), the shared-basis rank r_b, the
routed residual-rank levels with their draw probabilities, and the query
dtype.  The shapes follow the Llama-style decoder settings the method is
evaluated on (64K-token prefill in the experimental setup; 16K-128K contexts
for the needle sweep), with the values a serving deployment would pick.

This module holds shapes and distributions only: no arithmetic of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_layers: int
    window: int            # layers per depth window W_m
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    context: int           # tokens per sequence (fixed-length workloads)
    basis_rank: int        # r_b
    levels: tuple          # routed residual ranks, ascending
    probs: tuple           # draw probability of each level
    q_dtype: str           # "f16" or "bf16"
    seed: int
    ragged: tuple | None = None      # (lo, hi) inclusive per-sequence length range
    salient_frac: float = 0.0        # fraction of tokens inside salient spans
    salient_span: int = 64           # span length (tokens)
    salient_level: int = 0           # level index forced inside spans
    probe: bool = False              # attention-output probe on every layer
    coef_format: str = "f16"         # "f16" coefficient rows, or "int8" (8-bit blockwise)
    scale_mode: str = "uniform"      # residual scales: "uniform" U(0.01, 0.1), or "wide" (see generate)
    scale_period: int = 1024         # "wide": tokens per ramp of the scale exponent
    coef_scale_mode: str = "narrow"  # int8 block scales: "narrow" U(0.11, 0.14), or "wide"
    description: str = field(default="", compare=False)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_windows(self) -> int:
        return self.n_layers // self.window

    def seqlens(self):
        """Per-sequence token counts (ragged workloads draw them, seeded)."""
        if self.ragged is None:
            return [self.context] * self.batch
        import numpy as np
        rng = np.random.Generator(np.random.PCG64DXSM(
            np.random.SeedSequence([self.seed, 9])))
        lo, hi = self.ragged
        return [int(x) for x in rng.integers(lo, hi + 1, size=self.batch)]

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = Workload(
    name="tiny-4k", batch=1, n_layers=2, window=2, n_kv_heads=2, n_q_heads=8,
    head_dim=128, context=4096, basis_rank=32, levels=(0, 8, 16),
    probs=(0.80, 0.15, 0.05), q_dtype="f16", seed=1,
    description="1 seq, one window of 2 layers, 2 KV / 8 q heads, 4096 tokens, r_b 32")

LLAMA8B_32K = Workload(
    name="llama8b-32k", batch=1, n_layers=32, window=2, n_kv_heads=8,
    n_q_heads=32, head_dim=128, context=32768, basis_rank=32,
    levels=(0, 4, 8, 16), probs=(0.70, 0.15, 0.10, 0.05), q_dtype="bf16",
    seed=2, salient_frac=0.02, salient_span=64, salient_level=3,
    description="Llama-3-8B shape, windows of 2, 32768 tokens, r_b 32, 2% salient spans at rank 16")

LLAMA8B_64K = Workload(
    name="llama8b-64k", batch=1, n_layers=32, window=4, n_kv_heads=8,
    n_q_heads=32, head_dim=128, context=65536, basis_rank=48,
    levels=(0, 4, 8, 16), probs=(0.75, 0.12, 0.08, 0.05), q_dtype="bf16",
    seed=3,
    description="Llama-3-8B shape, windows of 4, 65536 tokens, r_b 48")

BATCH16 = Workload(
    name="batch16-ragged", batch=16, n_layers=32, window=2, n_kv_heads=8,
    n_q_heads=32, head_dim=128, context=16384, basis_rank=32,
    levels=(0, 8, 16), probs=(0.80, 0.15, 0.05), q_dtype="bf16", seed=4,
    ragged=(8192, 16384),
    description="16 sequences of 8192-16384 tokens (uniform), windows of 2, r_b 32")

LLAMA70B_128K = Workload(
    name="llama70b-128k", batch=2, n_layers=80, window=4, n_kv_heads=8,
    n_q_heads=64, head_dim=128, context=131072, basis_rank=64,
    levels=(0, 4, 8, 16, 32), probs=(0.70, 0.12, 0.10, 0.06, 0.02),
    q_dtype="bf16", seed=5, probe=True,
    description="Llama-70B shape, 2 x 131072 tokens, windows of 4, r_b 64, probe on every layer")

ALL = {w.name: w for w in (TINY, LLAMA8B_32K, LLAMA8B_64K, BATCH16, LLAMA70B_128K)}

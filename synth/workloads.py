"""Workload shapes for the compressed-KV path.

Each workload fixes the model shape (layers, KV heads, query heads, head
dimension), the residual top-k, the storage precision, the batch and context
lengths, the recipe of the synthetic cache (inter-layer correlation range and
planted needles) and how head modes are chosen.

The five named workloads are:

* ``tiny``      - 2 layers, 4 KV = 4 query heads, d=64, 512 tokens, fp32,
                  top-8, fixed modes [shared, residual, residual, exact].
* ``llama8b``   - 32 layers, 32 query heads on 8 KV heads, d=128, 32768
                  tokens, bf16, top-16, seeded 64/45/19 shared/residual/exact.
* ``batched8b`` - the llama8b shape at batch 16, ragged lengths U{4096..16384}.
* ``long70b``   - 80 layers, 64 query heads on 8 KV heads, d=128, 131072
                  tokens, bf16, top-16, seeded 128/128/64 modes.
* ``prefill8b`` - the llama8b cache (same seeded draws) plus a 256-row probe window per query
                  head; modes come from the probe and the byte budget of the
                  50/35/15 mix.

Variants: ``llama8b_e4m3`` (FP8 coefficients), ``llama8b_mixed`` (blocks of
four layers between pairs at both ends) and ``llama8b_tokres`` (token-level
residual sets of 5% of the tokens).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    topk: int
    dtype: str                     # "f32", "bf16" or "bf16_e4m3" (bf16 inputs, FP8 coefficients)
    seq_lens: Tuple[int, ...]      # one entry per sequence of the batch
    rho: Tuple[float, float]       # inter-layer correlation, U(lo, hi) per (seq, pair, head)
    n_needles: int                 # needle tokens per sequence
    needle_amp: float              # spike added to K and V at a needle
    needle_channels: int           # channels spiked per (pair, head, needle)
    needle_layer: str              # "odd": always layer 2b+1; "coin": seeded per (pair, head, needle)
    mode_counts: Optional[Tuple[int, int, int]] = None   # seeded exact S/R/E counts per sequence
    fixed_modes: Optional[Tuple[int, ...]] = None        # explicit modes per (pair, head)
    n_probe: int = 0               # probe rows per query head
    steps: int = 1                 # decode steps the workload describes
    seed: int = 0
    schedule: int = 0              # layer blocks: 0 pairs, 1 pairs-fours-pairs (first / last four layers in pairs), 2 fours
    residual: int = 0              # residual heads: 0 per-token channel top-k, 1 token-level set
    res_ppm: int = 0               # the token-level set's fraction of tokens (parts per million)
    res_rates: Tuple[int, ...] = ()  # candidate fractions routed per residual head (ppm), at most 8
    notes: str = field(default="", compare=False)

    @property
    def batch(self) -> int:
        return len(self.seq_lens)

    @property
    def n_pairs(self) -> int:
        return self.n_layers // 2

    @property
    def block_sizes(self) -> Tuple[int, ...]:
        """Layers per block, in layer order."""
        L = self.n_layers
        if self.schedule == 0:
            return (2,) * (L // 2)
        if self.schedule == 2:
            return (4,) * (L // 4)
        return (2, 2) + (4,) * ((L - 8) // 4) + (2, 2)

    @property
    def blocks(self) -> Tuple[Tuple[int, int], ...]:
        """``(first layer, size)`` of every block."""
        out, first = [], 0
        for B in self.block_sizes:
            out.append((first, B))
            first += B
        return tuple(out)

    @property
    def n_blocks(self) -> int:
        return len(self.block_sizes)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def max_seq_len(self) -> int:
        return max(self.seq_lens)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2   # input elements

    @property
    def coef_bytes(self) -> int:
        """Bytes per stored shared / residual coefficient."""
        return 1 if self.dtype == "bf16_e4m3" else self.elem_bytes

    def dims(self) -> dict:
        return dict(n_layers=self.n_layers, n_kv_heads=self.n_kv_heads,
                    n_q_heads=self.n_q_heads, head_dim=self.head_dim,
                    topk=self.topk, dtype=self.dtype, schedule=self.schedule,
                    residual=self.residual, res_ppm=self.res_ppm, res_rates=tuple(self.res_rates))


def _ragged_lengths(seed: int, cfg_id: int, batch: int, lo: int, hi: int) -> Tuple[int, ...]:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, cfg_id, 7777])))
    return tuple(int(x) for x in rng.integers(lo, hi + 1, size=batch))


def scaled(w: Workload, **over) -> Workload:
    """A copy of ``w`` with some fields replaced (used for small parity cases)."""
    return dataclasses.replace(w, **over)


TINY = Workload(
    name="tiny", cfg_id=1, n_layers=2, n_kv_heads=4, n_q_heads=4, head_dim=64,
    topk=8, dtype="f32", seq_lens=(512,), rho=(0.9, 0.9), n_needles=4,
    needle_amp=6.0, needle_channels=8, needle_layer="odd",
    fixed_modes=(0, 1, 1, 2), n_probe=32, steps=1,
    notes="2 layers, 4 KV heads = 4 query heads, d=64, 512 tokens, fp32, top-8",
)

LLAMA8B = Workload(
    name="llama8b", cfg_id=2, n_layers=32, n_kv_heads=8, n_q_heads=32, head_dim=128,
    topk=16, dtype="bf16", seq_lens=(32768,), rho=(0.75, 0.95), n_needles=16,
    needle_amp=5.0, needle_channels=16, needle_layer="coin",
    mode_counts=(64, 45, 19), n_probe=256, steps=100,
    notes="Llama-3-8B-shaped decode: 32 layers, 32 q heads on 8 KV heads, d=128, 32k tokens, bf16",
)

BATCHED8B = Workload(
    name="batched8b", cfg_id=3, n_layers=32, n_kv_heads=8, n_q_heads=32, head_dim=128,
    topk=16, dtype="bf16", seq_lens=_ragged_lengths(0, 3, 16, 4096, 16384),
    rho=(0.75, 0.95), n_needles=16, needle_amp=5.0, needle_channels=16,
    needle_layer="coin", mode_counts=(64, 45, 19), n_probe=256, steps=100,
    notes="8B shape, batch 16, ragged lengths U{4096..16384}",
)

LONG70B = Workload(
    name="long70b", cfg_id=4, n_layers=80, n_kv_heads=8, n_q_heads=64, head_dim=128,
    topk=16, dtype="bf16", seq_lens=(131072,), rho=(0.70, 0.95), n_needles=64,
    needle_amp=5.0, needle_channels=16, needle_layer="coin",
    mode_counts=(128, 128, 64), n_probe=256, steps=100,
    notes="70B-shaped decode on one GPU's cache share: 80 layers, 64 q heads on 8 KV heads, 131k tokens",
)

PREFILL8B = Workload(
    name="prefill8b", cfg_id=2, n_layers=32, n_kv_heads=8, n_q_heads=32, head_dim=128,
    topk=16, dtype="bf16", seq_lens=(32768,), rho=(0.75, 0.95), n_needles=16,
    needle_amp=5.0, needle_channels=16, needle_layer="coin",
    mode_counts=(64, 45, 19), n_probe=256, steps=1,
    notes="prefill probe + route + compress on the 8B cache, 256 probe rows per query head",
)

# the 8B decode workload with its shared / residual coefficients stored as FP8 E4M3
LLAMA8B_E4M3 = dataclasses.replace(
    LLAMA8B, name="llama8b_e4m3", dtype="bf16_e4m3",
    notes="llama8b with FP8 E4M3 shared planes and residual values (bf16 inputs and exact heads)")

# the 8B decode workload under the paper's default block setting: pairs for the first
# and last four layers, blocks of four between (10 blocks of 8 KV heads)
LLAMA8B_MIXED = dataclasses.replace(
    LLAMA8B, name="llama8b_mixed", schedule=1,
    notes="llama8b with blocks of four layers between pairs at both ends (the default block setting)")

# the 8B workload with the paper's token-level residual rule: residual heads keep every
# high-frequency coefficient of the 5% of tokens with the largest probe-logit change
LLAMA8B_TOKRES = dataclasses.replace(
    LLAMA8B, name="llama8b_tokres", topk=0, residual=1, res_ppm=50000,
    notes="llama8b with token-level residual sets (5% of tokens per residual head)")

# the token-level sets with the fraction chosen per residual head by the routing budget among
# five candidates (Section 3: r_{b,h} by the routing loss budget)
LLAMA8B_TOKRATES = dataclasses.replace(
    LLAMA8B, name="llama8b_tokrates", topk=0, residual=1, res_ppm=0, res_rates=(10000, 25000, 50000, 100000, 200000),
    notes="llama8b with token-level residual sets whose fraction (1% .. 20%) is routed per residual head")

WORKLOADS = {w.name: w for w in (TINY, LLAMA8B, BATCHED8B, LONG70B, PREFILL8B, LLAMA8B_E4M3, LLAMA8B_MIXED,
                                 LLAMA8B_TOKRES, LLAMA8B_TOKRATES)}

"""Seeded synthetic workloads shaped like the paper's training layers.

The paper trains on its own data and models, which are not available; these synthetic tensors stand in
for them. Nothing here computes any part of the quantization method: the module only draws bf16
tensors, sign masks, seeds and MoE group sizes, and is shared by the tests, the benchmark and the oracle
checks.

Every tensor is drawn on the CPU with ``torch.Generator().manual_seed(seed)`` in fp32, in the order
written below, then rounded to bf16.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

# ---------------------------------------------------------------------------------------------------
# MoE expert loads: Zipf(1.1) over experts (rank order = expert order), optionally capped
# ---------------------------------------------------------------------------------------------------


def zipf_counts(total: int, experts: int, exponent: float = 1.1, cap: int | None = None) -> list[int]:
    """Split `total` routed rows over `experts` with load proportional to rank^-exponent.

    Loads above `cap` are clipped to it and the excess is spread over the uncapped experts in proportion
    to their weights (repeated until no load exceeds the cap). Fractional loads are rounded by the
    largest-remainder method so the counts add up to `total`.
    """
    w = np.arange(1, experts + 1, dtype=np.float64) ** (-exponent)
    share = total * w / w.sum()
    if cap is not None:
        if cap * experts < total:
            raise ValueError("cap too small for the total")
        fixed = np.zeros(experts, dtype=bool)
        while True:
            over = (share > cap) & ~fixed
            if not over.any():
                break
            fixed |= over
            share[fixed] = cap
            rest = total - cap * fixed.sum()
            share[~fixed] = rest * w[~fixed] / w[~fixed].sum()
    base = np.floor(share).astype(np.int64)
    short = int(total - base.sum())
    order = np.argsort(-(share - base), kind="stable")
    base[order[:short]] += 1
    return [int(c) for c in base]


# ---------------------------------------------------------------------------------------------------
# Workload records
# ---------------------------------------------------------------------------------------------------


@dataclass
class LayerWorkload:
    """One linear layer: X [M, K], W [N, K] (or [E, N, K] for experts), dY [M, N], bf16 on the CPU."""

    name: str
    x: torch.Tensor
    w: torch.Tensor
    dy: torch.Tensor
    sign_mask: int
    seed: int
    counts: list[int] | None = None  # rows of X / dY per expert (expert-contiguous), None for dense
    extra: dict = field(default_factory=dict)

    @property
    def grouped(self) -> bool:
        return self.counts is not None


def _normal(g: torch.Generator, shape, std: float = 1.0) -> torch.Tensor:
    t = torch.randn(*shape, generator=g, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t


def _outlier_channels(g: torch.Generator, x: torch.Tensor, frac: float = 0.001, factor: float = 50.0):
    """Scale round(frac * channels) randomly chosen input channels (columns) of x by `factor`."""
    k = x.shape[1]
    n_out = max(1, int(round(frac * k)))
    ch = torch.randperm(k, generator=g)[:n_out]
    x[:, ch] *= factor
    return ch


def _student_t3_unit(g: torch.Generator, shape) -> torch.Tensor:
    """Student-t with 3 degrees of freedom, scaled to unit variance (variance of t_3 is 3)."""
    z = torch.randn(*shape, generator=g, dtype=torch.float32)
    chi2 = torch.zeros(*shape, dtype=torch.float32)
    for _ in range(3):
        chi2.add_(torch.randn(*shape, generator=g, dtype=torch.float32).square_())
    return z / torch.sqrt(chi2 / 3.0) / np.sqrt(3.0)


def _mask(g: torch.Generator) -> int:
    return int(torch.randint(0, 65536, (1,), generator=g).item())


def tiny(seed: int = 0) -> LayerWorkload:
    """Single small linear layer: X 256x256, W 512x256, dY 256x512, entries N(0,1)."""
    g = torch.Generator().manual_seed(seed)
    x = _normal(g, (256, 256))
    w = _normal(g, (512, 256))
    dy = _normal(g, (256, 512))
    m = _mask(g)
    return LayerWorkload("tiny 256x256x512", x.bfloat16(), w.bfloat16(), dy.bfloat16(), m, seed)


def dense_ffn(seed: int = 2, tokens: int = 8192, hidden: int = 2048, ffn: int = 8192) -> LayerWorkload:
    """Dense-1.5B-shaped FFN up-projection: X [tokens, hidden] N(0,1) with 0.1% of channels x50,
    W [ffn, hidden] N(0, 0.02^2), dY [tokens, ffn] N(0, 1e-3^2)."""
    g = torch.Generator().manual_seed(seed)
    x = _normal(g, (tokens, hidden))
    ch = _outlier_channels(g, x)
    w = _normal(g, (ffn, hidden), 0.02)
    dy = _normal(g, (tokens, ffn), 1e-3)
    m = _mask(g)
    return LayerWorkload(f"dense-1.5B FFN {tokens}x{hidden}->{ffn}", x.bfloat16(), w.bfloat16(),
                         dy.bfloat16(), m, seed, extra={"outlier_channels": ch.tolist()})


def moe_experts(seed: int, experts: int, hidden: int, ffn: int, routed: int, cap: int | None,
                student_t: bool, name: str) -> LayerWorkload:
    """Expert layer: routed X [routed, hidden] (expert-contiguous rows, Zipf(1.1) loads),
    W [experts, ffn, hidden] N(0, 0.02^2), dY [routed, ffn] N(0, 1e-3^2)."""
    g = torch.Generator().manual_seed(seed)
    counts = zipf_counts(routed, experts, 1.1, cap)
    if student_t:
        x = _student_t3_unit(g, (routed, hidden))
    else:
        x = _normal(g, (routed, hidden))
        _outlier_channels(g, x)
    w = _normal(g, (experts, ffn, hidden), 0.02)
    dy = _normal(g, (routed, ffn), 1e-3)
    m = _mask(g)
    return LayerWorkload(name, x.bfloat16(), w.bfloat16(), dy.bfloat16(), m, seed, counts=counts)


def moe_7_9b(seed: int = 3) -> LayerWorkload:
    """MoE-7.9B-shaped layer: 64 experts, hidden 2048 -> 1408, 16384 tokens routed top-6 (98304 rows),
    at most 16384 rows per expert."""
    return moe_experts(seed, 64, 2048, 1408, 16384 * 6, 16384, False, "MoE-7.9B experts 64x(2048->1408)")


def moe_124b_share(seed: int = 4) -> LayerWorkload:
    """One GPU's expert share of a MoE-124B-shaped layer: 8 experts, hidden 5120 -> 3072, 32768 routed
    rows, Student-t(3) activations."""
    return moe_experts(seed, 8, 5120, 3072, 32768, None, True, "MoE-124B share 8x(5120->3072)")


def square(seed: int = 5, n: int = 16384) -> LayerWorkload:
    """Square stress layer: X, W, dY all n x n, N(0,1)."""
    g = torch.Generator().manual_seed(seed)
    x = _normal(g, (n, n))
    w = _normal(g, (n, n))
    dy = _normal(g, (n, n))
    m = _mask(g)
    return LayerWorkload(f"square {n}^3", x.bfloat16(), w.bfloat16(), dy.bfloat16(), m, seed)


def quantizer_tensor(seed: int = 5, rows: int = 32768, cols: int = 16384) -> torch.Tensor:
    """Standalone quantizer input, N(0,1) bf16; 32768 x 16384 is 1 GiB."""
    g = torch.Generator().manual_seed(seed + 1000)
    return _normal(g, (rows, cols)).bfloat16()


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw uint16 bit patterns of a CPU bf16 tensor (a view, no copy)."""
    if t.dtype != torch.bfloat16:
        raise TypeError("expected a bfloat16 tensor")
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


CONFIGS = {
    "tiny": tiny,
    "dense": dense_ffn,
    "moe7.9b": moe_7_9b,
    "moe124b": moe_124b_share,
    "square": square,
}

"""Controlled randomness (Sec. III-B): how many distinct sampler seeds G GPUs
use, and which GPU uses which.

With a seed per GPU the sampled softmax keeps its accuracy but the union of
the sampled words grows with G; with one seed the union is small but every
GPU samples the same words. The paper finds that G^alpha seeds (alpha = 0.64,
the exponent of the type/token power law) match the accuracy of G seeds, and
also evaluates log2 G, ln G and log10 G seeds. A rule giving a fraction is
rounded up (at least that many seeds), and the GPUs are split into that many
contiguous groups of equal size (to within one), a group sharing a seed.
"""
from __future__ import annotations

import math

RULES = ("G", "pow0.64", "log2", "ln", "log10", "one")


def num_seeds(G: int, rule: str, alpha: float = 0.64) -> int:
    """Distinct seeds for G GPUs under a rule of Sec. III-B (1 <= n <= G)."""
    if G < 1:
        raise ValueError("G must be >= 1")
    x = {
        "G": float(G),
        "pow0.64": G ** alpha,
        "log2": math.log2(G),
        "ln": math.log(G),
        "log10": math.log10(G),
        "one": 1.0,
    }[rule]
    return max(1, min(G, math.ceil(x - 1e-9)))


def seed_index(g: int, G: int, n_seeds: int) -> int:
    """The seed (0 .. n_seeds-1) GPU g of G uses: floor(g * n_seeds / G)."""
    if not (0 <= g < G and 1 <= n_seeds <= G):
        raise ValueError("need 0 <= g < G and 1 <= n_seeds <= G")
    return (g * n_seeds) // G


def seed_of_gpus(G: int, rule: str) -> list:
    n = num_seeds(G, rule)
    return [seed_index(g, G, n) for g in range(G)]
